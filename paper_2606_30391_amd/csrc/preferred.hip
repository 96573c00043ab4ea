// preferred.hip -- MI355X (gfx950) kernels and C-ABI host dispatch of the preferred
// configuration of every active LLM (Festina, App. E, Eq. preferred_sm and
// Eq. preferred_frequency) and of the fleet's energy waste ratio (Sec. 3.5.1,
// Eq. energy_waste, energy_optimal, energy_waste_ratio).
//
// k_preferred: one wavefront per LLM instance slot.  For each phase the lanes span the
//   (SM level, frequency level) cells of the model's table row (prefill: the average
//   prompt's 256-token bucket, duration TTFT; decode: the batch row, duration
//   avg_out x TBT), mask cells whose latency is not strictly below the SLO, and reduce
//   (energy, cell) to the least-energy cell, lowest cell on exact ties, carrying its
//   duration and power.  Lane 0 then forms the time-weighted SM share and the
//   energy-weighted frequency.  Power is the placement model P = P0 + k*s*f^3*u with
//   u = min(B + 1, 32) / 32.
// k_ewr_single (fleets up to 16,384 GPUs, one launch) or k_ewr_gpu + k_ewr_total: a
//   thread per GPU takes F_g = the highest preferred frequency of its instances and its
//   waste sum t (F_g^3 - F_l^3) in float64; one block (or per-block partials in the
//   workspace, then one block) adds waste and optimal energy in a fixed order, so the
//   totals are deterministic.
//
// Exactness: SLO tests compare float32 table entries with float32 SLOs; the per-phase
// energies and the averages are float32 (P = fma(k*u*f^3, s, P0), E = P * duration); the
// EWR sums are float64 from float32 inputs.
#include <hip/hip_runtime.h>

#include <climits>
#include <cmath>
#include <cstddef>
#include <cstdint>

#include "festina.h"

namespace {

constexpr int kRows = FESTINA_N_ROWS;
constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kMaxCpl = FESTINA_MAX_CELLS / kWave;   // cells per lane
constexpr int kEwrBlock = 256;
constexpr float kInf = __builtin_huge_valf();

struct PrefArgs {
  int32_t M, NS, NF, C;
  const float *sm_level, *freq_level, *pf, *dc;
  float p0;
  int32_t G, K;
  const int32_t *n_inst, *model, *avg_in, *avg_out, *batch;
  const float *slo_ttft, *slo_tbt, *kdyn;
  festina_preferred out;
};

struct Best {
  float e, t, p;
  int cell;
};

// Least-energy feasible cell of one phase over the whole wavefront (lowest cell on ties).
template <int CPL>
__device__ Best phase_best(const PrefArgs &a, const float *row, float slo, float dur_scale, float ku) {
  const int lane = threadIdx.x & (kWave - 1);
  Best b{kInf, 0.f, 0.f, INT_MAX};
#pragma unroll
  for (int q = 0; q < CPL; ++q) {
    const int c = lane * CPL + q;
    if (c >= a.C) break;
    const float lat = row[c];
    if (!(lat < slo)) continue;
    const int j = c / a.NF, k = c - (c / a.NF) * a.NF;
    const float f = a.freq_level[k];
    const float P = fmaf(ku * (f * f * f), a.sm_level[j], a.p0);
    const float t = dur_scale * lat;
    const float e = P * t;
    if (!(e < kInf)) continue;
    if (e < b.e || (e == b.e && c < b.cell)) b = Best{e, t, P, c};
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float oe = __shfl_xor(b.e, off, kWave);
    const int oc = __shfl_xor(b.cell, off, kWave);
    const float ot = __shfl_xor(b.t, off, kWave);
    const float op = __shfl_xor(b.p, off, kWave);
    if (oe < b.e || (oe == b.e && oc < b.cell)) b = Best{oe, ot, op, oc};
  }
  return b;
}

template <int CPL>
__global__ void __launch_bounds__(kWavesPerBlock * kWave) k_preferred(PrefArgs a) {
  const long long slot = (long long)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  if (slot >= (long long)a.G * a.K) return;
  const int lane = threadIdx.x & (kWave - 1);
  const int g = (int)(slot / a.K), i = (int)(slot - (long long)g * a.K);
  const int n = a.n_inst[g];
  const int m = a.model[slot];
  const int B = a.batch[slot];
  const int tin = a.avg_in[slot], tout = a.avg_out[slot];
  const bool ok = n >= 0 && n <= a.K && i < n && m >= 0 && m < a.M && B >= 0 && tin >= 1 && tout >= 0;
  Best bp{kInf, 0.f, 0.f, INT_MAX}, bd{kInf, 0.f, 0.f, INT_MAX};
  if (ok) {
    const int bb = B + 1 > kRows ? kRows : B + 1;
    const int prow = min((int)(((unsigned)tin + 255u) >> 8), kRows) - 1;
    const float ku = a.kdyn[g] * ((float)bb * 0.03125f);
    const float *rp = a.pf + ((size_t)m * kRows + prow) * a.C;
    const float *rd = a.dc + ((size_t)m * kRows + (bb - 1)) * a.C;
    bp = phase_best<CPL>(a, rp, a.slo_ttft[slot], 1.f, ku);
    bd = phase_best<CPL>(a, rd, a.slo_tbt[slot], (float)tout, ku);
  }
  if (lane != 0) return;
  const bool hp = bp.cell != INT_MAX, hd = bd.cell != INT_MAX;
  const festina_preferred &o = a.out;
  o.sm_p[slot] = hp ? bp.cell / a.NF : -1;
  o.f_p[slot] = hp ? bp.cell % a.NF : -1;
  o.sm_d[slot] = hd ? bd.cell / a.NF : -1;
  o.f_d[slot] = hd ? bd.cell % a.NF : -1;
  o.t_p_ms[slot] = hp ? bp.t : 0.f;
  o.p_p_w[slot] = hp ? bp.p : 0.f;
  o.t_d_ms[slot] = hd ? bd.t : 0.f;
  o.p_d_w[slot] = hd ? bd.p : 0.f;
  o.t_ms[slot] = (hp ? bp.t : 0.f) + (hd ? bd.t : 0.f);
  o.feasible[slot] = (hp && hd) ? 1 : 0;
  float smp = __builtin_nanf(""), fpr = __builtin_nanf("");
  if (hp && hd) {
    const float sp = a.sm_level[bp.cell / a.NF], sd = a.sm_level[bd.cell / a.NF];
    const float fp = a.freq_level[bp.cell % a.NF], fd = a.freq_level[bd.cell % a.NF];
    smp = (sp * bp.t + sd * bd.t) / (bp.t + bd.t);
    const float ep = bp.p * bp.t, ed = bd.p * bd.t;
    fpr = (ep * fp + ed * fd) / (ep + ed);
  }
  o.sm_pref[slot] = smp;
  o.f_pref[slot] = fpr;
}

struct EwrArgs {
  int32_t G, K;
  const int32_t *n_inst;
  const float *f_pref, *t_ms;
  float *f_gpu;
  double *waste_gpu;
  double *totals;
  double *partial;               // [blocks][2] waste, optimal
};

__device__ __forceinline__ double cube64(double x) { return x * x * x; }

__device__ double block_sum(double v, double *s) {
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  __syncthreads();
  if (lane == 0) s[wv] = v;
  __syncthreads();
  double t = 0.0;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) t += s[w];
  return t;
}

// GPU g: F_g, its waste (written) and its optimal-energy share (returned in og).  With at
// most kEwrSlots slots per GPU every slot is loaded at once (one memory round trip) and
// masked by the instance count afterwards.
constexpr int kEwrSlots = 8;

__device__ __forceinline__ double ewr_one_gpu(const EwrArgs &a, int g, double &og) {
  const int n = a.n_inst[g];
  const int nn = (n >= 0 && n <= a.K) ? n : 0;
  const size_t base = (size_t)g * a.K;
  float fg = 0.f;
  double wg = 0.0;
  og = 0.0;
  if (a.K <= kEwrSlots) {
    float f[kEwrSlots], t[kEwrSlots];
#pragma unroll
    for (int i = 0; i < kEwrSlots; ++i) {
      f[i] = i < a.K ? a.f_pref[base + i] : 0.f;
      t[i] = i < a.K ? a.t_ms[base + i] : 0.f;
    }
#pragma unroll
    for (int i = 0; i < kEwrSlots; ++i)
      if (i < nn && isfinite(f[i]) && isfinite(t[i]) && f[i] > fg) fg = f[i];
    const double fg3 = cube64((double)fg);
#pragma unroll
    for (int i = 0; i < kEwrSlots; ++i)
      if (i < nn && isfinite(f[i]) && isfinite(t[i])) {
        const double fl3 = cube64((double)f[i]);
        wg += (double)t[i] * (fg3 - fl3);
        og += (double)t[i] * fl3;
      }
  } else {
    for (int i = 0; i < nn; ++i) {
      const float f = a.f_pref[base + i], t = a.t_ms[base + i];
      if (isfinite(f) && isfinite(t) && f > fg) fg = f;
    }
    const double fg3 = cube64((double)fg);
    for (int i = 0; i < nn; ++i) {
      const float f = a.f_pref[base + i], t = a.t_ms[base + i];
      if (!(isfinite(f) && isfinite(t))) continue;
      const double fl3 = cube64((double)f);
      wg += (double)t * (fg3 - fl3);
      og += (double)t * fl3;
    }
  }
  a.f_gpu[g] = fg;
  a.waste_gpu[g] = wg;
  return wg;
}

__global__ void __launch_bounds__(kEwrBlock) k_ewr_gpu(EwrArgs a) {
  __shared__ double s[kEwrBlock / kWave];
  const int g = blockIdx.x * kEwrBlock + threadIdx.x;
  double wg = 0.0, og = 0.0;
  if (g < a.G) wg = ewr_one_gpu(a, g, og);
  const double bw = block_sum(wg, s);
  const double bo = block_sum(og, s);
  if (threadIdx.x == 0) {
    a.partial[2 * blockIdx.x] = bw;
    a.partial[2 * blockIdx.x + 1] = bo;
  }
}

__global__ void __launch_bounds__(kEwrBlock) k_ewr_total(EwrArgs a, int32_t nblocks) {
  __shared__ double s[kEwrBlock / kWave];
  double w = 0.0, o = 0.0;
  for (int b = threadIdx.x; b < nblocks; b += kEwrBlock) {
    w += a.partial[2 * b];
    o += a.partial[2 * b + 1];
  }
  const double tw = block_sum(w, s);
  const double to = block_sum(o, s);
  if (threadIdx.x == 0) {
    a.totals[0] = tw;
    a.totals[1] = to;
    a.totals[2] = tw / to;
  }
}

// Fleets of at most kEwrSingle GPUs: one block of 1024 threads does everything in one
// launch (each thread a fixed stride of GPUs, then one block reduction: deterministic).
constexpr int kEwrSingleBlock = 1024;
constexpr int kEwrSingle = 16 * kEwrSingleBlock;

__global__ void __launch_bounds__(kEwrSingleBlock) k_ewr_single(EwrArgs a) {
  __shared__ double s[kEwrSingleBlock / kWave];
  double w = 0.0, o = 0.0;
  for (int g = threadIdx.x; g < a.G; g += kEwrSingleBlock) {
    double og;
    w += ewr_one_gpu(a, g, og);
    o += og;
  }
  const double tw = block_sum(w, s);
  const double to = block_sum(o, s);
  if (threadIdx.x == 0) {
    a.totals[0] = tw;
    a.totals[1] = to;
    a.totals[2] = tw / to;
  }
}

}  // namespace

extern "C" festina_status festina_preferred_configs(const festina_lut *L, const festina_llms *Q,
                                                    festina_preferred *out, void *stream) {
  if (!L || !Q || !out) return FESTINA_ERR_INVALID;
  if (L->n_models < 1 || L->n_rows != kRows || L->n_sm < 1 || L->n_freq < 1) return FESTINA_ERR_INVALID;
  if (Q->n_gpus < 0 || Q->max_inst < 1) return FESTINA_ERR_INVALID;
  const long long C = (long long)L->n_sm * L->n_freq;
  if (C > FESTINA_MAX_CELLS) return FESTINA_ERR_UNSUPPORTED;
  if (!L->sm_level || !L->freq_level || !L->pf || !L->dc) return FESTINA_ERR_INVALID;
  if (Q->n_gpus == 0) return FESTINA_OK;
  if (!Q->n_inst || !Q->model || !Q->avg_in_tokens || !Q->avg_out_tokens || !Q->batch || !Q->slo_ttft_ms ||
      !Q->slo_tbt_ms || !Q->k_dyn_w)
    return FESTINA_ERR_INVALID;
  if (!out->sm_p || !out->f_p || !out->sm_d || !out->f_d || !out->t_p_ms || !out->t_d_ms || !out->p_p_w ||
      !out->p_d_w || !out->t_ms || !out->sm_pref || !out->f_pref || !out->feasible)
    return FESTINA_ERR_INVALID;
  const long long slots = (long long)Q->n_gpus * Q->max_inst;
  const long long blocks = (slots + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks > INT_MAX) return FESTINA_ERR_INVALID;
  PrefArgs a;
  a.M = L->n_models;
  a.NS = L->n_sm;
  a.NF = L->n_freq;
  a.C = (int32_t)C;
  a.sm_level = L->sm_level;
  a.freq_level = L->freq_level;
  a.pf = L->pf;
  a.dc = L->dc;
  a.p0 = L->p0_w;
  a.G = Q->n_gpus;
  a.K = Q->max_inst;
  a.n_inst = Q->n_inst;
  a.model = Q->model;
  a.avg_in = Q->avg_in_tokens;
  a.avg_out = Q->avg_out_tokens;
  a.batch = Q->batch;
  a.slo_ttft = Q->slo_ttft_ms;
  a.slo_tbt = Q->slo_tbt_ms;
  a.kdyn = Q->k_dyn_w;
  a.out = *out;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const dim3 grid((unsigned)blocks), block(kWavesPerBlock * kWave);
  if (C <= kWave)
    k_preferred<1><<<grid, block, 0, st>>>(a);
  else if (C <= 2 * kWave)
    k_preferred<2><<<grid, block, 0, st>>>(a);
  else
    k_preferred<kMaxCpl><<<grid, block, 0, st>>>(a);
  return hipGetLastError() == hipSuccess ? FESTINA_OK : FESTINA_ERR_DEVICE;
}

extern "C" size_t festina_ewr_workspace_bytes(int32_t n_gpus) {
  if (n_gpus < 1) return 0;
  const size_t blocks = ((size_t)n_gpus + kEwrBlock - 1) / kEwrBlock;
  return (blocks * 2 * sizeof(double) + 255) & ~(size_t)255;
}

extern "C" festina_status festina_fleet_ewr(int32_t n_gpus, int32_t max_inst, const int32_t *n_inst,
                                            const float *f_pref, const float *t_ms, festina_ewr *out,
                                            void *workspace, size_t workspace_bytes, void *stream) {
  if (n_gpus < 1 || max_inst < 1 || !n_inst || !f_pref || !t_ms || !out) return FESTINA_ERR_INVALID;
  if (!out->f_gpu || !out->waste_gpu || !out->totals) return FESTINA_ERR_INVALID;
  const size_t need = festina_ewr_workspace_bytes(n_gpus);
  if (!workspace || workspace_bytes < need || (((uintptr_t)workspace) & 255) != 0) return FESTINA_ERR_INVALID;
  EwrArgs a;
  a.G = n_gpus;
  a.K = max_inst;
  a.n_inst = n_inst;
  a.f_pref = f_pref;
  a.t_ms = t_ms;
  a.f_gpu = out->f_gpu;
  a.waste_gpu = out->waste_gpu;
  a.totals = out->totals;
  a.partial = static_cast<double *>(workspace);
  const int blocks = (int)(((long long)n_gpus + kEwrBlock - 1) / kEwrBlock);
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (n_gpus <= kEwrSingle) {
    k_ewr_single<<<1, kEwrSingleBlock, 0, st>>>(a);
    return hipGetLastError() == hipSuccess ? FESTINA_OK : FESTINA_ERR_DEVICE;
  }
  k_ewr_gpu<<<blocks, kEwrBlock, 0, st>>>(a);
  if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  k_ewr_total<<<1, kEwrBlock, 0, st>>>(a, blocks);
  return hipGetLastError() == hipSuccess ? FESTINA_OK : FESTINA_ERR_DEVICE;
}
