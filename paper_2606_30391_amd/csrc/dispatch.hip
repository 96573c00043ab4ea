// dispatch.hip -- MI355X (gfx950) kernels and C-ABI host dispatch of the paper's own
// request dispatcher (Festina, Sec. 3.3 as the paper runs it): one operating point per GPU
// (its current frequency and the SMs free when the request's memory is available), the
// 2% stability tie-break, the F_max fallback ordered by availability, and a new GPU's
// least-energy level.
//
// k_dsp_hosts  one block per model: ascending list of the GPUs hosting it (wavefront
//                ballots), in the caller's workspace; with at most 4 profile steps, also a
//                64-byte record per (model, host) with everything Phase One reads, so that
//                the 16 lanes of a request load their hosts with coalesced 16-byte loads.
// k_dispatch   16 lanes per request (four per wavefront; 32 lanes in a launch of at most
//                8,192 requests, 64 in one of at most 2,048) stride over the model's hosts.  Per host:
//                the first free-memory profile step that holds Req_mem gives T_avail and
//                SM_free; the point (SM_free, F_curr) is feasible when T_avail + TTFT and
//                TBT meet the SLOs; E = P * (TTFT + Lout * TBT) in float64.  One pass
//                evaluates every host (a lane's first four hosts stay in registers) and
//                the group takes E_min; among hosts with E <= E_min + 0.02 |E_min| the largest
//                stability key (most memory, most SMs, lowest id packed in 64 bits) wins,
//                and the lane holding it writes the result.  With no
//                candidate: the hosts feasible at the top level, earliest T_avail (then
//                lowest id).  Else lane k scores a new GPU at level k and the least energy
//                (lowest k on ties) wins.
// Over arrival waves (festina_dispatch_waves): k_wave_init copies the caller's state into a
//                workspace buffer; one k_dispatch per wave reads the state with the previous
//                wave's commits applied, stores that state for the next wave, and commits its
//                own placements (batch, memory from the admitting step on, F_max boost) with
//                atomics; k_wave_final writes the last state back.
//
// Exactness: the energies are float64 in the same order of operations as any float64
// evaluation of P0 + k*s*f^3*u and P * (TTFT + Lout*TBT) without contraction, so the 2%
// test and every comparison are decided on identical values; the SLO tests add or compare
// float32 inputs exactly.
#include <hip/hip_runtime.h>

#include <climits>
#include <cstddef>
#include <cstdint>

#include "festina.h"

namespace {

constexpr int kRows = FESTINA_N_ROWS;
constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kHostBlock = 256;
constexpr int kMaxSteps = 8;                 // profile steps loaded at once
constexpr double kStability = 0.02;          // energies within 2% of the least tie

// Wave-by-wave calls keep two kinds of buffers in the workspace, each one allocation:
//   state   int32 [G][2] (current level, batch) then int32 [G][S] free MiB per profile step;
//   commits uint64 [G] (requests placed in the low 32 bits, bit 32 set by an F_max
//           placement) then uint64 [G][S] MiB taken per step (a request admitted at step s
//           counts at s and at every later step).
__device__ __forceinline__ int2 *state_fb(int32_t *st) { return reinterpret_cast<int2 *>(st); }
__device__ __forceinline__ int32_t *state_mem(int32_t *st, int G) { return st + 2 * (size_t)G; }
__device__ __forceinline__ unsigned long long *commit_taken(unsigned long long *c, int G) { return c + G; }

struct DspArgs {
  int32_t M, NS, NF, C, words;
  const float *sm_level, *freq_level, *pf, *dc;
  double p0;
  int32_t G, S;
  const int32_t *freq_cur, *batch;
  const float *kdyn;
  const uint32_t *resident;
  const float *t_avail;
  const int32_t *mem_free, *sm_free, *kv;
  double k_new;
  int32_t R;
  const int32_t *model, *prompt, *pred;
  const float *slo_ttft, *slo_tbt;
  int32_t *out_gpu, *out_freq, *out_sm;
  uint8_t *out_phase;
  float *out_energy;
  int32_t *host_cnt, *host_list;     // workspace: [M], [M][G]
  int4 *hrec;                        // workspace: [M][G][4] host records when S <= 4
  int32_t packed;
  int32_t r0;                        // first request of the launch (a.R: one past the last)
  // Wave-by-wave calls only (the kWaves kernels): the state this wave sees is `wstate` with
  // the previous wave's commits `wprev` applied (freq_cur, batch and mem_free are unused).
  // The launch also writes that state to `wfold` (the next wave's state), commits this
  // wave's placements to `wcur`, and clears `wnext` (the commits of the wave after).
  int32_t *wstate, *wfold;
  unsigned long long *wprev, *wcur, *wnext;
};

typedef int v4i __attribute__((ext_vector_type(4)));

// Energy on one operating point: P = p0 + k*s*f^3*u, E = P * (ttft + lout*tbt), each
// operation rounded separately (no fused multiply-add).
__device__ __forceinline__ double point_energy(double p0, double kg, double s, double f, double u, double ttft,
                                            double lout, double tbt) {
#pragma clang fp contract(off)
  const double f3 = f * f * f;
  const double P = p0 + kg * s * f3 * u;
  return P * (ttft + lout * tbt);
}

__global__ void __launch_bounds__(kHostBlock) k_dsp_hosts(DspArgs a) {
  const int m = blockIdx.x;
  __shared__ int wsum[kHostBlock / kWave];
  __shared__ int base_s;
  if (threadIdx.x == 0) base_s = 0;
  __syncthreads();
  const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x >> 6;
  for (int g0 = 0; g0 < a.G; g0 += kHostBlock) {
    const int g = g0 + threadIdx.x;
    const bool has = g < a.G && ((a.resident[(size_t)g * a.words + (m >> 5)] >> (m & 31)) & 1u);
    const unsigned long long bal = __ballot(has);
    const int before = __popcll(bal & ((1ull << lane) - 1ull));
    if (lane == 0) wsum[wv] = __popcll(bal);
    __syncthreads();
    int off = base_s;
    for (int i = 0; i < wv; ++i) off += wsum[i];
    if (has) {
      const size_t at = (size_t)m * a.G + off + before;
      a.host_list[at] = g;
      if (a.packed) {
        // one 64-byte record per (model, host): id, batch row + 1 (-1: no candidate),
        // current level, k; the profile's free memory, times and SM levels
        const int B = a.batch[g];
        int4 r0 = make_int4(g, B < 0 ? -1 : (B + 1 > kRows ? kRows : B + 1), a.freq_cur[g], __float_as_int(a.kdyn[g]));
        int mem[4] = {0, 0, 0, 0}, tt[4] = {0, 0, 0, 0}, sm[4] = {-1, -1, -1, -1};
        for (int s = 0; s < a.S; ++s) {
          mem[s] = a.mem_free[(size_t)g * a.S + s];
          tt[s] = __float_as_int(a.t_avail[(size_t)g * a.S + s]);
          sm[s] = a.sm_free[(size_t)g * a.S + s];
        }
        int4 *rec = a.hrec + at * 4;
        rec[0] = r0;
        rec[1] = make_int4(mem[0], mem[1], mem[2], mem[3]);
        rec[2] = make_int4(tt[0], tt[1], tt[2], tt[3]);
        rec[3] = make_int4(sm[0], sm[1], sm[2], sm[3]);
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int t = 0;
      for (int i = 0; i < kHostBlock / kWave; ++i) t += wsum[i];
      base_s += t;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) a.host_cnt[m] = base_s;
}

struct Point {
  int ok;                        // the host has a profile step holding the memory
  double ta;                     // T_avail
  int sm, mem, b;
};

// GPU g's state as the launch sees it: the stored one, and in a wave-by-wave call with
// the previous wave's commits applied (batch grown, level boosted, memory taken; a step
// left short of memory reads -1 MiB).
template <bool kWaves>
__device__ __forceinline__ int view_batch(const DspArgs &a, int g) {
  if (!kWaves) return a.batch[g];
  return state_fb(a.wstate)[g].y + (int)(uint32_t)a.wprev[g];
}
template <bool kWaves>
__device__ __forceinline__ int view_freq(const DspArgs &a, int g) {
  if (!kWaves) return a.freq_cur[g];
  return (a.wprev[g] >> 32) ? a.NF - 1 : state_fb(a.wstate)[g].x;
}
template <bool kWaves>
__device__ __forceinline__ int view_mem(const DspArgs &a, int g, int s) {
  if (!kWaves) return a.mem_free[(size_t)g * a.S + s];
  const long long v = (long long)state_mem(a.wstate, a.G)[(size_t)g * a.S + s] - (long long)commit_taken(a.wprev, a.G)[(size_t)g * a.S + s];
  return v < -1 ? -1 : (int)v;
}

// Phase One for host g: first profile step whose free memory holds `need` KiB.
template <bool kWaves>
__device__ __forceinline__ Point host_point(const DspArgs &a, int g, long long need) {
  Point p{0, 0.0, -1, 0, 1};
  const int B = view_batch<kWaves>(a, g);
  if (B < 0) return p;
  p.b = B + 1 > kRows ? kRows : B + 1;
  const size_t base = (size_t)g * a.S;
  if (a.S <= kMaxSteps) {
    int mem[kMaxSteps];
#pragma unroll
    for (int s = 0; s < kMaxSteps; ++s) mem[s] = s < a.S ? view_mem<kWaves>(a, g, s) : 0;
    int st = -1;
#pragma unroll
    for (int s = kMaxSteps - 1; s >= 0; --s)
      if (s < a.S && (long long)mem[s] * 1024 >= need) st = s;
    if (st < 0) return p;
    p.ok = 1;
    p.ta = (double)a.t_avail[base + st];
    p.sm = a.sm_free[base + st];
#pragma unroll
    for (int s = 0; s < kMaxSteps; ++s)
      if (s == st) p.mem = mem[s];
    return p;
  }
  for (int s = 0; s < a.S; ++s) {
    const int mem = view_mem<kWaves>(a, g, s);
    if ((long long)mem * 1024 >= need) {
      p.ok = 1;
      p.ta = (double)a.t_avail[base + s];
      p.sm = a.sm_free[base + s];
      p.mem = mem;
      return p;
    }
  }
  return p;
}

struct Host {
  int g, kcur;
  double kd;
  Point p;
};

// Phase One inputs of host number h of model m: from the packed record, or gathered.
template <bool kWaves>
__device__ __forceinline__ Host load_host(const DspArgs &a, int m, int h, const int *hl, long long need) {
  Host o;
  if (!kWaves && a.packed) {
    const v4i *rec = reinterpret_cast<const v4i *>(a.hrec + ((size_t)m * a.G + h) * 4);
    const v4i r0 = rec[0], mem = rec[1], tt = rec[2], sm = rec[3];
    __builtin_amdgcn_sched_barrier(0);   // the four loads in flight together, before any test
    o.g = r0.x;
    o.kcur = r0.z;
    o.kd = (double)__int_as_float(r0.w);
    o.p = Point{0, 0.0, -1, 0, r0.y};
    if (r0.y < 0) return o;
    int st = -1;
#pragma unroll
    for (int s = 3; s >= 0; --s)
      if (s < a.S && (long long)mem[s] * 1024 >= need) st = s;
    if (st < 0) return o;
    o.p.ok = 1;
    o.p.ta = (double)__int_as_float(st == 0 ? tt.x : st == 1 ? tt.y : st == 2 ? tt.z : tt.w);
    o.p.sm = st == 0 ? sm.x : st == 1 ? sm.y : st == 2 ? sm.z : sm.w;
    o.p.mem = st == 0 ? mem.x : st == 1 ? mem.y : st == 2 ? mem.z : mem.w;
    return o;
  }
  o.g = hl[h];
  o.kcur = view_freq<kWaves>(a, o.g);
  o.kd = (double)a.kdyn[o.g];
  o.p = host_point<kWaves>(a, o.g, need);
  return o;
}

// The SLO test and energy of one operating point from its gathered values: does the request
// (SLOs slo_ttft, slo_tbt) meet both starting at ta with batch b?  Energy if so.
__device__ __forceinline__ bool point_test(const DspArgs &a, float ttft, float tbt, float s, float f, int b, double ta,
                                           double kg, double lout, float slo_ttft, float slo_tbt, double &e) {
  if (!(ta + (double)ttft < (double)slo_ttft && tbt < slo_tbt)) return false;
  e = point_energy(a.p0, kg, (double)s, (double)f, (double)b / 32.0, (double)ttft, lout, (double)tbt);
  return (float)e < __builtin_huge_valf();
}

// Does the request meet its SLOs on (j, k) starting at ta with batch b?  Energy if so.
__device__ __forceinline__ bool point_ok(const DspArgs &a, int m, int prow, int b, int j, int k, double ta,
                                         double kg, double lout, float slo_ttft, float slo_tbt, double &e) {
  if (j < 0 || j >= a.NS || k < 0 || k >= a.NF) return false;
  const size_t cell = (size_t)j * a.NF + k;
  const float ttft = a.pf[((size_t)m * kRows + (prow >= 0 ? prow : b - 1)) * a.C + cell];
  const float tbt = a.dc[((size_t)m * kRows + (b - 1)) * a.C + cell];
  return point_test(a, ttft, tbt, a.sm_level[j], a.freq_level[k], b, ta, kg, lout, slo_ttft, slo_tbt, e);
}

// Stability order as one integer: more free memory, then more free SMs, then a lower GPU id
// is a larger key (memory biased to unsigned; SM level < 256; id < 2^24); 0 = no candidate.
__device__ __forceinline__ unsigned long long stability_key(int mem, int sm, int g) {
  return ((unsigned long long)((unsigned)mem ^ 0x80000000u) << 32) | ((unsigned long long)(sm & 0xff) << 24) |
         (unsigned long long)(0xffffffu - (unsigned)g);
}

// Lanes per request: 16 (four requests per wavefront) when a launch holds enough requests
// to fill the GPU, else 32 or 64, so that a request's hosts take fewer rounds of loads.
constexpr int kWideRequests = 2048;              // at most this many requests: 64 lanes each
constexpr int kMidRequests = 8192;               // at most this many: 32 lanes each
constexpr int kCached = 4;                       // hosts per lane whose Phase One result stays in registers

template <int kGroup>
__device__ __forceinline__ unsigned long long shfl_xor_u64(unsigned long long v, int off) {
  const unsigned lo = __shfl_xor((unsigned)v, off, kGroup), hi = __shfl_xor((unsigned)(v >> 32), off, kGroup);
  return ((unsigned long long)hi << 32) | lo;
}

// kGroup lanes per request (64 / kGroup requests per wavefront); lane s of a request strides
// over its model's hosts (s, s + kGroup, ...), all reductions stay inside the group.
template <int kGroup, bool kWaves>
__global__ void __launch_bounds__(kWavesPerBlock * kWave) k_dispatch(DspArgs a) {
#pragma clang fp contract(off)
  constexpr int kReqPerWave = kWave / kGroup;
  if (kWaves) {
    // the state this wave sees, stored for the next wave; the commits after that cleared
    for (int g = blockIdx.x * blockDim.x + threadIdx.x; g < a.G; g += gridDim.x * blockDim.x) {
      state_fb(a.wfold)[g] = make_int2(view_freq<true>(a, g), view_batch<true>(a, g));
      a.wnext[g] = 0ull;
      for (int s = 0; s < a.S; ++s) {
        const size_t at = (size_t)g * a.S + s;
        state_mem(a.wfold, a.G)[at] = view_mem<true>(a, g, s);
        commit_taken(a.wnext, a.G)[at] = 0ull;
      }
    }
  }
  const int lane = threadIdx.x & (kWave - 1);
  const int sub = lane & (kGroup - 1);
  const int r = a.r0 + (blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6)) * kReqPerWave + lane / kGroup;
  if (r >= a.R) return;
  const double inf = __builtin_huge_val();
  const int m = a.model[r];
  const int pt = a.prompt[r], pd = a.pred[r];
  const float slo_ttft = a.slo_ttft[r], slo_tbt = a.slo_tbt[r];
  int gsel = -1, ksel = -1, jsel = -1, phase = 0;
  double esel = inf;
  bool writer = sub == 0;
  long long need = 0;
  if (m >= 0 && m < a.M && pd >= 0 && pt >= 0) {
    const int prow = pt == 0 ? -1 : (min((int)(((unsigned)pt + 255u) >> 8), kRows) - 1);
    const long long lout_i = ((long long)pd * 105 + 99) / 100;
    const double lout = (double)lout_i;
    need = (long long)a.kv[m] * ((long long)pt + lout_i);
    const int nh = a.host_cnt[m];
    const int *hl = a.host_list + (size_t)m * a.G;
    // Phase One at every host, least energy; the first kCached hosts of a lane are kept
    double emin = inf;
    double ec[kCached];
    unsigned long long kc[kCached];
#pragma unroll
    for (int i = 0; i < kCached; ++i) {
      ec[i] = inf;
      kc[i] = 0ull;
    }
    for (int i = 0, h = sub; h < nh; ++i, h += kGroup) {
      const Host H = load_host<kWaves>(a, m, h, hl, need);
      const int g = H.g;
      const Point &p = H.p;
      double e;
      if (!(p.ok && point_ok(a, m, prow, p.b, p.sm, H.kcur, p.ta, H.kd, lout, slo_ttft, slo_tbt, e))) continue;
      emin = fmin(emin, e);
#pragma unroll
      for (int c = 0; c < kCached; ++c)
        if (i == c) {
          ec[c] = e;
          kc[c] = stability_key(p.mem, p.sm, g);
        }
    }
    for (int off = kGroup / 2; off >= 1; off >>= 1) emin = fmin(emin, __shfl_xor(emin, off, kGroup));
    if (emin < inf) {
      // Phase Two: the largest stability key among the hosts within 2% of the least energy
      const double bound = emin + kStability * fabs(emin);
      unsigned long long best = 0ull;
      double ebest = inf;
#pragma unroll
      for (int c = 0; c < kCached; ++c)
        if (kc[c] > best && ec[c] <= bound) {
          best = kc[c];
          ebest = ec[c];
        }
      for (int h = sub + kCached * kGroup; h < nh; h += kGroup) {   // hosts past the cached ones
        const Host H = load_host<kWaves>(a, m, h, hl, need);
        const int g = H.g;
        const Point &p = H.p;
        double e;
        if (!(p.ok && point_ok(a, m, prow, p.b, p.sm, H.kcur, p.ta, H.kd, lout, slo_ttft, slo_tbt, e))) continue;
        const unsigned long long key = stability_key(p.mem, p.sm, g);
        if (e <= bound && key > best) {
          best = key;
          ebest = e;
        }
      }
      unsigned long long wbest = best;
      for (int off = kGroup / 2; off >= 1; off >>= 1) {
        const unsigned long long o = shfl_xor_u64<kGroup>(wbest, off);
        wbest = o > wbest ? o : wbest;
      }
      if (wbest != 0ull) {                 // the least-energy host is always within the bound
        writer = best == wbest;            // exactly one lane of the group holds the winning key
        gsel = (int)(0xffffffu - (unsigned)(wbest & 0xffffffull));
        jsel = (int)((wbest >> 24) & 0xffull);
        ksel = view_freq<kWaves>(a, gsel);   // the winner's current level
        phase = 1;
        esel = ebest;
      }
    } else {
      // Phase Three: the earliest available host that meets the SLOs at the top level
      const int kmax = a.NF - 1;
      int bg = INT_MAX, bsm = -1;
      double bt = inf, be = inf;
      for (int h = sub; h < nh; h += kGroup) {
        const Host H = load_host<kWaves>(a, m, h, hl, need);
        const int g = H.g;
        const Point &p = H.p;
        double e;
        if (!(p.ok && point_ok(a, m, prow, p.b, p.sm, kmax, p.ta, H.kd, lout, slo_ttft, slo_tbt, e))) continue;
        if (p.ta < bt || (p.ta == bt && g < bg)) {
          bg = g;
          bt = p.ta;
          bsm = p.sm;
          be = e;
        }
      }
      for (int off = kGroup / 2; off >= 1; off >>= 1) {
        const int og = __shfl_xor(bg, off, kGroup), os = __shfl_xor(bsm, off, kGroup);
        const double ot = __shfl_xor(bt, off, kGroup), oe = __shfl_xor(be, off, kGroup);
        if (ot < bt || (ot == bt && og < bg)) {
          bg = og;
          bt = ot;
          bsm = os;
          be = oe;
        }
      }
      if (bg != INT_MAX) {
        gsel = bg;
        ksel = kmax;
        jsel = bsm;
        phase = 2;
        esel = be;
      } else {
        // scale out: a new GPU (batch 1, every SM, available now), lane s scores levels s, s + 16, ...
        int bk = INT_MAX;
        double bke = inf;
        for (int k = sub; k < a.NF; k += kGroup) {
          double e;
          if (point_ok(a, m, prow, 1, a.NS - 1, k, 0.0, a.k_new, lout, slo_ttft, slo_tbt, e) && (e < bke || (e == bke && k < bk))) {
            bke = e;
            bk = k;
          }
        }
        for (int off = kGroup / 2; off >= 1; off >>= 1) {
          const int ok = __shfl_xor(bk, off, kGroup);
          const double oe = __shfl_xor(bke, off, kGroup);
          if (oe < bke || (oe == bke && ok < bk)) {
            bke = oe;
            bk = ok;
          }
        }
        if (bk != INT_MAX) {
          ksel = bk;
          jsel = a.NS - 1;
          phase = 3;
          esel = bke;
        }
      }
    }
  }
  if (writer) {
    a.out_gpu[r] = gsel;
    a.out_freq[r] = ksel;
    a.out_sm[r] = jsel;
    a.out_phase[r] = (uint8_t)phase;
    a.out_energy[r] = (float)esel;
    if (kWaves && (phase == 1 || phase == 2)) {
      // commit to the chosen GPU: one more request in its batch, and ceil(Req_mem / 1024)
      // MiB from the step that admitted it (the first whose free memory holds Req_mem) on
      const size_t base = (size_t)gsel * a.S;
      int st = 0;
      while (st < a.S - 1 && (long long)view_mem<true>(a, gsel, st) * 1024 < need) ++st;
      const unsigned long long q = (unsigned long long)((need + 1023) / 1024);
      atomicAdd(&a.wcur[gsel], phase == 2 ? (1ull << 32) | 1ull : 1ull);
      for (int s = st; s < a.S; ++s) atomicAdd(&commit_taken(a.wcur, a.G)[base + s], q);
    }
  }
}

// Start of a wave-by-wave call: the caller's state copied into the first state buffer, the
// three commit buffers cleared.
__global__ void __launch_bounds__(kHostBlock) k_wave_init(int32_t G, int32_t S, int32_t *st0, unsigned long long *c0,
                                                          unsigned long long *c1, unsigned long long *c2,
                                                          const int32_t *freq0, const int32_t *batch0,
                                                          const int32_t *mem0) {
  const int g = blockIdx.x * kHostBlock + threadIdx.x;
  if (g >= G) return;
  state_fb(st0)[g] = make_int2(freq0[g], batch0[g]);
  c0[g] = c1[g] = c2[g] = 0ull;
  for (int s = 0; s < S; ++s) {
    const size_t at = (size_t)g * S + s;
    state_mem(st0, G)[at] = mem0[at];
    commit_taken(c0, G)[at] = commit_taken(c1, G)[at] = commit_taken(c2, G)[at] = 0ull;
  }
}

// End of a wave-by-wave call: the last state with the last wave's commits applied, into
// the caller's arrays.
__global__ void __launch_bounds__(kHostBlock) k_wave_final(DspArgs a, int32_t *freq, int32_t *batch, int32_t *mem) {
  const int g = blockIdx.x * kHostBlock + threadIdx.x;
  if (g >= a.G) return;
  batch[g] = view_batch<true>(a, g);
  freq[g] = view_freq<true>(a, g);
  for (int s = 0; s < a.S; ++s) mem[(size_t)g * a.S + s] = view_mem<true>(a, g, s);
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

bool dsp_shapes_ok(const festina_lut *L, const festina_gpu_avail *A) {
  if (!L || !A) return false;
  if (L->n_models < 1 || L->n_rows != kRows || L->n_sm < 1 || L->n_freq < 1) return false;
  if (A->n_gpus < 1 || A->n_steps < 1) return false;
  if ((long long)L->n_models * A->n_gpus > INT_MAX) return false;
  if (A->n_gpus > 0xffffff) return false;       // GPU ids are packed in 24 bits
  return true;
}

}  // namespace

extern "C" size_t festina_dispatch_workspace_bytes(const festina_lut *L, const festina_gpu_avail *A) {
  if (!dsp_shapes_ok(L, A)) return 0;
  size_t bytes = align256(sizeof(int32_t) * L->n_models) + align256(sizeof(int32_t) * (size_t)L->n_models * A->n_gpus);
  if (A->n_steps <= 4) bytes += align256((size_t)64 * L->n_models * A->n_gpus);     // host records
  return bytes;
}

// k_dispatch over requests lo .. hi-1, with the group width their number calls for.
template <bool kWaves>
static festina_status launch_dispatch(DspArgs a, int32_t lo, int32_t hi, hipStream_t st) {
  a.r0 = lo;
  a.R = hi;
  const long long n = (long long)hi - lo;
  if (n <= kWideRequests) {
    const long long per_block = (long long)kWavesPerBlock * (kWave / 64);
    k_dispatch<64, kWaves><<<(unsigned)((n + per_block - 1) / per_block), kWavesPerBlock * kWave, 0, st>>>(a);
  } else if (n <= kMidRequests) {
    const long long per_block = (long long)kWavesPerBlock * (kWave / 32);
    k_dispatch<32, kWaves><<<(unsigned)((n + per_block - 1) / per_block), kWavesPerBlock * kWave, 0, st>>>(a);
  } else {
    const long long per_block = (long long)kWavesPerBlock * (kWave / 16);
    k_dispatch<16, kWaves><<<(unsigned)((n + per_block - 1) / per_block), kWavesPerBlock * kWave, 0, st>>>(a);
  }
  return hipGetLastError() == hipSuccess ? FESTINA_OK : FESTINA_ERR_DEVICE;
}

// Checks the arguments common to both dispatch calls; fills everything but the workspace.
static festina_status dsp_args(const festina_lut *L, const festina_gpu_avail *A, const festina_requests *Q,
                               festina_dispatches *out, DspArgs &a) {
  if (!dsp_shapes_ok(L, A) || !Q || !out || Q->n_requests < 0) return FESTINA_ERR_INVALID;
  const long long C = (long long)L->n_sm * L->n_freq;
  if (C > FESTINA_MAX_CELLS) return FESTINA_ERR_UNSUPPORTED;
  if (!L->sm_level || !L->freq_level || !L->pf || !L->dc) return FESTINA_ERR_INVALID;
  if (!A->freq_cur || !A->batch || !A->k_dyn_w || !A->resident || !A->t_avail_ms || !A->mem_free_mib ||
      !A->sm_free || !A->kv_kib_per_token)
    return FESTINA_ERR_INVALID;
  if (Q->n_requests > 0) {
    if (!Q->model || !Q->prompt_tokens || !Q->pred_out_tokens || !Q->slo_ttft_ms || !Q->slo_tbt_ms)
      return FESTINA_ERR_INVALID;
    if (!out->gpu || !out->freq_level || !out->sm_level || !out->phase || !out->energy_mj) return FESTINA_ERR_INVALID;
  }
  a.M = L->n_models;
  a.NS = L->n_sm;
  a.NF = L->n_freq;
  a.C = (int32_t)C;
  a.words = (L->n_models + 31) / 32;
  a.sm_level = L->sm_level;
  a.freq_level = L->freq_level;
  a.pf = L->pf;
  a.dc = L->dc;
  a.p0 = (double)L->p0_w;
  a.G = A->n_gpus;
  a.S = A->n_steps;
  a.freq_cur = A->freq_cur;
  a.batch = A->batch;
  a.kdyn = A->k_dyn_w;
  a.resident = A->resident;
  a.t_avail = A->t_avail_ms;
  a.mem_free = A->mem_free_mib;
  a.sm_free = A->sm_free;
  a.kv = A->kv_kib_per_token;
  a.k_new = (double)A->k_new_w;
  a.R = Q->n_requests;
  a.model = Q->model;
  a.prompt = Q->prompt_tokens;
  a.pred = Q->pred_out_tokens;
  a.slo_ttft = Q->slo_ttft_ms;
  a.slo_tbt = Q->slo_tbt_ms;
  a.out_gpu = out->gpu;
  a.out_freq = out->freq_level;
  a.out_sm = out->sm_level;
  a.out_phase = out->phase;
  a.out_energy = out->energy_mj;
  a.r0 = 0;
  a.wstate = a.wfold = nullptr;
  a.wprev = a.wcur = a.wnext = nullptr;
  a.packed = 0;
  a.hrec = nullptr;
  return FESTINA_OK;
}

extern "C" festina_status festina_dispatch_requests(const festina_lut *L, const festina_gpu_avail *A,
                                                    const festina_requests *Q, festina_dispatches *out,
                                                    void *workspace, size_t workspace_bytes, void *stream) {
  DspArgs a;
  const festina_status chk = dsp_args(L, A, Q, out, a);
  if (chk != FESTINA_OK) return chk;
  const size_t need = festina_dispatch_workspace_bytes(L, A);
  if (!workspace || workspace_bytes < need || (((uintptr_t)workspace) & 255) != 0) return FESTINA_ERR_INVALID;
  if (Q->n_requests == 0) return FESTINA_OK;
  char *ws = static_cast<char *>(workspace);
  a.host_cnt = reinterpret_cast<int32_t *>(ws);
  a.host_list = reinterpret_cast<int32_t *>(ws + align256(sizeof(int32_t) * L->n_models));
  a.packed = A->n_steps <= 4 ? 1 : 0;
  a.hrec = reinterpret_cast<int4 *>(ws + align256(sizeof(int32_t) * L->n_models) +
                                    align256(sizeof(int32_t) * (size_t)L->n_models * A->n_gpus));
  hipStream_t st = static_cast<hipStream_t>(stream);
  k_dsp_hosts<<<a.M, kHostBlock, 0, st>>>(a);
  if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  return launch_dispatch<false>(a, 0, a.R, st);
}

// Workspace of a wave-by-wave call: host counts and lists, two state buffers (the state
// each wave sees alternates between them) and three commit buffers (the previous wave's,
// read; the current wave's, written; the next wave's, cleared).
static size_t state_bytes(size_t G, size_t S) { return align256(sizeof(int32_t) * (2 * G + G * S)); }
static size_t commit_bytes(size_t G, size_t S) { return align256(sizeof(unsigned long long) * (G + G * S)); }

extern "C" size_t festina_dispatch_waves_workspace_bytes(const festina_lut *L, const festina_gpu_avail *A) {
  if (!dsp_shapes_ok(L, A)) return 0;
  const size_t G = (size_t)A->n_gpus, S = (size_t)A->n_steps;
  return align256(sizeof(int32_t) * L->n_models) + align256(sizeof(int32_t) * (size_t)L->n_models * G) +
         2 * state_bytes(G, S) + 3 * commit_bytes(G, S);
}

extern "C" festina_status festina_dispatch_waves(const festina_lut *L, const festina_gpu_avail *A,
                                                 const festina_requests *Q, int32_t n_waves,
                                                 const int32_t *wave_start, festina_gpu_state *state,
                                                 festina_dispatches *out, void *workspace, size_t workspace_bytes,
                                                 void *stream) {
  DspArgs a;
  const festina_status chk = dsp_args(L, A, Q, out, a);
  if (chk != FESTINA_OK) return chk;
  if (!state || !state->freq_cur || !state->batch || !state->mem_free_mib || n_waves < 0) return FESTINA_ERR_INVALID;
  if (n_waves == 0) {
    if (Q->n_requests != 0) return FESTINA_ERR_INVALID;
  } else {
    if (!wave_start || wave_start[0] != 0 || wave_start[n_waves] != Q->n_requests) return FESTINA_ERR_INVALID;
    for (int32_t w = 0; w < n_waves; ++w)
      if (wave_start[w + 1] < wave_start[w]) return FESTINA_ERR_INVALID;
  }
  const size_t need = festina_dispatch_waves_workspace_bytes(L, A);
  if (!workspace || workspace_bytes < need || (((uintptr_t)workspace) & 255) != 0) return FESTINA_ERR_INVALID;
  const size_t G = (size_t)A->n_gpus, S = (size_t)A->n_steps;
  char *ws = static_cast<char *>(workspace);
  size_t at = 0;
  auto take = [&](size_t bytes) {
    char *p = ws + at;
    at += align256(bytes);
    return p;
  };
  a.host_cnt = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * L->n_models));
  a.host_list = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * (size_t)L->n_models * G));
  int32_t *sb[2];
  for (int32_t *&x : sb) x = reinterpret_cast<int32_t *>(take(sizeof(int32_t) * (2 * G + G * S)));
  unsigned long long *db[3];
  for (unsigned long long *&x : db) x = reinterpret_cast<unsigned long long *>(take(sizeof(unsigned long long) * (G + G * S)));
  hipStream_t st = static_cast<hipStream_t>(stream);
  const unsigned gblocks = (unsigned)((G + kHostBlock - 1) / kHostBlock);
  k_wave_init<<<gblocks, kHostBlock, 0, st>>>(A->n_gpus, A->n_steps, sb[0], db[0], db[1], db[2], A->freq_cur,
                                              A->batch, A->mem_free_mib);
  if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  if (Q->n_requests > 0) {
    k_dsp_hosts<<<a.M, kHostBlock, 0, st>>>(a);
    if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  }
  // Launch v (of the non-empty waves) sees sb[v % 2] with db[(v + 2) % 3] applied, stores
  // that in sb[(v + 1) % 2], commits to db[v % 3] and clears db[(v + 1) % 3].
  a.freq_cur = a.batch = a.mem_free = nullptr;
  int v = 0;
  for (int32_t w = 0; w < n_waves; ++w) {
    const int32_t lo = wave_start[w], hi = wave_start[w + 1];
    if (hi == lo) continue;
    a.wstate = sb[v % 2];
    a.wfold = sb[(v + 1) % 2];
    a.wprev = db[(v + 2) % 3];
    a.wcur = db[v % 3];
    a.wnext = db[(v + 1) % 3];
    if (launch_dispatch<true>(a, lo, hi, st) != FESTINA_OK) return FESTINA_ERR_DEVICE;
    ++v;
  }
  a.wstate = sb[v % 2];
  a.wprev = db[(v + 2) % 3];
  k_wave_final<<<gblocks, kHostBlock, 0, st>>>(a, state->freq_cur, state->batch, state->mem_free_mib);
  return hipGetLastError() == hipSuccess ? FESTINA_OK : FESTINA_ERR_DEVICE;
}
