// sweep.hip -- MI355X (gfx950) kernel and C-ABI host dispatch of the local scheduler's
// joint SM/frequency sweep (Festina, Sec. 3.4, runtime resource allocation), batched
// over many GPUs' task batches in one launch.
//
// For a batch of tasks (prefill units and decode steps) and each frequency level k, every
// task takes the smallest SM level whose profiled latency is strictly below its slack;
// level k is usable when every task has such a level and their integer SM shares sum to
// strictly less than the device budget; the batch energy at k is the sum over tasks of
// (P0 + k_dyn * s_j * f_k^3 * u) * latency (static power per task), or P0 times the
// longest task's latency plus the sum over tasks of k_dyn * s_j * f_k^3 * u * latency
// (static power per batch).  The least-energy usable level wins, the lowest k on exact
// ties.
//
// Layout of the work: one wavefront per batch.  The batch's slot fields arrive in one
// memory round trip (lane t loads slot t) and go to LDS as a table offset, phase and slack
// per task.  Lane l then serves frequency level k = l mod NFp (NFp = NF rounded up to a
// power of two) for the tasks of slot group l / NFp (tasks g, g + groups, ...), so every
// lane works for NF = 16 (four groups of 16 levels).  Two tasks at a time, a lane issues
// the latencies at the first 8 SM levels of both (16 loads in flight, 64-byte segments per
// group), keeps the first one below each slack, and accumulates SM shares and energy;
// xor-shuffles add the groups' partial sums, and a wavefront (energy, level) minimum picks
// the level.  The lanes of the chosen level write their first two tasks' SM levels from
// registers and repeat the search (bit-identical) for any further task.  Tables are read
// through L2 (a batch touches a few KB of them); nothing else is staged.
//
// Exactness: the SM-level choice compares a float32 table entry with a float32 slack and
// the budget test adds integers, so both are decided exactly.  Energies are float32:
// P = fma(k_dyn * u * f^3, s_j, P0), E = sum of fma(P, latency, E) per task; per batch
// E = fma(P0, longest latency, sum of fma(k_dyn * u * f^3 * s_j, latency, E)).
#include <hip/hip_runtime.h>

#include <climits>
#include <cstddef>
#include <cstdint>

#include "festina.h"

namespace {

constexpr int kRows = FESTINA_N_ROWS;
constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kMaxSm = FESTINA_MAX_CELLS;   // SM levels staged in LDS
constexpr int kJChunk = 8;                  // table loads in flight per lane
constexpr float kInf = __builtin_huge_valf();

struct SweepArgs {
  int32_t M, NS, NF;
  const float *sm_level, *freq_level, *pf, *dc;
  int32_t B, T;
  const int32_t *n_tasks, *model, *phase, *tokens;
  const float *slack, *kdyn, *util;
  const int32_t *units;
  int32_t budget;
  float p0_task;                 // P0 in each task's power (static power per task), else 0
  float p0_batch;                // P0 over the longest task (static power per batch), else 0
  int32_t lg;                    // log2 of the lanes per slot group (NF <= 1 << lg)
  int32_t *level;
  uint8_t *feasible;
  float *energy;
  int32_t *task_sm;
};

// Table row of a task (prefill: 256-token prompt bucket; decode: batch size - 1), or -1
// for an invalid task (model out of range, no tokens, unknown phase).
__device__ __forceinline__ int task_row(const SweepArgs &a, int m, int ph, int tok) {
  if (m < 0 || m >= a.M || tok < 1) return -1;
  if (ph == 0) return min((int)(((unsigned)tok + 255u) >> 8), kRows) - 1;
  if (ph == 1) return min(tok, kRows) - 1;
  return -1;
}

// A fresh copy of a wave-uniform value: what is computed from it (the column strides and
// level tests of a chunk) is computed where it is used instead of being kept, one scalar
// register pair per level, across the whole task loop.
__device__ __forceinline__ int fresh_s(int v) {
  asm volatile("" : "+s"(v));
  return v;
}

// Smallest SM level j with latency[j][k] < slack for the task whose (model, row) table
// column starts at `col`; -1 if none.  `lat` receives that latency.
__device__ __forceinline__ int min_sm_level(const SweepArgs &a, const float *col, float slack, float &lat) {
  int jj = -1;
  lat = 0.f;
  for (int j0 = 0; j0 < a.NS && jj < 0; j0 += kJChunk) {
    const int ns = fresh_s(a.NS), nf = fresh_s(a.NF);
    float v[kJChunk];
#pragma unroll
    for (int q = 0; q < kJChunk; ++q)
      v[q] = j0 + q < ns ? col[(size_t)(j0 + q) * nf] : __builtin_nanf("");
#pragma unroll
    for (int q = kJChunk - 1; q >= 0; --q)
      if (v[q] < slack) {
        jj = j0 + q;
        lat = v[q];
      }
  }
  return jj;
}

// First table chunk of a task column: kJChunk loads issued together (NaN past NS and for
// lanes without work), then the smallest level below the slack; -1 if none in the chunk.
__device__ __forceinline__ void load_chunk(const SweepArgs &a, const float *col, bool on, float (&v)[kJChunk]) {
  const int ns = fresh_s(a.NS), nf = fresh_s(a.NF);
#pragma unroll
  for (int q = 0; q < kJChunk; ++q)
    v[q] = (on && q < ns) ? col[(size_t)q * nf] : __builtin_nanf("");
}

__device__ __forceinline__ int first_below(const float (&v)[kJChunk], float slack, float &lat) {
  int jj = -1;
  lat = 0.f;
#pragma unroll
  for (int q = kJChunk - 1; q >= 0; --q)
    if (v[q] < slack) {
      jj = q;
      lat = v[q];
    }
  return jj;
}

// Smallest level from kJChunk on (tables with more than kJChunk SM levels).
__device__ int min_sm_level_from_chunk(const SweepArgs &a, const float *col, float slack, float &lat) {
  int jj = -1;
  lat = 0.f;
  for (int j0 = kJChunk; j0 < a.NS && jj < 0; j0 += kJChunk) {
    const int ns = fresh_s(a.NS), nf = fresh_s(a.NF);
    float v[kJChunk];
#pragma unroll
    for (int q = 0; q < kJChunk; ++q)
      v[q] = j0 + q < ns ? col[(size_t)(j0 + q) * nf] : __builtin_nanf("");
#pragma unroll
    for (int q = kJChunk - 1; q >= 0; --q)
      if (v[q] < slack) {
        jj = j0 + q;
        lat = v[q];
      }
  }
  return jj;
}

__global__ void __launch_bounds__(kWavesPerBlock * kWave) k_sweep(SweepArgs a) {
  __shared__ float s_lev[kMaxSm];
  __shared__ int s_units[kMaxSm];
  __shared__ long long s_col[kWavesPerBlock][kWave];   // table offset of each task's (model, row)
  __shared__ float s_slack[kWavesPerBlock][kWave];
  __shared__ int s_ph[kWavesPerBlock][kWave];
  for (int j = threadIdx.x; j < a.NS; j += blockDim.x) {
    s_lev[j] = a.sm_level[j];
    s_units[j] = a.units[j];
  }
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int b = blockIdx.x * kWavesPerBlock + wv;
  const bool live = b < a.B;
  const int lane = threadIdx.x & (kWave - 1);
  const size_t row0 = (size_t)(live ? b : 0) * a.T;

  // one memory round trip for the batch: its size, GPU terms, and every slot's task fields
  // (all max_tasks slots are read, independently of the task count)
  const bool slot = live && lane < a.T;
  int m = 0, ph = 0, tok = 0;
  float sl = 0.f;
  if (slot) {
    m = a.model[row0 + lane];
    ph = a.phase[row0 + lane];
    tok = a.tokens[row0 + lane];
    sl = a.slack[row0 + lane];
  }
  const int n = live ? a.n_tasks[b] : 0;
  const float kd = live ? a.kdyn[b] : 0.f, u = live ? a.util[b] : 0.f;
  const bool n_ok = n >= 0 && n <= a.T;
  const int nn = n_ok ? n : 0;
  int row = 0;
  if (lane < nn) {
    row = task_row(a, m, ph, tok);
    s_col[wv][lane] = row >= 0 ? ((long long)m * kRows + row) * a.NS * a.NF : 0;
    s_slack[wv][lane] = sl;
    s_ph[wv][lane] = ph;
  }
  __syncthreads();
  if (!live) return;
  const bool bad = !n_ok || __any(lane < nn && row < 0);   // an invalid task voids the batch

  const int nfp = 1 << a.lg;
  const int k = lane & (nfp - 1);
  const int grp = lane >> a.lg;
  const int ngrp = kWave >> a.lg;
  const bool kv = k < a.NF;
  const float f = kv ? a.freq_level[k] : 1.f;
  const float c = kd * u * (f * f * f);
  long long units = 0;
  float E = 0.f, lmax = 0.f;     // energy, the longest task's latency
  int miss = 0;                  // some task has no SM level meeting its slack at k
  int jk0 = -1, jk1 = -1;        // SM levels of the lane's first two tasks
  // two tasks per step: 2 * kJChunk table loads in flight per lane
  for (int t0 = grp; !bad && t0 < nn; t0 += 2 * ngrp) {
    const int t1 = t0 + ngrp;
    const bool on0 = kv, on1 = kv && t1 < nn;
    const int t1c = on1 ? t1 : t0;             // a slot index inside the batch either way
    const float *col0 = (s_ph[wv][t0] == 0 ? a.pf : a.dc) + s_col[wv][t0] + k;
    const float *col1 = (s_ph[wv][t1c] == 0 ? a.pf : a.dc) + s_col[wv][t1c] + k;
    float v0[kJChunk], v1[kJChunk];
    load_chunk(a, col0, on0, v0);
    load_chunk(a, col1, on1, v1);
    if (!kv) continue;
    const float sl0 = s_slack[wv][t0];
    float lat0;
    int j0 = first_below(v0, sl0, lat0);
    if (j0 < 0 && a.NS > kJChunk) j0 = min_sm_level_from_chunk(a, col0, sl0, lat0);
    if (j0 < 0) {
      miss = 1;
    } else {
      units += s_units[j0];
      E = fmaf(fmaf(c, s_lev[j0], a.p0_task), lat0, E);
      lmax = fmaxf(lmax, lat0);
    }
    int j1 = -1;
    if (on1) {
      const float sl1 = s_slack[wv][t1];
      float lat1;
      j1 = first_below(v1, sl1, lat1);
      if (j1 < 0 && a.NS > kJChunk) j1 = min_sm_level_from_chunk(a, col1, sl1, lat1);
      if (j1 < 0) {
        miss = 1;
      } else {
        units += s_units[j1];
        E = fmaf(fmaf(c, s_lev[j1], a.p0_task), lat1, E);
        lmax = fmaxf(lmax, lat1);
      }
    }
    if (t0 == grp) {
      jk0 = j0;
      jk1 = j1;
    }
  }
  // add the slot groups' partial results (lanes of one level k across groups)
  for (int off = nfp; off < kWave; off <<= 1) {
    units += __shfl_xor(units, off, kWave);
    E += __shfl_xor(E, off, kWave);
    lmax = fmaxf(lmax, __shfl_xor(lmax, off, kWave));
    miss |= __shfl_xor(miss, off, kWave);
  }
  E = fmaf(a.p0_batch, lmax, E);         // static power over the longest task (per batch)
  const bool usable = kv && !bad && !miss && units < (long long)a.budget && E < kInf;
  float be = usable ? E : kInf;
  int bk = usable ? k : INT_MAX;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float oe = __shfl_xor(be, off, kWave);
    const int ok = __shfl_xor(bk, off, kWave);
    if (oe < be || (oe == be && ok < bk)) {
      be = oe;
      bk = ok;
    }
  }
  const bool found = bk != INT_MAX;
  if (lane == 0) {
    a.level[b] = found ? bk : -1;
    a.feasible[b] = found ? 1 : 0;
    a.energy[b] = found ? be : kInf;
  }
  // each task's SM level at the chosen frequency level: kept for the lane's first two
  // tasks, the same search repeated (bit-identical) for any further ones
  if (found && k == bk) {
    if (grp < nn) a.task_sm[row0 + grp] = jk0;
    if (grp + ngrp < nn) a.task_sm[row0 + grp + ngrp] = jk1;
    for (int t = grp + 2 * ngrp; t < nn; t += ngrp) {
      const float *col = (s_ph[wv][t] == 0 ? a.pf : a.dc) + s_col[wv][t] + k;
      float lat;
      a.task_sm[row0 + t] = min_sm_level(a, col, s_slack[wv][t], lat);
    }
  }
  for (int t = lane; t < a.T; t += kWave)
    if (!found || t >= nn) a.task_sm[row0 + t] = -1;
}

// Tables of 8 SM x 16 frequency levels and batches of at most 16 task slots: four batches
// per wavefront, 16 lanes each (lane = frequency level k), each lane walking its batch's
// tasks two at a time with all 16 table loads in flight.  Per (task, k) the SM level goes
// to LDS; after the 16-lane (energy, level) minimum, lane t of the batch writes task t's
// level at the chosen frequency.  Same arithmetic as k_sweep, so the same results.
constexpr int kFNS = 8, kFNF = 16, kFT = 16;
constexpr int kTasksInFlight = 2;             // 2 x 8 table loads issued together per lane
constexpr long long kSweepGrid = 8192;        // blocks of the grid-stride loop (one pass up to 131072 batches)
constexpr int kBatchesPerWave = kWave / kFNF;

__global__ void __launch_bounds__(kWavesPerBlock * kWave) k_sweep_8x16(SweepArgs a) {
  __shared__ float s_lev[kFNS];
  __shared__ int s_units[kFNS];
  __shared__ int s_col[kWavesPerBlock][kWave];       // [batch in wave * 16 + slot]
  __shared__ float s_slack[kWavesPerBlock][kWave];
  __shared__ int s_ph[kWavesPerBlock][kWave];
  __shared__ int8_t s_j[kWavesPerBlock][kBatchesPerWave][kFT][kFNF];
  if (threadIdx.x < kFNS) {
    s_lev[threadIdx.x] = a.sm_level[threadIdx.x];
    s_units[threadIdx.x] = a.units[threadIdx.x];
  }
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & (kWave - 1);
  const int g = lane >> 4, k = lane & (kFNF - 1);
  const int gs = g * kFNF;
  const float f = a.freq_level[k];
  const float f3 = f * f * f;
  constexpr int kPerBlock = kWavesPerBlock * kBatchesPerWave;
  const int n_units = (a.B + kPerBlock - 1) / kPerBlock;
  // grid-stride over groups of 16 batches (the loop count is uniform per block); a grid of
  // one block per group measured fastest, so the loop only serves very large calls
  for (int unit = blockIdx.x; unit < n_units; unit += gridDim.x) {
    const int b = (unit * kWavesPerBlock + wv) * kBatchesPerWave + g;
    const bool live = b < a.B;
    const size_t row0 = (size_t)(live ? b : 0) * a.T;

    // one memory round trip: lane k of a batch's group loads slot k
    int m = 0, ph = 0, tok = 0;
    float sl = 0.f;
    if (live && k < a.T) {
      m = a.model[row0 + k];
      ph = a.phase[row0 + k];
      tok = a.tokens[row0 + k];
      sl = a.slack[row0 + k];
    }
    const int n = live ? a.n_tasks[b] : 0;
    const float kd = live ? a.kdyn[b] : 0.f, u = live ? a.util[b] : 0.f;
    const bool n_ok = n >= 0 && n <= a.T;
    const int nn = n_ok ? n : 0;
    int row = 0;
    if (k < nn) {
      row = task_row(a, m, ph, tok);
      s_col[wv][lane] = row >= 0 ? (m * kRows + row) * (kFNS * kFNF) : 0;
      s_slack[wv][lane] = sl;
      s_ph[wv][lane] = ph;
    }
    __syncthreads();
    const unsigned long long badm = __ballot(k < nn && row < 0);
    const bool bad = !live || !n_ok || ((badm >> (kFNF * g)) & 0xffffull) != 0;

    const float c = kd * u * f3;
    long long units = 0;
    float E = 0.f, lmax = 0.f;
    int miss = 0;
    for (int t = 0; !bad && t < nn; t += kTasksInFlight) {
      const float *cp[kTasksInFlight];
      float slk[kTasksInFlight];
#pragma unroll
      for (int i = 0; i < kTasksInFlight; ++i) {
        const int ti = t + i < nn ? t + i : t;   // a slot of this batch either way
        cp[i] = (s_ph[wv][gs + ti] == 0 ? a.pf : a.dc) + s_col[wv][gs + ti] + k;
        slk[i] = s_slack[wv][gs + ti];
      }
      float v[kTasksInFlight][kJChunk];
#pragma unroll
      for (int i = 0; i < kTasksInFlight; ++i)
#pragma unroll
        for (int q = 0; q < kJChunk; ++q) v[i][q] = cp[i][q * kFNF];
#pragma unroll
      for (int i = 0; i < kTasksInFlight; ++i) {
        if (t + i >= nn) break;
        float lat;
        const int j = first_below(v[i], slk[i], lat);
        s_j[wv][g][t + i][k] = (int8_t)j;
        if (j < 0) {
          miss = 1;
        } else {
          units += s_units[j];
          E = fmaf(fmaf(c, s_lev[j], a.p0_task), lat, E);
          lmax = fmaxf(lmax, lat);
        }
      }
    }
    E = fmaf(a.p0_batch, lmax, E);       // static power over the longest task (per batch)
    const bool usable = !bad && !miss && units < (long long)a.budget && E < kInf;
    float be = usable ? E : kInf;
    int bk = usable ? k : INT_MAX;
#pragma unroll
    for (int off = kFNF / 2; off >= 1; off >>= 1) {
      const float oe = __shfl_xor(be, off, kWave);
      const int ok = __shfl_xor(bk, off, kWave);
      if (oe < be || (oe == be && ok < bk)) {
        be = oe;
        bk = ok;
      }
    }
    const bool found = bk != INT_MAX;
    __syncthreads();                       // the SM levels in s_j are visible to every lane
    if (live) {
      if (k == 0) {
        a.level[b] = found ? bk : -1;
        a.feasible[b] = found ? 1 : 0;
        a.energy[b] = found ? be : kInf;
      }
      if (k < a.T) a.task_sm[row0 + k] = (found && k < nn) ? (int)s_j[wv][g][k][bk] : -1;
    }
  }
}

}  // namespace

extern "C" festina_status festina_sweep_batches(const festina_lut *L, const festina_batches *S,
                                                festina_sweep_result *out, void *stream) {
  if (!L || !S || !out) return FESTINA_ERR_INVALID;
  if (L->n_models < 1 || L->n_rows != kRows || L->n_sm < 1 || L->n_freq < 1) return FESTINA_ERR_INVALID;
  if (S->n_batches < 0 || S->max_tasks < 1) return FESTINA_ERR_INVALID;
  if (S->static_power != FESTINA_STATIC_PER_TASK && S->static_power != FESTINA_STATIC_PER_BATCH)
    return FESTINA_ERR_INVALID;
  if (L->n_freq > FESTINA_MAX_FREQ_SWEEP || L->n_sm > kMaxSm || S->max_tasks > FESTINA_MAX_TASKS)
    return FESTINA_ERR_UNSUPPORTED;
  if (!L->sm_level || !L->freq_level || !L->pf || !L->dc || !S->sm_units) return FESTINA_ERR_INVALID;
  if (S->n_batches == 0) return FESTINA_OK;
  if (!S->n_tasks || !S->task_model || !S->task_phase || !S->task_tokens || !S->task_slack_ms ||
      !S->k_dyn_w || !S->util)
    return FESTINA_ERR_INVALID;
  if (!out->freq_level || !out->feasible || !out->energy_mj || !out->task_sm) return FESTINA_ERR_INVALID;
  SweepArgs a;
  a.M = L->n_models;
  a.NS = L->n_sm;
  a.NF = L->n_freq;
  a.sm_level = L->sm_level;
  a.freq_level = L->freq_level;
  a.pf = L->pf;
  a.dc = L->dc;
  a.B = S->n_batches;
  a.T = S->max_tasks;
  a.n_tasks = S->n_tasks;
  a.model = S->task_model;
  a.phase = S->task_phase;
  a.tokens = S->task_tokens;
  a.slack = S->task_slack_ms;
  a.kdyn = S->k_dyn_w;
  a.util = S->util;
  a.units = S->sm_units;
  a.budget = S->sm_budget;
  a.p0_task = S->static_power == FESTINA_STATIC_PER_TASK ? L->p0_w : 0.f;
  a.p0_batch = S->static_power == FESTINA_STATIC_PER_BATCH ? L->p0_w : 0.f;
  a.lg = 0;
  while ((1 << a.lg) < a.NF) ++a.lg;
  a.level = out->freq_level;
  a.feasible = out->feasible;
  a.energy = out->energy_mj;
  a.task_sm = out->task_sm;
  hipStream_t st = static_cast<hipStream_t>(stream);
  // the specialised kernel: 8 x 16 tables, at most 16 slots, 32-bit table offsets
  const bool fast = a.NS == kFNS && a.NF == kFNF && a.T <= kFT && a.M <= (INT_MAX / (kRows * kFNS * kFNF));
  if (fast) {
    const long long per = (long long)kWavesPerBlock * kBatchesPerWave;
    const long long units = ((long long)a.B + per - 1) / per;
    const long long blocks = units < kSweepGrid ? units : kSweepGrid;
    k_sweep_8x16<<<(unsigned)blocks, kWavesPerBlock * kWave, 0, st>>>(a);
  } else {
    const long long blocks = ((long long)a.B + kWavesPerBlock - 1) / kWavesPerBlock;
    k_sweep<<<(unsigned)blocks, kWavesPerBlock * kWave, 0, st>>>(a);
  }
  return hipGetLastError() == hipSuccess ? FESTINA_OK : FESTINA_ERR_DEVICE;
}
