// festina.hip -- MI355X (gfx950) kernels and C-ABI host dispatch of the batched
// energy-aware placement and migration search (Festina, Sec. 3.3 and Sec. 3.5).
//
// Placement pipeline (one call, five launches on the caller's stream):
//   k_zero      clear the bucket counters
//   k_prep      requests: validity, bucket key (wave, model, has-prompt), the bucket count
//                 and the request's position within its bucket; hosts: per-model list of
//                 hosting GPUs in ascending order; GPU records: per (wave, GPU) the
//                 post-admission batch row, k_g * u_g and the SM caps
//   k_scan      one block: bucket offsets and the tile table (only with more buckets than
//                 an LDS histogram holds)
//   k_scatter   request records (5% output pad, prompt bucket, SLOs) grouped by bucket
//   k_score     one workgroup per tile (requests of one bucket): the model's decode table is
//                 staged in LDS; each wave scores Q requests at once, lanes spanning the
//                 (SM level, frequency level) cells, looping over the hosting GPUs; the
//                 per-request argmin is fused (running minimum per lane, then a wavefront
//                 reduction with lowest-index tie-break); only 9 bytes per request reach HBM
// Migration pipeline:
//   k_fleet     per GPU: bitmask of frequency levels at which all instances meet their SLOs,
//                 its lowest level and the dynamic-power baseline f[kd0]^3 * u
//   k_migrate   two sources per block, each source's destinations split over two
//                 wavefronts, lanes spanning destinations; fused per-source argmax with
//                 lowest-destination tie-break
//
// Exactness: every SLO and budget test compares a table entry with an SLO, or integers,
// so it is decided bit-identically to any other correct implementation.  Energies are
// float32: Pp = fma(k_g*u_g, s*f^3, P0), X = Pp*TTFT, Y = Pd*TBT, E = fma(Lout, Y, X).
#include <hip/hip_runtime.h>

#include <atomic>
#include <climits>
#include <cmath>
#include <cstddef>
#include <cstdint>
#include <mutex>

#include "festina.h"

namespace {

constexpr int kRows = FESTINA_N_ROWS;
constexpr int kWave = 64;
constexpr int kQ = 4;            // requests scored together by one wavefront
constexpr int kPrepBlock = 256;
constexpr float kInf = __builtin_huge_valf();
// Value of a masked (SLO-missing) latency: a quiet NaN stays NaN through every multiply and
// FMA whatever the sign of the power terms, and NaN < x is false, so it never wins.
constexpr float kMask = __builtin_nanf("");

struct HostRec {                 // per (wave, GPU), 16 bytes
  int32_t row_off;               // (b - 1) * cells, or -1 when the GPU has no candidates
  float kappa;                   // k_g * b / 32
  int32_t caps;                  // cap_pf | cap_dc << 8
  int32_t pad;
};

struct ReqRec {                  // one request in bucket order, 32 bytes
  int32_t r;                     // request index
  int32_t row;                   // prompt row (-1: the decode batch row)
  float lout;                    // padded output tokens
  float slo_ttft, slo_tbt;
  float rlout;                   // 1 / lout when lout is in [1, 2^40], else 0
  int32_t pad[2];
};

struct PlaceArgs {
  // table
  int32_t M, NS, NF, C;          // C = NS * NF
  const float *sm_level, *freq_level, *pf, *dc;
  float p0;
  // gpus
  int32_t G, W, words;
  const int32_t *batch;
  const float *kdyn;
  const uint32_t *resident;
  const int8_t *cap_pf, *cap_dc;
  int32_t has_caps;
  // requests
  int32_t R;
  const int32_t *model, *wave, *prompt, *pred;
  const float *slo_ttft, *slo_tbt;
  // outputs
  int32_t *choice;
  uint8_t *feasible;
  float *energy;
  // workspace
  int32_t NB;                    // buckets = 2 * W * M
  int32_t tile;                  // requests per tile
  int32_t max_tiles;
  int32_t *cnt;                  // [NB4] counters
  int32_t *bstart;               // [NB + 1]
  int32_t *n_tiles;              // [1]
  int2 *tiles;                   // [max_tiles] {bucket, first position}
  int32_t *host_cnt;             // [M]
  int32_t *host_list;            // [M][G]
  HostRec *recs;                 // [W][G]
  ReqRec *preq;                  // [R] request records in bucket order
  int32_t *key;                  // [R]
  int32_t *off;                  // [R] position of request r within its bucket
};

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

__device__ __forceinline__ float cube(float f) { return f * f * f; }

// Read-only view in the constant address space: buffers that a kernel never writes
// (tables, request fields, the host lists and records made by earlier launches) are
// then read with scalar loads into SGPRs wherever the address is wave-uniform.
template <typename T>
__device__ __forceinline__ const __attribute__((address_space(4))) T *ro(const T *p) {
  return (const __attribute__((address_space(4))) T *)(p);
}

typedef int v4i __attribute__((ext_vector_type(4)));

__device__ __forceinline__ HostRec load_rec(const __attribute__((address_space(4))) HostRec *rw, int g) {
  const auto p = reinterpret_cast<const __attribute__((address_space(4))) v4i *>(rw) + g;
  const v4i v = *p;
  HostRec r;
  r.row_off = v.x;
  r.kappa = __int_as_float(v.y);
  r.caps = v.z;
  r.pad = v.w;
  return r;
}

// Request record at bucket position pos (wave-uniform): two scalar 16-byte loads.
__device__ __forceinline__ ReqRec load_req(const PlaceArgs &a, int pos) {
  const auto p = ro(reinterpret_cast<const v4i *>(a.preq + pos));
  const v4i x = p[0], y = p[1];
  ReqRec q;
  q.r = x.x;
  q.row = x.y;
  q.lout = __int_as_float(x.z);
  q.slo_ttft = __int_as_float(x.w);
  q.slo_tbt = __int_as_float(y.x);
  q.rlout = __int_as_float(y.y);
  q.pad[0] = q.pad[1] = 0;
  return q;
}

// Request record at bucket position pos, per lane (vector loads).
__device__ __forceinline__ ReqRec load_req_lane(const PlaceArgs &a, int pos) {
  const v4i *p = reinterpret_cast<const v4i *>(a.preq + pos);
  const v4i x = p[0], y = p[1];
  ReqRec q;
  q.r = x.x;
  q.row = x.y;
  q.lout = __int_as_float(x.z);
  q.slo_ttft = __int_as_float(x.w);
  q.slo_tbt = __int_as_float(y.x);
  q.rlout = __int_as_float(y.y);
  q.pad[0] = q.pad[1] = 0;
  return q;
}

// ------------------------------------------------------------------ prologue kernels
// Inclusive prefix sum over a wavefront.
__device__ __forceinline__ int wave_scan(int v) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    const int o = __shfl_up(v, off, kWave);
    if (lane >= off) v += o;
  }
  return v;
}

__global__ void k_zero(int32_t *p, int32_t n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

// The fields of request r that decide its bucket.
struct ReqKeyFields {
  int m, w, pt, pr;
};
__device__ __forceinline__ ReqKeyFields load_key_fields(const PlaceArgs &a, int r) {
  return ReqKeyFields{a.model[r], a.wave ? a.wave[r] : 0, a.prompt[r], a.pred[r]};
}

// Validity and bucket key (wave, model, has-prompt) of request r from its fields.  Returns
// the key, or -1 (and writes the infeasible result) for an invalid request.
__device__ __forceinline__ int prep_request(const PlaceArgs &a, int r, const ReqKeyFields &f) {
  const bool ok = f.m >= 0 && f.m < a.M && f.w >= 0 && f.w < a.W && f.pt >= 0 && f.pr >= 0;
  if (!ok) {
    a.key[r] = -1;
    a.choice[r] = -1;
    a.feasible[r] = 0;
    a.energy[r] = kInf;
    return -1;
  }
  const int k = ((f.w * a.M + f.m) << 1) | (f.pt == 0 ? 1 : 0);
  a.key[r] = k;
  return k;
}

__device__ const int8_t kNoCap = 0;                // read in place of absent cap arrays

constexpr int kReqPerPrepBlock = 4 * kPrepBlock;  // requests per request block of k_prep / k_scatter
constexpr int kHistMax = 8192;                    // buckets counted in LDS (else global atomics)

// Blocks [0, nbr): kReqPerPrepBlock requests each, counted per bucket in an LDS histogram
// and flushed with one global atomic per non-empty bucket; the atomics' old values give each
// request its position within its bucket (its rank in the block's count plus the block's
// base), so the scatter needs no further atomics.  Blocks [nbr, nbr + M): host list of model
// (block - nbr).  Blocks after: GPU records, one thread per (wave, GPU).
__global__ void __launch_bounds__(kPrepBlock) k_prep(PlaceArgs a, int32_t nbr) {
  __shared__ int hist[kHistMax];
  const int b = blockIdx.x;
  if (b < nbr) {
    const bool local = a.NB <= kHistMax;
    constexpr int U = kReqPerPrepBlock / kPrepBlock;
    // every request's fields are requested before the first is used (one memory round trip);
    // a thread past the last request reads the last one (R >= 1 in a request block) and
    // drops it
    ReqKeyFields f[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      f[u] = load_key_fields(a, min(b * kReqPerPrepBlock + u * kPrepBlock + (int)threadIdx.x, a.R - 1));
    if (local) {
      for (int k = threadIdx.x; k < a.NB; k += kPrepBlock) hist[k] = 0;
      __syncthreads();
    }
    int key[U], pos[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = b * kReqPerPrepBlock + u * kPrepBlock + threadIdx.x;
      key[u] = r < a.R ? prep_request(a, r, f[u]) : -1;
      pos[u] = key[u] >= 0 ? atomicAdd(local ? &hist[key[u]] : &a.cnt[key[u]], 1) : 0;
    }
    if (local) {
      __syncthreads();
      for (int k = threadIdx.x; k < a.NB; k += kPrepBlock)
        if (hist[k]) hist[k] = atomicAdd(&a.cnt[k], hist[k]);   // this block's base in bucket k
      __syncthreads();
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (key[u] >= 0) pos[u] += hist[key[u]];
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (key[u] >= 0) a.off[b * kReqPerPrepBlock + u * kPrepBlock + threadIdx.x] = pos[u];
    return;
  }
  if (b < nbr + a.M) {
    // ascending list of GPUs whose resident mask has bit m
    const int m = b - nbr;
    __shared__ int wsum[kPrepBlock / kWave];
    __shared__ int base_s;
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x >> 6;
    if (threadIdx.x == 0) base_s = 0;
    __syncthreads();
    for (int g0 = 0; g0 < a.G; g0 += kPrepBlock) {
      const int g = g0 + threadIdx.x;
      const bool has = g < a.G && ((a.resident[(size_t)g * a.words + (m >> 5)] >> (m & 31)) & 1u);
      const unsigned long long bal = __ballot(has);
      const int before = __popcll(bal & ((1ull << lane) - 1ull));
      if (lane == 0) wsum[wv] = __popcll(bal);
      __syncthreads();
      int off = base_s;
      for (int i = 0; i < wv; ++i) off += wsum[i];
      if (has) a.host_list[(size_t)m * a.G + off + before] = g;
      __syncthreads();
      if (threadIdx.x == 0) {
        int t = 0;
        for (int i = 0; i < kPrepBlock / kWave; ++i) t += wsum[i];
        base_s += t;
      }
      __syncthreads();
    }
    if (threadIdx.x == 0) a.host_cnt[m] = base_s;
    return;
  }
  const long long i = (long long)(b - nbr - a.M) * kPrepBlock + threadIdx.x;
  if (i >= (long long)a.W * a.G) return;
  const int g = (int)(i % a.G);
  // all four loads in flight together: without caps the cap loads read a constant in
  // device memory and are replaced by NS - 1
  const int B = a.batch[i];
  const float kd = a.kdyn[g];
  const int8_t cpv = *(a.cap_pf ? a.cap_pf + g : &kNoCap);
  const int8_t cdv = *(a.cap_dc ? a.cap_dc + g : &kNoCap);
  const int cp = a.cap_pf ? (int)cpv : a.NS - 1;
  const int cd = a.cap_dc ? (int)cdv : a.NS - 1;
  HostRec rec;
  const bool ok = B >= 0 && cp >= 0 && cp < a.NS && cd >= 0 && cd < a.NS;
  const int bb = B + 1 > kRows ? kRows : B + 1;
  rec.row_off = ok ? (bb - 1) * a.C : -1;
  // u = b / 32 is exact; a GPU without candidates gets NaN so that every energy on it is NaN
  rec.kappa = ok ? kd * ((float)bb * 0.03125f) : kMask;
  rec.caps = ok ? (cp | (cd << 8)) : 0;
  rec.pad = 0;
  a.recs[i] = rec;
}

constexpr int kScanLds = 16384;   // bucket counts staged in LDS by k_scan (64 KB)

// Scan body over bucket counts `cnt` (LDS copy or the global counters themselves).
template <typename P>
__device__ __forceinline__ void scan_buckets(const PlaceArgs &a, P cnt, int *s_cnt, int *s_til) {
  const int T = blockDim.x;
  const int per = (a.NB + T - 1) / T;
  const int lo = threadIdx.x * per;
  const int hi = min(lo + per, a.NB);
  int c = 0, t = 0;
  for (int i = lo; i < hi; ++i) {
    const int n = cnt[i];
    c += n;
    t += (n + a.tile - 1) / a.tile;
  }
  const int ic = wave_scan(c), it = wave_scan(t);
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  if (lane == kWave - 1) {
    s_cnt[wv] = ic;
    s_til[wv] = it;
  }
  __syncthreads();
  int pc = ic - c, pt = it - t;                  // exclusive prefix within the wave
  int tot_c = 0, tot_t = 0;
  for (int i = 0; i < T / kWave; ++i) {
    if (i < wv) {
      pc += s_cnt[i];
      pt += s_til[i];
    }
    tot_c += s_cnt[i];
    tot_t += s_til[i];
  }
  for (int i = lo; i < hi; ++i) {
    const int n = cnt[i];
    a.bstart[i] = pc;
    const int nt = (n + a.tile - 1) / a.tile;
    for (int q = 0; q < nt; ++q) a.tiles[pt + q] = make_int2(i, pc + q * a.tile);
    pc += n;
    pt += nt;
  }
  if (threadIdx.x == 0) {
    a.bstart[a.NB] = tot_c;
    *a.n_tiles = tot_t;
  }
}

// One block of 1024 threads: exclusive scans of bucket counts and tiles-per-bucket, and
// the tile table.  Counts are first copied to LDS in one coalesced
// pass when they fit, so the scan never waits on a global load after a global store.
__global__ void __launch_bounds__(1024) k_scan(PlaceArgs a) {
  __shared__ int s_cnt[1024 / kWave];
  __shared__ int s_til[1024 / kWave];
  extern __shared__ int lcnt[];     // [NB] when NB <= kScanLds
  if (a.NB <= kScanLds) {
    constexpr int U = 4;            // loads in flight per thread before the first wait
    for (int i0 = 0; i0 < a.NB; i0 += U * 1024) {
      int v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * 1024 + threadIdx.x;
        v[u] = i < a.NB ? __builtin_nontemporal_load(&a.cnt[i]) : 0;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int i = i0 + u * 1024 + threadIdx.x;
        if (i < a.NB) lcnt[i] = v[u];
      }
    }
    __syncthreads();
    scan_buckets(a, lcnt, s_cnt, s_til);
  } else {
    scan_buckets(a, a.cnt, s_cnt, s_til);
  }
}

// Record of valid request r: prompt bucket min(ceil(tokens / 256), 32) - 1 (unsigned: no
// overflow for any int32 token count; 0 tokens -> -1, the decode batch row), the 5% output
// pad ceil(1.05 * pred) = (105 * pred + 99) / 100 in 64-bit, its reciprocal (0 outside
// [1, 2^40]), and the SLOs.
__device__ __forceinline__ ReqRec make_req_rec(const PlaceArgs &a, int r) {
  const int pt = a.prompt[r];
  ReqRec q;
  q.r = r;
  q.row = pt == 0 ? -1 : (min((int)(((unsigned)pt + 255u) >> 8), kRows) - 1);
  q.lout = (float)(((long long)a.pred[r] * 105 + 99) / 100);
  q.slo_ttft = a.slo_ttft[r];
  q.slo_tbt = a.slo_tbt[r];
  q.rlout = q.lout >= 1.f && q.lout <= 0x1p40f ? 1.f / q.lout : 0.f;
  q.pad[0] = q.pad[1] = 0;
  return q;
}

// Exclusive scans of the bucket counts (requests and tiles) inside one block of k_scatter,
// into the LDS array `start`.  Thread t holds buckets [t*per, t*per + per), per a multiple
// of 4 (at most 32), loaded by load_scan_counts as 8 int4 loads that are all in flight
// before the first use; the counter array is padded to a multiple of 4 with zeros.  Every block scans all buckets
// (a few KB from L2); the global starts and tiles of thread t's buckets are written by block
// t mod grid, so the tile table is spread over the grid, and block 0 writes the totals.
constexpr int kScanChunks = kHistMax / kPrepBlock / 4;   // int4 chunks of counts per thread

// Thread t's bucket range [lo, hi) of the block scan: per buckets, a multiple of 4.
__device__ __forceinline__ int2 scan_range(const PlaceArgs &a) {
  const int per = (((a.NB + kPrepBlock - 1) / kPrepBlock) + 3) & ~3;
  const int lo = min((int)threadIdx.x * per, a.NB);
  return make_int2(lo, min(lo + per, a.NB));
}

// Thread t's bucket counts for the block scan, requested without waiting: chunk q is read at
// min(lo + 4q, NB4 - 4), always inside the padded counter array, and block_scan_buckets
// counts it as zero past hi.
__device__ __forceinline__ void load_scan_counts(const PlaceArgs &a, v4i (&v)[kScanChunks]) {
  const int lo = scan_range(a).x;
  const int last4 = ((a.NB + 3) & ~3) - 4;
#pragma unroll
  for (int q = 0; q < kScanChunks; ++q) v[q] = *reinterpret_cast<const v4i *>(a.cnt + min(lo + 4 * q, last4));
}

__device__ void block_scan_buckets(const PlaceArgs &a, int *start, v4i (&v)[kScanChunks]) {
  __shared__ int s_c[kPrepBlock / kWave];
  __shared__ int s_t[kPrepBlock / kWave];
  constexpr int V = kScanChunks;
  const int lo = scan_range(a).x, hi = scan_range(a).y;
  const int tsh = __builtin_ctz((unsigned)a.tile);   // the tile size is a power of two
#pragma unroll
  for (int q = 0; q < V; ++q)
    if (lo + 4 * q >= hi) v[q] = v4i{0, 0, 0, 0};
  int c = 0, t = 0;
#pragma unroll
  for (int q = 0; q < V; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int n = v[q][e];
      c += n;
      t += (n + a.tile - 1) >> tsh;
    }
  const int ic = wave_scan(c), it = wave_scan(t);
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  if (lane == kWave - 1) {
    s_c[wv] = ic;
    s_t[wv] = it;
  }
  __syncthreads();
  int pc = ic - c, pt = it - t;
  int tot_c = 0, tot_t = 0;
  for (int i = 0; i < kPrepBlock / kWave; ++i) {
    if (i < wv) {
      pc += s_c[i];
      pt += s_t[i];
    }
    tot_c += s_c[i];
    tot_t += s_t[i];
  }
  // thread t's buckets are published by block t mod grid (every t < 256 names one block)
  const bool writer = (int)threadIdx.x % (int)gridDim.x == (int)blockIdx.x;
#pragma unroll
  for (int q = 0; q < V; ++q)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int i = lo + 4 * q + e;
      if (i < hi) {
        const int n = v[q][e];
        const int nt = (n + a.tile - 1) >> tsh;
        start[i] = pc;
        if (writer) {
          a.bstart[i] = pc;
          for (int k = 0; k < nt; ++k) a.tiles[pt + k] = make_int2(i, pc + k * a.tile);
        }
        pc += n;
        pt += nt;
      }
    }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    a.bstart[a.NB] = tot_c;
    *a.n_tiles = tot_t;
  }
  __syncthreads();
}

// Requests grouped by bucket: request r goes to its bucket's start plus its position from
// k_prep.  With at most kHistMax buckets each block scans the bucket counts itself (dynamic
// LDS: starts [NB]); with more, k_scan has written the bucket starts.
constexpr int kScatterU = kReqPerPrepBlock / kPrepBlock;

// Request u of this thread: bucket key (-1: none), position and record.  Every load is issued
// before the first use; a thread past the last request reads the last one (R >= 1) and drops
// it, and an invalid request's position (never written) is not used.
__device__ __forceinline__ void scatter_loads(const PlaceArgs &a, int (&key)[kScatterU], int (&pos)[kScatterU],
                                              ReqRec (&rec)[kScatterU]) {
#pragma unroll
  for (int u = 0; u < kScatterU; ++u) {
    const int r = blockIdx.x * kReqPerPrepBlock + u * kPrepBlock + threadIdx.x;
    const int rc = min(r, a.R - 1);
    key[u] = a.key[rc];
    pos[u] = a.off[rc];
    rec[u] = make_req_rec(a, rc);
    if (r >= a.R) key[u] = -1;
  }
}

__global__ void __launch_bounds__(kPrepBlock) k_scatter(PlaceArgs a) {
  extern __shared__ int start[];
  int key[kScatterU], pos[kScatterU];
  ReqRec rec[kScatterU];
  if (a.NB <= kHistMax) {
    // the bucket counts are requested together with the request fields: one round trip
    v4i cv[kScanChunks];
    load_scan_counts(a, cv);
    scatter_loads(a, key, pos, rec);
    __builtin_amdgcn_sched_barrier(0);   // no use of a loaded value is scheduled before a load
    block_scan_buckets(a, start, cv);    // ends with a barrier
#pragma unroll
    for (int u = 0; u < kScatterU; ++u)
      if (key[u] >= 0) a.preq[start[key[u]] + pos[u]] = rec[u];
  } else {
    scatter_loads(a, key, pos, rec);
#pragma unroll
    for (int u = 0; u < kScatterU; ++u)
      if (key[u] >= 0) a.preq[a.bstart[key[u]] + pos[u]] = rec[u];
  }
}

// ------------------------------------------------------------------ scoring kernel
// (E, idx) lexicographic minimum across the wavefront; idx = INT_MAX means "none".
__device__ __forceinline__ void wave_argmin(float &e, int &id) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float oe = __shfl_xor(e, off, kWave);
    const int oi = __shfl_xor(id, off, kWave);
    if (oe < e || (oe == e && oi < id)) {
      e = oe;
      id = oi;
    }
  }
}

// CPL = cells per lane (consecutive cells c = lane*CPL + t).
// LDS floats needed by k_score<CPL>: the decode table plus a pad that lanes past the
// last cell may read (their values are masked), s*f^3, and the per-wave prompt rows.
__host__ __device__ constexpr size_t score_lds_floats(int C, int CPL, int waves) {
  return (size_t)kRows * C + (size_t)kWave * CPL + C + (size_t)waves * kQ * C;
}

template <int CPL>
__device__ void score_tile_generic(const PlaceArgs &a, int t, float *lds) {
  const int C = a.C, NF = a.NF;
  float *dcs = lds;                                   // [32 * C + pad] decode table of the tile's model
  float *pds = lds + kRows * C + kWave * CPL;         // [C] s_j * f_k^3
  float *rows = pds + C;                              // [waves][Q][C] prompt rows (capped GPUs)

  const auto tp = ro(reinterpret_cast<const int32_t *>(a.tiles));
  const int bucket = tp[2 * t];
  const bool noprompt = bucket & 1;
  const int wm = bucket >> 1;
  const int w = wm / a.M, m = wm - (wm / a.M) * a.M;
  const int beg = tp[2 * t + 1];
  const int end = min(beg + a.tile, ro(a.bstart)[bucket + 1]);

  // stage the model's decode table and the dynamic-power factors
  {
    const float *src = a.dc + (size_t)m * kRows * C;
    const int n = kRows * C;
    if ((((uintptr_t)src) & 15) == 0) {
      const float4 *s4 = reinterpret_cast<const float4 *>(src);
      float4 *d4 = reinterpret_cast<float4 *>(dcs);
      for (int i = threadIdx.x; i < n / 4; i += blockDim.x) d4[i] = s4[i];
    } else {
      for (int i = threadIdx.x; i < n; i += blockDim.x) dcs[i] = src[i];
    }
    for (int i = threadIdx.x; i < kWave * CPL; i += blockDim.x) dcs[n + i] = 0.f;
    for (int i = threadIdx.x; i < C; i += blockDim.x) {
      const int j = i / NF, k = i - (i / NF) * NF;
      pds[i] = a.sm_level[j] * cube(a.freq_level[k]);
    }
  }
  __syncthreads();

  const int nwaves = blockDim.x / kWave;
  const int wv = uniform(threadIdx.x >> 6);
  const int lane = threadIdx.x & (kWave - 1);
  float *myrows = rows + (size_t)wv * kQ * C;
  const int hcnt = ro(a.host_cnt)[m];
  const auto hl = ro(a.host_list + (size_t)m * a.G);
  const auto rw = ro(a.recs + (size_t)w * a.G);
  const float p0 = a.p0;
  const bool caps = a.has_caps != 0;

  int cj[CPL], ck[CPL];
  bool live[CPL];
  float pdl[CPL];
#pragma unroll
  for (int u = 0; u < CPL; ++u) {
    const int c = lane * CPL + u;
    live[u] = c < C;
    const int cc = live[u] ? c : 0;
    cj[u] = cc / NF;
    ck[u] = cc - cj[u] * NF;
    pdl[u] = pds[cc];
  }

  for (int base = beg + wv * kQ; base < end; base += nwaves * kQ) {
    int rq[kQ];
    float lo[kQ], st[kQ], sb[kQ];
    int prw[kQ];
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const int pos = base + q;
      const ReqRec rr = load_req(a, pos < end ? pos : beg);
      rq[q] = pos < end ? rr.r : -1;
      if (rq[q] >= 0) {
        lo[q] = rr.lout;
        st[q] = rr.slo_ttft;
        sb[q] = rr.slo_tbt;
        prw[q] = rr.row;
      } else {
        lo[q] = 0.f;
        st[q] = -kInf;                    // nothing is below -inf: never feasible
        sb[q] = -kInf;
        prw[q] = 0;
      }
    }
    float be[kQ][CPL];
    int bg[kQ][CPL];
#pragma unroll
    for (int q = 0; q < kQ; ++q)
#pragma unroll
      for (int u = 0; u < CPL; ++u) {
        be[q][u] = kInf;
        bg[q][u] = -1;
      }

    if (noprompt) {
      // TTFT from the prefill table at the decode batch row (global, L2-resident)
      const float *pfm = a.pf + (size_t)m * kRows * C;
      for (int i = 0; i < hcnt; ++i) {
        const int g = hl[i];
        const HostRec rec = load_rec(rw, g);
        if (rec.row_off < 0) continue;
        const int cp = rec.caps & 0xff, cd = (rec.caps >> 8) & 0xff;
#pragma unroll
        for (int u = 0; u < CPL; ++u) {
          const int cP = min(cj[u], cp) * NF + ck[u];
          const int cD = min(cj[u], cd) * NF + ck[u];
          const float tbt = dcs[rec.row_off + cD];
          const float ttft = pfm[rec.row_off + cP];
          const float Pp = fmaf(rec.kappa, pds[cP], p0);
          const float Pd = fmaf(rec.kappa, pds[cD], p0);
          const float X = Pp * ttft;
          const float Y = Pd * tbt;
#pragma unroll
          for (int q = 0; q < kQ; ++q) {
            const float E = fmaf(lo[q], Y, X);
            const bool ok = live[u] && ttft < st[q] && tbt < sb[q] && E < be[q][u];
            be[q][u] = ok ? E : be[q][u];
            bg[q][u] = ok ? g : bg[q][u];
          }
        }
      }
    } else if (!caps) {
      // uncapped: the request's TTFT cells stay in registers, masked by its TTFT SLO
      float tt[kQ][CPL];
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
        const float *pr = a.pf + ((size_t)m * kRows + prw[q]) * C;
#pragma unroll
        for (int u = 0; u < CPL; ++u) {
          const float v = (rq[q] >= 0 && live[u]) ? pr[lane * CPL + u] : kInf;
          tt[q][u] = v < st[q] ? v : kMask;
        }
      }
      for (int i = 0; i < hcnt; ++i) {
        const int g = hl[i];
        const HostRec rec = load_rec(rw, g);
        if (rec.row_off < 0) continue;
        const float *drow = dcs + rec.row_off + lane * CPL;
#pragma unroll
        for (int u = 0; u < CPL; ++u) {
          const float tbt = drow[u];
          const float P = fmaf(rec.kappa, pdl[u], p0);
          const float Y = P * tbt;
#pragma unroll
          for (int q = 0; q < kQ; ++q) {
            const float X = P * tt[q][u];
            const float E = fmaf(lo[q], Y, X);
            const bool ok = tbt < sb[q] && E < be[q][u];
            be[q][u] = ok ? E : be[q][u];
            bg[q][u] = ok ? g : bg[q][u];
          }
        }
      }
    } else {
      // capped GPUs: stage each request's masked prompt row in LDS, read at min(j, cap)
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
        const float *pr = a.pf + ((size_t)m * kRows + prw[q]) * C;
        for (int c = lane; c < C; c += kWave) {
          const float v = rq[q] >= 0 ? pr[c] : kInf;
          myrows[q * C + c] = v < st[q] ? v : kMask;
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      for (int i = 0; i < hcnt; ++i) {
        const int g = hl[i];
        const HostRec rec = load_rec(rw, g);
        if (rec.row_off < 0) continue;
        const int cp = rec.caps & 0xff, cd = (rec.caps >> 8) & 0xff;
#pragma unroll
        for (int u = 0; u < CPL; ++u) {
          const int cP = min(cj[u], cp) * NF + ck[u];
          const int cD = min(cj[u], cd) * NF + ck[u];
          const float tbt = dcs[rec.row_off + cD];
          const float Pp = fmaf(rec.kappa, pds[cP], p0);
          const float Pd = fmaf(rec.kappa, pds[cD], p0);
          const float Y = Pd * tbt;
#pragma unroll
          for (int q = 0; q < kQ; ++q) {
            const float X = Pp * myrows[q * C + cP];
            const float E = fmaf(lo[q], Y, X);
            const bool ok = live[u] && tbt < sb[q] && E < be[q][u];
            be[q][u] = ok ? E : be[q][u];
            bg[q][u] = ok ? g : bg[q][u];
          }
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }

    // per request: lane minimum over its cells, then the wavefront argmin
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      float e = kInf;
      int id = INT_MAX;
#pragma unroll
      for (int u = 0; u < CPL; ++u) {
        if (bg[q][u] >= 0) {
          const int cand = bg[q][u] * C + lane * CPL + u;
          if (be[q][u] < e || (be[q][u] == e && cand < id)) {
            e = be[q][u];
            id = cand;
          }
        }
      }
      wave_argmin(e, id);
      if (lane == 0 && rq[q] >= 0) {
        const bool found = id != INT_MAX;
        a.choice[rq[q]] = found ? id : -1;
        a.feasible[rq[q]] = found ? 1 : 0;
        a.energy[rq[q]] = found ? e : kInf;
      }
    }
  }
}

template <int CPL>
__global__ void __launch_bounds__(256) k_score(PlaceArgs a) {
  extern __shared__ __align__(16) float lds[];
  if ((int)blockIdx.x >= *ro(a.n_tiles)) return;
  score_tile_generic<CPL>(a, blockIdx.x, lds);
}

// ------------------------------------------------------------------ 8 x 16 scoring kernel
// Tables of 8 SM levels x 16 frequency levels (128 cells).  Lane l owns cells 2l and 2l+1,
// which share SM level j = l / 8, so a capped cell offset is one min on byte offsets,
// min(j * 64, cap * 64) + k * 4, and the LDS offsets below are compile-time immediates.
//
// A workgroup takes a tile of WPB * kQF requests of one (wave, model) bucket; each
// wavefront scores its kQF requests together against every hosting GPU.
//   pass 1: per (request, cell) the minimum key over the GPUs, where a candidate's key is
//           its energy divided by the request's Lout, Pp * (TT / Lout) + Pd * TBT (Eq.
//           energy, Sec. 3.3).  The tile's GPU records are staged in LDS grouped by SM-cap
//           class (cap_pf, cap_dc); the prompt rows are staged already divided by Lout,
//           and per class the capped row values of the kQF requests and the power factors
//           s*f^3 sit in registers, so each GPU costs one record and one TBT read.  Per candidate: one FMA and half a v_min3 (GPUs taken in pairs).
//           Cells above max(cap_pf, cap_dc) repeat that level's cell exactly (same
//           latencies, same power) at a higher index, so they get NaN power and never
//           compete.  A wavefront with a request whose Lout is below 1 (or a prompt
//           latency far outside the float range that division keeps normal) keeps TT and
//           evaluates the energy itself: one multiply and one FMA per candidate.
//   pass 2: K* = the wavefront minimum; for each cell whose minimum equals K*, the lowest
//           GPU id whose key -- recomputed with the same operations, hence bit-identical
//           -- equals K*; the smallest index (g * 128 + cell) wins.  That is the
//           (key, index) lexicographic minimum, and the energy is Lout * K*.
// Masked (SLO-missing) latencies are NaN, which min ignores and == never matches.
constexpr int kQF = 8;
constexpr int kC = 128;
constexpr int kXcds = 8;                         // MI355X: 8 XCDs, each with its own L2
constexpr int kNS8 = 8;
constexpr int kClasses = kNS8 * kNS8;            // (cap_pf, cap_dc) pairs
constexpr int kHcap = 256;                       // host records staged in LDS per chunk
constexpr int kWblkB = (1 + kQF) * kC * 4;       // per wave: s*f^3 row + kQF prompt rows
// Decode-table rows are padded to 130 floats in LDS: row r starts at bank 2r, so pass-2
// reads of one cell from many rows hit distinct banks, and rows stay 8-byte aligned.
constexpr int kRowB = 130 * 4;

__host__ __device__ constexpr int fast_rec_off(int wpb) { return wpb * kWblkB; }
__host__ __device__ constexpr int fast_dcs_off(int wpb) { return wpb * kWblkB + kHcap * 16; }
__host__ __device__ constexpr size_t fast_lds_bytes(int wpb) {
  return (size_t)fast_dcs_off(wpb) + (size_t)kRows * kRowB;
}

typedef float v2f __attribute__((ext_vector_type(2)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v2f lds2(const char *base, uint32_t off) {
  return *reinterpret_cast<const v2f *>(base + off);
}
__device__ __forceinline__ float lds1(const char *base, uint32_t off) {
  return *reinterpret_cast<const float *>(base + off);
}

// v_min_f32 / v_min3_f32 as single instructions.  Operands are results of arithmetic or
// +inf, and a quiet-NaN operand yields the other operands, which is the masking rule;
// fminf would make the compiler add a canonicalising v_max_f32 per operand in IEEE mode.
__device__ __forceinline__ float vmin(float x, float y) {
  float r;
  asm("v_min_f32 %0, %1, %2" : "=v"(r) : "v"(x), "v"(y));
  return r;
}
__device__ __forceinline__ float vmin3(float x, float y, float z) {
  float r;
  asm("v_min3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "v"(y), "v"(z));
  return r;
}

// Energy of one candidate.  Pass 1 and pass 2 both evaluate exactly these operations.
__device__ __forceinline__ float cell_energy(float kap, float pdp, float pdd, float tbt, float tt,
                                            float p0, float lo, float slo_tbt) {
  const float Pp = fmaf(kap, pdp, p0);
  const float Pd = fmaf(kap, pdd, p0);
  const float Ym = tbt < slo_tbt ? Pd * tbt : kMask;
  return fmaf(lo, Ym, Pp * tt);
}

// The same candidate's energy divided by Lout (Lout >= 1): the key Pp * (TT / Lout) + Pd * TBT,
// one FMA once TT / Lout is staged.  Lout is one positive scale per request, so the
// request's keys are ordered as its energies (up to rounding), and its energy is Lout times
// its least key.  Pass 1 and pass 2 both evaluate exactly these operations.
__device__ __forceinline__ float cell_key(float kap, float pdp, float pdd, float tbt, float ttl, float p0,
                                         float slo_tbt) {
  const float Pp = fmaf(kap, pdp, p0);
  const float Pd = fmaf(kap, pdd, p0);
  const float Ym = tbt < slo_tbt ? Pd * tbt : kMask;
  return fmaf(Pp, ttl, Ym);
}

// A prompt latency x scaled to s = x / Lout keeps its precision: s is NaN, infinite or
// normal, or zero because x is.  (Class mask: signaling and quiet NaN, +-infinity,
// +-normal.)
__device__ __forceinline__ bool scaled_ok(float s, float x) {
  return __builtin_amdgcn_classf(s, 0x30f) | (x == 0.f);
}

// TBT-SLO handling of pass 1:
//   kPremasked  every live request of the tile has the same TBT SLO and the staged decode
//               table already holds NaN where TBT misses it;
//   kWaveSame   the wavefront's live requests share one TBT SLO: one test per (GPU, cell);
//   kMixed      one test per (request, GPU, cell).
enum { kPremasked = 0, kWaveSame = 1, kMixed = 2 };

// Per-class registers of one wavefront: capped prompt-row values of its requests, the
// power factors, and the decode-cell offset.
struct ClassRegs {
  v2f tt[kQF];
  v2f pdp, pdd;
  uint32_t mD;
};

template <int MODE>
__device__ __forceinline__ void host_terms(const char *L, v4u r, const ClassRegs &cr, float p0, float sb0,
                                           float (&Pp)[2], float (&Y)[2], float (&tbt)[2]) {
  const float kap = __uint_as_float(r.y);
  const v2f t = lds2(L, r.x + cr.mD);
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    Pp[c] = fmaf(kap, cr.pdp[c], p0);
    const float Pd = fmaf(kap, cr.pdd[c], p0);
    tbt[c] = t[c];
    Y[c] = MODE == kWaveSame ? (t[c] < sb0 ? Pd * t[c] : kMask) : Pd * t[c];
  }
}

// Pass 1 over the records [cs, ce) of one class.  NORM: the staged prompt rows hold TT / Lout
// and a candidate costs one FMA (its key); otherwise they hold TT and the candidate is its
// energy.
template <int MODE, bool NORM>
__device__ __forceinline__ void class_pass1(const char *L, uint32_t recB, int cs, int ce, const ClassRegs &cr,
                                            float p0, const float (&lo)[kQF], const float (&sb)[kQF],
                                            float sb0, float (&mn)[kQF][2]) {
  int i = cs;
  for (; i + 1 < ce; i += 2) {
    const v4u r0 = *reinterpret_cast<const v4u *>(L + recB + i * 16);
    const v4u r1 = *reinterpret_cast<const v4u *>(L + recB + (i + 1) * 16);
    float Pp0[2], Y0[2], T0[2], Pp1[2], Y1[2], T1[2];
    host_terms<MODE>(L, r0, cr, p0, sb0, Pp0, Y0, T0);
    host_terms<MODE>(L, r1, cr, p0, sb0, Pp1, Y1, T1);
#pragma unroll
    for (int q = 0; q < kQF; ++q)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const float y0 = MODE == kMixed ? (T0[c] < sb[q] ? Y0[c] : kMask) : Y0[c];
        const float y1 = MODE == kMixed ? (T1[c] < sb[q] ? Y1[c] : kMask) : Y1[c];
        if (NORM)
          mn[q][c] = vmin3(mn[q][c], fmaf(Pp0[c], cr.tt[q][c], y0), fmaf(Pp1[c], cr.tt[q][c], y1));
        else
          mn[q][c] = vmin3(mn[q][c], fmaf(lo[q], y0, Pp0[c] * cr.tt[q][c]), fmaf(lo[q], y1, Pp1[c] * cr.tt[q][c]));
      }
  }
  if (i < ce) {
    const v4u r0 = *reinterpret_cast<const v4u *>(L + recB + i * 16);
    float Pp0[2], Y0[2], T0[2];
    host_terms<MODE>(L, r0, cr, p0, sb0, Pp0, Y0, T0);
#pragma unroll
    for (int q = 0; q < kQF; ++q)
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const float y0 = MODE == kMixed ? (T0[c] < sb[q] ? Y0[c] : kMask) : Y0[c];
        mn[q][c] = vmin(mn[q][c], NORM ? fmaf(Pp0[c], cr.tt[q][c], y0) : fmaf(lo[q], y0, Pp0[c] * cr.tt[q][c]));
      }
  }
}

// SM-cap classes are numbered so that ascending number means ascending
// m = max(cap_pf, cap_dc): the 2m + 1 classes of m take the numbers m^2 .. (m + 1)^2 - 1.
__device__ __forceinline__ int class_id(int p, int d) {
  const int m = max(p, d);
  return m * m + (p == m ? d : m + 1 + p);
}
// The inverse, as cap_pf * 8 + cap_dc.
__device__ __forceinline__ int class_caps(int t) {
  int m = 0;
#pragma unroll
  for (int k = 1; k < kNS8; ++k) m += t >= k * k;
  const int r = t - m * m;
  return r <= m ? m * kNS8 + r : (r - m - 1) * kNS8 + m;
}

// Per-class registers for the SM level at byte offset je64 of this lane; a level above
// max(cap_pf, cap_dc) only repeats the class's top level, so its power is NaN.
__device__ __forceinline__ ClassRegs class_regs(const char *L, uint32_t wblkB, uint32_t je64, uint32_t k04,
                                                uint32_t cpB, uint32_t cdB) {
  ClassRegs cr;
  const uint32_t aP = wblkB + min(je64, cpB) + k04;
  cr.mD = min(je64, cdB) + k04;
  cr.pdp = lds2(L, aP);
  cr.pdd = lds2(L, wblkB + cr.mD);
  if (je64 > max(cpB, cdB)) cr.pdp = v2f{kMask, kMask};
#pragma unroll
  for (int q = 0; q < kQF; ++q) cr.tt[q] = lds2(L, aP + (1 + q) * kC * 4);
  return cr;
}

// Pass 1 over one class in the common mode (premasked TBT, keys), H GPUs per step: H = 1
// is the plain layout; H = 2 or 4 packs a class whose SM levels above m = max(cap_pf,
// cap_dc) only repeat level m, with 8 / H levels per GPU (a power of two >= m + 1), so
// lane l works on GPU (step start + slot), slot = (l / 8) / (8 / H), at SM level
// (l / 8) % (8 / H).  The partial minima of one cell then sit in the lanes that share its
// level until fold_levels gathers them.  A lane past the class's last GPU reads that GPU's
// record with NaN power (with H = 1 every step's GPU exists and no lane needs the clamp).
template <int H>
__device__ __forceinline__ void class_pass1_common(const char *L, uint32_t recB, int cs, int ce,
                                                   const ClassRegs &cr, float p0, int slot,
                                                   float (&mn)[kQF][2]) {
  constexpr bool ONE = H == 1;
  if (ONE) slot = 0;
  int i = cs;
  for (; i + H < ce; i += 2 * H) {
    const int h1 = i + H + slot;
    const v4u r0 = *reinterpret_cast<const v4u *>(L + recB + (i + slot) * 16);
    v4u r1 = *reinterpret_cast<const v4u *>(L + recB + (ONE ? h1 : min(h1, ce - 1)) * 16);
    if (!ONE) r1.y = h1 < ce ? r1.y : __float_as_uint(kMask);
    float Pp0[2], Y0[2], T0[2], Pp1[2], Y1[2], T1[2];
    host_terms<kPremasked>(L, r0, cr, p0, 0.f, Pp0, Y0, T0);
    host_terms<kPremasked>(L, r1, cr, p0, 0.f, Pp1, Y1, T1);
#pragma unroll
    for (int q = 0; q < kQF; ++q)
#pragma unroll
      for (int c = 0; c < 2; ++c)
        mn[q][c] = vmin3(mn[q][c], fmaf(Pp0[c], cr.tt[q][c], Y0[c]), fmaf(Pp1[c], cr.tt[q][c], Y1[c]));
  }
  if (i < ce) {
    const int h0 = i + slot;
    v4u r0 = *reinterpret_cast<const v4u *>(L + recB + (ONE ? h0 : min(h0, ce - 1)) * 16);
    if (!ONE) r0.y = h0 < ce ? r0.y : __float_as_uint(kMask);
    float Pp0[2], Y0[2], T0[2];
    host_terms<kPremasked>(L, r0, cr, p0, 0.f, Pp0, Y0, T0);
#pragma unroll
    for (int q = 0; q < kQF; ++q)
#pragma unroll
      for (int c = 0; c < 2; ++c) mn[q][c] = vmin(mn[q][c], fmaf(Pp0[c], cr.tt[q][c], Y0[c]));
  }
}

// Gathers packed partial minima: lanes whose SM levels agree modulo NLP combine (xor 16
// and xor 32 over the lane index for NLP = 2, xor 32 for NLP = 4), lanes at levels below
// NLP keep the result, and the others restart from +inf for the classes still to come.
template <int NLP>
__device__ __forceinline__ void fold_levels(float (&mn)[kQF][2], int j) {
#pragma unroll
  for (int q = 0; q < kQF; ++q)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      float v = mn[q][c];
      if (NLP <= 2) {
        const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
        v = vmin(__uint_as_float(r[0]), __uint_as_float(r[1]));
      }
      const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
      v = vmin(__uint_as_float(r[0]), __uint_as_float(r[1]));
      mn[q][c] = j < NLP ? v : kInf;
    }
}

// Pass 1 over the class list of one chunk, every class in the plain layout.
template <int MODE, bool NORM>
__device__ __forceinline__ void pass1_classes(const char *L, uint32_t recB, uint32_t wblkB, const int *clist,
                                              int ncls, uint32_t j64, uint32_t k04, float p0,
                                              const float (&lo)[kQF], const float (&sb)[kQF], float sb0,
                                              float (&mn)[kQF][2]) {
  for (int k = 0; k < ncls; ++k) {
    const int packed = uniform(clist[k]);
    const int cls = packed & 63, cs = (packed >> 6) & 511, ce = (packed >> 15) & 511;
    const ClassRegs cr = class_regs(L, wblkB, j64, k04, (uint32_t)(cls / kNS8) * 64u, (uint32_t)(cls % kNS8) * 64u);
    class_pass1<MODE, NORM>(L, recB, cs, ce, cr, p0, lo, sb, sb0, mn);
  }
}

// Pass 1 over the classes [k, ncls) of one chunk in the common mode that have 8 / H levels per
// GPU, H GPUs per step; returns the first class with more levels.
template <int H>
__device__ __forceinline__ int pass1_group(const char *L, uint32_t recB, uint32_t wblkB, const int *clist, int k,
                                           int ncls, bool pk, int j, uint32_t k04, float p0, float (&mn)[kQF][2]) {
  constexpr int lg = H == 4 ? 1 : H == 2 ? 2 : 3;   // log2 of the levels per GPU
  for (; k < ncls; ++k) {
    const int packed = uniform(clist[k]);
    const int cls = packed & 63, cs = (packed >> 6) & 511, ce = (packed >> 15) & 511;
    const int mc = max(cls / kNS8, cls % kNS8);
    if (H > 1 && (!pk || (mc < 2 ? 1 : mc < 4 ? 2 : 3) != lg)) break;
    const ClassRegs cr = class_regs(L, wblkB, (uint32_t)(j & ((1 << lg) - 1)) * 64u, k04,
                                    (uint32_t)(cls / kNS8) * 64u, (uint32_t)(cls % kNS8) * 64u);
    class_pass1_common<H>(L, recB, cs, ce, cr, p0, j >> lg, mn);
  }
  return k;
}

// Pass 1 over the class list of one chunk in the common mode.  With pk (the tile's GPUs fit
// one chunk) capped classes are packed.  Classes come in ascending max cap m, so they form
// three groups in order, each run by a loop of its own: m <= 1 (2 levels, 4 GPUs per step),
// m = 2 or 3 (4 levels, 2 GPUs per step), each folded into the plain layout when it ends, and
// m >= 4 (one GPU per step; every class without pk).
__device__ __forceinline__ void pass1_common(const char *L, uint32_t recB, uint32_t wblkB, const int *clist,
                                             int ncls, bool pk, int j, uint32_t k04, float p0,
                                             float (&mn)[kQF][2]) {
  int k = 0;
  if (pk) {
    const int k1 = pass1_group<4>(L, recB, wblkB, clist, 0, ncls, pk, j, k04, p0, mn);
    if (k1 > 0) fold_levels<2>(mn, j);
    const int k2 = pass1_group<2>(L, recB, wblkB, clist, k1, ncls, pk, j, k04, p0, mn);
    if (k2 > k1) fold_levels<4>(mn, j);
    k = k2;
  }
  pass1_group<1>(L, recB, wblkB, clist, k, ncls, pk, j, k04, p0, mn);
}

// DPP lane moves within rows of 16 lanes (every source lane exists).
constexpr int kDppRor8 = 0x128;        // row_ror:8: lane i reads lane i ^ 8 of its row
constexpr int kDppHalfMirror = 0x141;  // lane i reads lane 7 - i of its group of 8
constexpr int kDppQuad2301 = 0x4E;     // lane i reads lane i ^ 2 of its quad
constexpr int kDppQuad1032 = 0xB1;     // lane i reads lane i ^ 1 of its quad

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}

// est[q] = min over the wavefront's lanes of min(m[q][0], m[q][1]), for the kQF = 8
// requests at once, as a transposing reduction: each exchange halves the values a lane
// holds (xor 32 and xor 16 by permlane swaps, xor 8 by DPP) until lane l holds request
// l / 8's partial minimum, then three DPP steps reduce each group of 8 lanes.  Returns
// est[l / 8] in lane l.
__device__ __forceinline__ float wave_min8(const float (&m)[kQF][2], float (&est)[kQF]) {
  static_assert(kQF == 8, "the exchange pattern is written for 8 requests per wavefront");
  float v[8], u[4], w[2];
#pragma unroll
  for (int q = 0; q < 8; ++q) v[q] = vmin(m[q][0], m[q][1]);
  // lanes 0-31 keep requests 0-3, lanes 32-63 requests 4-7
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[p]), __float_as_uint(v[p + 4]), false, false);
    u[p] = vmin(__uint_as_float(r[0]), __uint_as_float(r[1]));
  }
  // even rows of 16 lanes keep the first two of their half's four, odd rows the last two
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(u[p]), __float_as_uint(u[p + 2]), false, false);
    w[p] = vmin(__uint_as_float(r[0]), __uint_as_float(r[1]));
  }
  // lanes with bit 3 clear keep the first of the two, the others the second
  const bool hi = (__lane_id() & 8) != 0;
  float c = vmin(hi ? w[1] : w[0], dpp<kDppRor8>(hi ? w[0] : w[1]));
  c = vmin(c, dpp<kDppHalfMirror>(c));
  c = vmin(c, dpp<kDppQuad2301>(c));
  c = vmin(c, dpp<kDppQuad1032>(c));
#pragma unroll
  for (int q = 0; q < 8; ++q) est[q] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(c), 8 * q));
  return c;
}

// One pass-2 round: for each request q with cell[q] >= 0, the lowest GPU id whose candidate at
// that cell reaches the request's minimum est[q], recomputed with the operations of pass 1
// (hence bit-identical); best[q] = min(best[q], g * 128 + cell).  Lane l takes host b0 + l of
// the model's ascending host list, reads its record once and evaluates every request's
// cell; the first set lane of a request's match mask is its lowest GPU id, so a request
// stops at the first block of 64 hosts with a match.
template <bool NRM>
__device__ __forceinline__ void pass2_round(const PlaceArgs &a, const char *L, uint32_t recB, uint32_t dcsB,
                                            uint32_t wblkB, const short *s_pos, const int32_t *hl, const HostRec *rw,
                                            bool recs_in_lds, int hcnt, float p0, const int (&cell)[kQF],
                                            const float (&est)[kQF], const float (&lo)[kQF], const float (&sb)[kQF],
                                            int (&best)[kQF]) {
  const int lane = __lane_id();
  uint32_t cj64[kQF], ck4[kQF], base[kQF];
  unsigned pending = 0;
#pragma unroll
  for (int q = 0; q < kQF; ++q) {
    const int c = cell[q] >= 0 ? cell[q] : 0;
    cj64[q] = (uint32_t)(c >> 4) * 64u;
    ck4[q] = (uint32_t)(c & 15) * 4u;
    base[q] = wblkB + ck4[q];
    pending |= cell[q] >= 0 ? 1u << q : 0u;
  }
  for (int b0 = 0; b0 < hcnt && pending != 0u; b0 += kWave) {
    const int i = b0 + lane;
    const bool valid = i < hcnt;
    const int ic = valid ? i : hcnt - 1;
    uint32_t rowB;
    int g, caps;
    float kap;
    if (recs_in_lds) {                    // host i (ascending GPU id) sits at slot s_pos[i]
      const v4u r = *reinterpret_cast<const v4u *>(L + recB + (int)s_pos[ic] * 16);
      rowB = r.x;
      kap = __uint_as_float(r.y);
      g = (int)r.z;
      caps = (int)r.w;
    } else {
      g = hl[ic];
      const HostRec r = rw[g];
      rowB = dcsB + (uint32_t)(max(r.row_off, 0) / kC) * kRowB;
      kap = r.kappa;
      caps = r.caps;
    }
    const uint32_t cpB = (uint32_t)(caps & 0xff) * 64u, cdB = (uint32_t)((caps >> 8) & 0xff) * 64u;
    const uint32_t mxB = max(cpB, cdB);
#pragma unroll
    for (int q = 0; q < kQF; ++q) {
      // a cell above max(cap_pf, cap_dc) repeats a lower cell of the same GPU: pass 1 gave it
      // NaN power, so it never matches
      const uint32_t jP = min(cj64[q], cpB), jD = min(cj64[q], cdB);
      const uint32_t aP = base[q] + jP, aD = base[q] + jD;
      const float pdp = lds1(L, aP), pdd = lds1(L, aD);
      const float tbt = lds1(L, rowB + jD + ck4[q]);
      const float tt = lds1(L, aP + (1 + q) * kC * 4);
      const float E = NRM ? cell_key(kap, pdp, pdd, tbt, tt, p0, sb[q])
                          : cell_energy(kap, pdp, pdd, tbt, tt, p0, lo[q], sb[q]);
      const bool hit = (E == est[q]) & valid & (cj64[q] <= mxB);
      const unsigned long long m = __ballot(hit);
      if (((pending >> q) & 1u) && m != 0ull) {
        const int gw = __builtin_amdgcn_readlane(g, __builtin_ctzll(m));
        best[q] = min(best[q], gw * kC + cell[q]);
        pending &= ~(1u << q);
      }
    }
  }
}

template <int WPB>
__global__ void __launch_bounds__(WPB * 64) k_score_c128(PlaceArgs a) {
  extern __shared__ __align__(16) float lds[];
  __shared__ int s_live[WPB], s_same[WPB], s_sb[WPB];
  __shared__ int s_cls[kClasses + 1];     // class counts, then class starts
  __shared__ int s_clist[kClasses + 1];   // non-empty classes: cls | start << 6 | end << 15; [64] = count
  __shared__ short s_pos[kHcap];          // slot of host i's record after the class sort
  char *L = reinterpret_cast<char *>(lds);
  constexpr uint32_t recB = fast_rec_off(WPB);
  constexpr uint32_t dcsB = fast_dcs_off(WPB);
  constexpr int T = WPB * 64;
  // XCD-aware tile order: workgroups are dealt to the 8 XCDs round-robin, so XCD x takes
  // the contiguous tile range [x * per, (x + 1) * per) -- the same arrival waves and GPU
  // records -- instead of every eighth tile.  per = ceil(n_tiles / 8) <= grid / 8.
  const int ntiles = *ro(a.n_tiles);
  const int per = (ntiles + kXcds - 1) / kXcds;
  const int idx = blockIdx.x / kXcds;
  const int t = (blockIdx.x % kXcds) * per + idx;
  if (idx >= per || t >= ntiles) return;
  const auto tp = ro(reinterpret_cast<const int32_t *>(a.tiles));
  const int bucket = tp[2 * t];
  if (bucket & 1) {                       // prompt-less requests: TTFT from the batch row
    score_tile_generic<2>(a, t, lds);
    return;
  }
  const int wm = bucket >> 1;
  const int w = wm / a.M, m = wm - (wm / a.M) * a.M;
  const int beg = tp[2 * t + 1];
  const int end = min(beg + a.tile, ro(a.bstart)[bucket + 1]);

  // Staging and the class sort wait on memory and barriers while other workgroups' pass 1
  // keeps the VALU busy: at a raised wavefront priority their instructions issue first, and
  // pass 1 runs at the normal priority.
  __builtin_amdgcn_s_setprio(2);
  const int wv = uniform(threadIdx.x >> 6);
  const int lane = threadIdx.x & (kWave - 1);
  const uint32_t wblkB = (uint32_t)wv * kWblkB;
  const int j = lane >> 3;
  const uint32_t j64 = (uint32_t)j * 64u;          // byte offset of SM level j in a row
  const uint32_t k04 = (uint32_t)(lane & 7) * 8u;  // byte offset of frequency level 2 * (lane % 8)
  {
    v2f pd;
    pd.x = a.sm_level[j] * cube(a.freq_level[2 * (lane & 7)]);
    pd.y = a.sm_level[j] * cube(a.freq_level[2 * (lane & 7) + 1]);
    *reinterpret_cast<v2f *>(L + wblkB + j64 + k04) = pd;
  }

  // this wavefront's requests and their prompt rows
  const int q0 = beg + wv * kQF;
  const int nq = max(0, min(kQF, end - q0));
  // Lane l stages 16 cells of request l / 8's prompt row and keeps that request's fields;
  // a missing request reads the tile's first record and row 0 and is masked.  Rows: NaN
  // where TTFT misses the SLO, scaled by 1 / Lout when every request of the wavefront has a
  // usable reciprocal and every scaled value stays normal (or NaN), or is zero because the
  // latency is.
  const int sq = lane >> 3;
  const bool shas = sq < nq;
  bool nrm;
  unsigned long long livem;
  const ReqRec myr = load_req_lane(a, shas ? q0 + sq : beg);
  const int r_l = shas ? myr.r : -1;
  const float lo_l = shas ? myr.lout : 0.f;
  const float sb_l = shas ? myr.slo_tbt : -kInf;
  {
    const float st = shas ? myr.slo_ttft : -kInf;
    const float rl = shas ? myr.rlout : 1.f;
    // lane l takes the 16-byte chunks l % 8 + 8u (u < 4) of the row, so each load and each
    // store of a request's 8 lanes covers 128 contiguous bytes
    const float *pr = a.pf + ((size_t)m * kRows + (shas ? myr.row : 0)) * kC;
    const int x8 = lane & 7;
    float v[16];
    if ((reinterpret_cast<uintptr_t>(a.pf) & 15) == 0) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float4 x = reinterpret_cast<const float4 *>(pr)[8 * u + x8];
        v[4 * u] = x.x;
        v[4 * u + 1] = x.y;
        v[4 * u + 2] = x.z;
        v[4 * u + 3] = x.w;
      }
    } else {
#pragma unroll
      for (int u = 0; u < 16; ++u) v[u] = pr[(8 * (u >> 2) + x8) * 4 + (u & 3)];
    }
    bool ok = rl > 0.f, any = false;
    float sc[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      v[u] = v[u] < st ? v[u] : kMask;
      sc[u] = v[u] * rl;
      ok = ok & scaled_ok(sc[u], v[u]);
      any = any | (v[u] == v[u]);
    }
    nrm = __ballot(!ok) == 0ull;
    float4 *d = reinterpret_cast<float4 *>(L + wblkB + (1 + sq) * kC * 4);
#pragma unroll
    for (int u = 0; u < 4; ++u)
      d[8 * u + x8] = nrm ? make_float4(sc[4 * u], sc[4 * u + 1], sc[4 * u + 2], sc[4 * u + 3])
                 : make_float4(v[4 * u], v[4 * u + 1], v[4 * u + 2], v[4 * u + 3]);
    livem = __ballot(any);
  }
  // per-request uniform values: Lout and the TBT SLO from lane 8q
  float lo[kQF], sb[kQF];
#pragma unroll
  for (int q = 0; q < kQF; ++q) {
    lo[q] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lo_l), 8 * q));
    sb[q] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sb_l), 8 * q));
  }
  // a request whose whole row is NaN is dead: infeasible whatever the TBT test says, so it
  // takes no part in the TBT-SLO uniformity checks
  bool live_any = false, wsame = true;
  float sb0 = 0.f;
#pragma unroll
  for (int q = 0; q < kQF; ++q) {
    if ((livem >> (8 * q)) & 0xffull) {
      if (!live_any) sb0 = sb[q];
      wsame = wsame && __float_as_int(sb[q]) == __float_as_int(sb0);
      live_any = true;
    }
  }
  if (lane == 0) {
    s_live[wv] = live_any;
    s_same[wv] = wsame;
    s_sb[wv] = __float_as_int(sb0);
  }
  __syncthreads();
  bool tile_live = false, tile_same = true;
  int tile_sb = 0;
  for (int v = 0; v < WPB; ++v) {
    if (!s_live[v]) continue;
    if (!tile_live) tile_sb = s_sb[v];
    tile_same = tile_same && s_same[v] && s_sb[v] == tile_sb;
    tile_live = true;
  }
  const float tsb = __int_as_float(tile_sb);

  {  // the model's decode table, rows padded to kRowB bytes; NaN where TBT misses the
     // tile's common TBT SLO
    const float *src = a.dc + (size_t)m * kRows * kC;
    if ((((uintptr_t)src) & 15) == 0) {
      const float4 *s4 = reinterpret_cast<const float4 *>(src);
      for (int i = threadIdx.x; i < kRows * kC / 4; i += T) {
        float4 v = s4[i];
        if (tile_same) {
          v.x = v.x < tsb ? v.x : kMask;
          v.y = v.y < tsb ? v.y : kMask;
          v.z = v.z < tsb ? v.z : kMask;
          v.w = v.w < tsb ? v.w : kMask;
        }
        v2f *d = reinterpret_cast<v2f *>(L + dcsB + (i >> 5) * kRowB + (i & 31) * 16);
        d[0] = v2f{v.x, v.y};
        d[1] = v2f{v.z, v.w};
      }
    } else {
      for (int i = threadIdx.x; i < kRows * kC; i += T) {
        float v = src[i];
        if (tile_same) v = v < tsb ? v : kMask;
        *reinterpret_cast<float *>(L + dcsB + (i >> 7) * kRowB + (i & 127) * 4) = v;
      }
    }
  }

  float mn[kQF][2];
#pragma unroll
  for (int q = 0; q < kQF; ++q) mn[q][0] = mn[q][1] = kInf;

  const int hcnt = tile_live ? ro(a.host_cnt)[m] : 0;   // a tile of dead requests scores nothing
  const int32_t *hl = a.host_list + (size_t)m * a.G;
  const HostRec *rw = a.recs + (size_t)w * a.G;
  const float p0 = a.p0;
  constexpr int kPer = kHcap / T > 0 ? kHcap / T : 1;  // host records per thread per chunk
  for (int c0 = 0; c0 < hcnt; c0 += kHcap) {
    const int n = min(kHcap, hcnt - c0);
    __syncthreads();                      // previous records no longer in use; table staged
    __builtin_amdgcn_s_setprio(2);          // the next chunk's class sort
    for (int i = threadIdx.x; i < kClasses; i += T) s_cls[i] = 0;
    __syncthreads();
    // records of this chunk, grouped by (cap_pf, cap_dc) class with an LDS counting sort,
    // classes in ascending max(cap_pf, cap_dc)
    v4u rec[kPer];
    int key[kPer], rank[kPer];
#pragma unroll
    for (int u = 0; u < kPer; ++u) {
      const int i = u * T + threadIdx.x;
      key[u] = -1;
      if (i < n) {
        const int g = hl[c0 + i];
        const HostRec r = rw[g];
        rec[u].x = dcsB + (uint32_t)(max(r.row_off, 0) / kC) * kRowB;
        rec[u].y = __float_as_uint(r.kappa);
        rec[u].z = (uint32_t)g;
        rec[u].w = (uint32_t)r.caps;
        key[u] = class_id(r.caps & 0xff, (r.caps >> 8) & 0xff);
        rank[u] = atomicAdd(&s_cls[key[u]], 1);
      }
    }
    __syncthreads();
    if (threadIdx.x < kWave) {            // exclusive prefix over the 64 classes, and the
      const int cnt = s_cls[threadIdx.x];  // compact list of the non-empty ones
      const int inc = wave_scan(cnt);
      s_cls[threadIdx.x] = inc - cnt;
      const unsigned long long ne = __ballot(cnt > 0);
      const int pos = __popcll(ne & ((1ull << threadIdx.x) - 1ull));
      if (cnt > 0) s_clist[pos] = class_caps(threadIdx.x) | ((inc - cnt) << 6) | (inc << 15);
      if (threadIdx.x == kWave - 1) {
        s_cls[kClasses] = inc;
        s_clist[kClasses] = __popcll(ne);
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kPer; ++u)
      if (key[u] >= 0) {
        const int pos = s_cls[key[u]] + rank[u];
        *reinterpret_cast<v4u *>(L + recB + pos * 16) = rec[u];
        s_pos[u * T + threadIdx.x] = (short)pos;
      }
    __syncthreads();
    __builtin_amdgcn_s_setprio(0);
    if (live_any) {
      const int ncls = uniform(s_clist[kClasses]);
      if (tile_same && nrm)
        pass1_common(L, recB, wblkB, s_clist, ncls, hcnt <= kHcap, j, k04, p0, mn);
      else if (nrm && wsame)
        pass1_classes<kWaveSame, true>(L, recB, wblkB, s_clist, ncls, j64, k04, p0, lo, sb, sb0, mn);
      else if (nrm)
        pass1_classes<kMixed, true>(L, recB, wblkB, s_clist, ncls, j64, k04, p0, lo, sb, sb0, mn);
      else if (tile_same)
        pass1_classes<kPremasked, false>(L, recB, wblkB, s_clist, ncls, j64, k04, p0, lo, sb, sb0, mn);
      else if (wsame)
        pass1_classes<kWaveSame, false>(L, recB, wblkB, s_clist, ncls, j64, k04, p0, lo, sb, sb0, mn);
      else
        pass1_classes<kMixed, false>(L, recB, wblkB, s_clist, ncls, j64, k04, p0, lo, sb, sb0, mn);
    }
  }

  // pass 2: per request the winning energy E* (key K*: E* = Lout * K*), then the lowest index
  // that reaches it.  One round per tied cell of a request (one round unless two different
  // cells reach exactly E*); in a round every lane takes one host, in ascending GPU id.
  const bool recs_in_lds = hcnt <= kHcap;
  float est[kQF];
  unsigned long long t0[kQF], t1[kQF];
  bool rounds = false;
  const float cmin = wave_min8(mn, est);   // request sq's minimum
#pragma unroll
  for (int q = 0; q < kQF; ++q) {
    const bool feas = q < nq && (nrm ? lo[q] * est[q] : est[q]) < kInf;
    t0[q] = __ballot(feas && mn[q][0] == est[q]);
    t1[q] = __ballot(feas && mn[q][1] == est[q]);
    rounds = rounds || (t0[q] | t1[q]) != 0ull;
  }
  int best[kQF];                          // lowest index reaching E*, per request
#pragma unroll
  for (int q = 0; q < kQF; ++q) best[q] = INT_MAX;
  while (rounds) {
    rounds = false;
    int cell[kQF];                        // next tied cell of each request, ascending; -1: none
#pragma unroll
    for (int q = 0; q < kQF; ++q) {
      cell[q] = -1;
      if ((t0[q] | t1[q]) != 0ull) {
        const int l0 = t0[q] ? __builtin_ctzll(t0[q]) : 64;
        const int l1 = t1[q] ? __builtin_ctzll(t1[q]) : 64;
        cell[q] = l0 <= l1 ? 2 * l0 : 2 * l1 + 1;
        if (l0 <= l1)
          t0[q] &= t0[q] - 1ull;
        else
          t1[q] &= t1[q] - 1ull;
      }
      rounds = rounds || (t0[q] | t1[q]) != 0ull;
    }
    if (nrm)
      pass2_round<true>(a, L, recB, dcsB, wblkB, s_pos, hl, rw, recs_in_lds, hcnt, p0, cell, est, lo, sb, best);
    else
      pass2_round<false>(a, L, recB, dcsB, wblkB, s_pos, hl, rw, recs_in_lds, hcnt, p0, cell, est, lo, sb, best);
  }
  // lane 8q writes request q: its record and minimum sit in lanes l / 8 = q
  int myb = best[0];
#pragma unroll
  for (int q = 1; q < kQF; ++q) myb = sq == q ? best[q] : myb;
  if ((lane & 7) == 0 && shas) {
    const bool found = myb != INT_MAX;
    a.choice[r_l] = found ? myb : -1;
    a.feasible[r_l] = found ? 1 : 0;
    a.energy[r_l] = found ? (nrm ? lo_l * cmin : cmin) : kInf;
  }
}

// ------------------------------------------------------------------ migration kernels
struct MigArgs {
  int32_t M, NS, NF, C;
  const float *freq_level, *pf, *dc;
  float p0;
  int32_t G, K;
  const int32_t *n_inst, *inst_model, *inst_prompt, *inst_batch, *inst_sm;
  const float *inst_slo_ttft, *inst_slo_tbt;
  const int32_t *hbm, *smpm;
  const float *util, *kdyn;
  int32_t hbm_cap, sm_cap;
  int32_t *best_dst;
  float *saving;
  int32_t *level;
  v4i *drec;                     // [G][2] destination records from k_fleet:
                                 // {hbm, SM per-mille, level mask, k_d}, {u, f[kd0]^3 * u, 0, 0}
};

// One wavefront per GPU: lane k tests frequency level k (NF <= 32) for each instance, a
// ballot turns the tests into that instance's level mask, and the GPU's mask is the AND.
// With at most kFleetUnroll instances per GPU every instance's fields, then every table
// value, are requested before the first is used (two memory round trips per GPU).
constexpr int kFleetUnroll = 4;

__device__ __forceinline__ bool inst_ok(int m, int j, int B, int pt, const MigArgs &a) {
  return m >= 0 && m < a.M && j >= 0 && j < a.NS && B >= 0 && pt >= 0;
}

// Level mask of instance (m, j, B, pt) with SLOs (st, sb): lane k's test, as a ballot.
__device__ __forceinline__ uint32_t inst_mask(const MigArgs &a, int lane, int m, int j, int B, int pt, float st,
                                              float sb) {
  const int bb = B + 1 > kRows ? kRows : B + 1;
  const int prow = pt == 0 ? bb - 1 : (min((int)(((unsigned)pt + 255u) >> 8), kRows) - 1);
  const float *pr = a.pf + (((size_t)m * kRows + prow) * a.NS + j) * a.NF;
  const float *dr = a.dc + (((size_t)m * kRows + (bb - 1)) * a.NS + j) * a.NF;
  const int k = lane < a.NF ? lane : 0;
  const bool pass = lane < a.NF && pr[k] < st && dr[k] < sb;
  return (uint32_t)__ballot(pass);
}

__global__ void __launch_bounds__(256) k_fleet(MigArgs a) {
  const int g = blockIdx.x * 4 + uniform(threadIdx.x >> 6);
  const int lane = threadIdx.x & (kWave - 1);
  if (g >= a.G) return;
  const int n = ro(a.n_inst)[g];
  uint32_t fm = (n >= 1 && n <= a.K) ? (a.NF >= 32 ? 0xffffffffu : ((1u << a.NF) - 1u)) : 0u;
  if (a.K <= kFleetUnroll) {
    int m[kFleetUnroll], j[kFleetUnroll], B[kFleetUnroll], pt[kFleetUnroll];
    float st[kFleetUnroll], sb[kFleetUnroll];
#pragma unroll
    for (int i = 0; i < kFleetUnroll; ++i) {
      const size_t at = (size_t)g * a.K + (i < n ? i : 0);
      m[i] = ro(a.inst_model)[at];
      j[i] = ro(a.inst_sm)[at];
      B[i] = ro(a.inst_batch)[at];
      pt[i] = ro(a.inst_prompt)[at];
      st[i] = ro(a.inst_slo_ttft)[at];
      sb[i] = ro(a.inst_slo_tbt)[at];
    }
    // every instance's mask without an early exit (an AND that reached 0 stays 0), so that
    // no instance's table loads wait for another's ballot
#pragma unroll
    for (int i = 0; i < kFleetUnroll; ++i) {
      if (i >= n) continue;
      if (!inst_ok(m[i], j[i], B[i], pt[i], a)) {   // never read the tables at a bad index
        fm = 0;
        continue;
      }
      fm &= inst_mask(a, lane, m[i], j[i], B[i], pt[i], st[i], sb[i]);
    }
  } else {
    for (int i = 0; i < n && i < a.K && fm; ++i) {
      const size_t at = (size_t)g * a.K + i;
      const int m = ro(a.inst_model)[at], j = ro(a.inst_sm)[at], B = ro(a.inst_batch)[at];
      const int pt = ro(a.inst_prompt)[at];
      if (!inst_ok(m, j, B, pt, a)) {
        fm = 0;
        break;
      }
      fm &= inst_mask(a, lane, m, j, B, pt, ro(a.inst_slo_ttft)[at], ro(a.inst_slo_tbt)[at]);
    }
  }
  if (lane == 0) {
    const float u = a.util[g];
    const float base = fm ? cube(a.freq_level[__builtin_ctz(fm)]) * u : 0.f;
    a.drec[2 * g] = v4i{a.hbm[g], a.smpm[g], (int)fm, __float_as_int(a.kdyn[g])};
    a.drec[2 * g + 1] = v4i{__float_as_int(u), __float_as_int(base), 0, 0};
  }
}

constexpr int kMigSrcPerBlock = 2;   // sources per block; each source's destinations in 2 halves

// Best (largest saving, then lowest destination) of two candidates.
__device__ __forceinline__ void keep_best(float &v, int &d, int &k, float ov, int od, int ok) {
  if (ov > v || (ov == v && od < d)) {
    v = ov;
    d = od;
    k = ok;
  }
}

// Four wavefronts per block: wavefront w scores source blockIdx.x * 2 + w / 2 against the
// destinations of half w % 2, lanes spanning destinations, reading the 32-byte destination
// records straight from the cache (the whole fleet's records, 32 B per GPU, stay in L2).  The
// two halves' bests meet in LDS: largest saving, ties to the lowest destination.
__global__ void __launch_bounds__(256) k_migrate(MigArgs a) {
  __shared__ float f3[32];
  __shared__ float s_v[4];
  __shared__ int s_d[4], s_k[4];
  if (threadIdx.x < 32) f3[threadIdx.x] = threadIdx.x < a.NF ? cube(a.freq_level[threadIdx.x]) : 0.f;
  __syncthreads();
  const int lane = threadIdx.x & (kWave - 1);
  const int wv = uniform(threadIdx.x >> 6);
  const int src = blockIdx.x * kMigSrcPerBlock + (wv >> 1);
  const bool valid = src < a.G;
  const int s = valid ? src : 0;
  const long long rh = (long long)a.hbm_cap - a.hbm[s];
  const long long ru = (long long)a.sm_cap - a.smpm[s];
  const bool any = valid && rh >= (long long)INT_MIN && ru >= (long long)INT_MIN;
  const int remH = (int)(rh > INT_MAX ? INT_MAX : (rh < INT_MIN ? INT_MIN : rh));
  const int remU = (int)(ru > INT_MAX ? INT_MAX : (ru < INT_MIN ? INT_MIN : ru));
  const v4i sx = ro(a.drec)[2 * (size_t)s], sy = ro(a.drec)[2 * (size_t)s + 1];
  const uint32_t fms = any ? (uint32_t)sx.z : 0u;
  const float us = __int_as_float(sy.x);
  const int per = (a.G + 1) >> 1;
  const int lo = (wv & 1) * per, hi = min(a.G, lo + per);
  float bs = -kInf;
  int bd = INT_MAX, bk = -1;
  if (fms != 0u) {
#pragma unroll 4
    for (int d = lo + lane; d < hi; d += kWave) {
      const v4i r = a.drec[2 * (size_t)d], r2 = a.drec[2 * (size_t)d + 1];
      const uint32_t f = fms & (uint32_t)r.z;
      const bool ok = d != src && r.x <= remH && r.y <= remU && f != 0u;
      const int k = __builtin_ctz(f | 0x80000000u);
      const float added = f3[k] * (us + __int_as_float(r2.x)) - __int_as_float(r2.y);
      const float sv = fmaf(-__int_as_float(r.w), added, a.p0);
      const bool better = ok && sv > bs;
      bs = better ? sv : bs;
      bd = better ? d : bd;
      bk = better ? k : bk;
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1)
    keep_best(bs, bd, bk, __shfl_xor(bs, off, kWave), __shfl_xor(bd, off, kWave), __shfl_xor(bk, off, kWave));
  if (lane == 0) {
    s_v[wv] = bs;
    s_d[wv] = bd;
    s_k[wv] = bk;
  }
  __syncthreads();
  if ((wv & 1) == 0 && lane == 0 && valid) {
    keep_best(bs, bd, bk, s_v[wv + 1], s_d[wv + 1], s_k[wv + 1]);
    const bool found = bd != INT_MAX;
    a.best_dst[src] = found ? bd : -1;
    a.saving[src] = found ? bs : -kInf;
    a.level[src] = found ? bk : -1;
  }
}

// ------------------------------------------------------------------ host helpers
size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

struct PlaceLayout {
  size_t cnt, bstart, ntiles, tiles, host_cnt, host_list, recs, preq, key, off, total;
  int32_t NB, tile, max_tiles, waves_per_block;
  bool fast;                     // 8 SM x 16 frequency levels: the specialised kernel
};

bool place_shapes_ok(const festina_lut *L, const festina_gpus *G, const festina_requests *Q) {
  if (!L || !G || !Q) return false;
  if (L->n_models < 1 || L->n_rows != kRows || L->n_sm < 1 || L->n_freq < 1) return false;
  if (G->n_gpus < 1 || G->n_waves < 1 || Q->n_requests < 0) return false;
  return true;
}

bool place_layout(const festina_lut *L, const festina_gpus *G, const festina_requests *Q, PlaceLayout *o) {
  if (!place_shapes_ok(L, G, Q)) return false;
  const long long M = L->n_models, Gn = G->n_gpus, W = G->n_waves, R = Q->n_requests;
  const long long C = (long long)L->n_sm * L->n_freq;
  const long long NB = 2 * W * M;
  if (NB > INT_MAX / 2 - 4 || Gn * C > INT_MAX || W * Gn > INT_MAX || M * Gn > INT_MAX) return false;
  // tile size: large tiles amortise the table staging, small ones fill the chip
  const bool fast = L->n_sm == 8 && L->n_freq == 16;
  int wpb = 4, tile;
  if (fast) {                    // one group of kQF requests per wavefront
    tile = 4 * kQF;
    if (R < 1024LL * tile) {
      wpb = 1;
      tile = kQF;
    }
  } else {
    tile = 2 * 4 * kQ;
    if (R < 2048LL * tile) {
      tile = 4 * kQ;
      if (R < 1024LL * tile) {
        wpb = 1;
        tile = kQ;
      }
    }
  }
  o->fast = fast;
  const long long max_tiles = (R + tile - 1) / tile + NB;
  if (max_tiles > INT_MAX - 8) return false;   // the grid is rounded up to a multiple of 8
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align256(off + bytes);
    return at;
  };
  o->cnt = take(sizeof(int32_t) * ((NB + 3) & ~3LL));       // counters
  o->bstart = take(sizeof(int32_t) * (NB + 1));
  o->ntiles = take(sizeof(int32_t));
  o->tiles = take(sizeof(int2) * max_tiles);
  o->host_cnt = take(sizeof(int32_t) * M);
  o->host_list = take(sizeof(int32_t) * M * Gn);
  o->recs = take(sizeof(HostRec) * W * Gn);
  o->preq = take(sizeof(ReqRec) * (R > 0 ? R : 1));
  o->key = take(sizeof(int32_t) * (R > 0 ? R : 1));
  o->off = take(sizeof(int32_t) * (R > 0 ? R : 1));
  o->total = off;
  o->NB = (int32_t)NB;
  static_assert((kQF & (kQF - 1)) == 0 && (kQ & (kQ - 1)) == 0, "tile sizes are powers of two");
  o->tile = tile;                       // a power of two: the bucket scans shift by its log2
  o->max_tiles = (int32_t)max_tiles;
  o->waves_per_block = wpb;
  return true;
}

// events recorded around the scoring kernels (measurement hook; per host thread)
thread_local hipEvent_t t_events[4] = {nullptr, nullptr, nullptr, nullptr};

hipError_t mark(int which, hipStream_t st) {
  return t_events[which] ? hipEventRecord(t_events[which], st) : hipSuccess;
}

template <int CPL>
hipError_t launch_score(const PlaceArgs &a, int blocks, int wpb, size_t lds, hipStream_t st) {
  k_score<CPL><<<blocks, wpb * kWave, lds, st>>>(a);
  return hipGetLastError();
}

}  // namespace

// ====================================================================== C ABI
extern "C" {

int32_t festina_abi_version(void) { return FESTINA_ABI_VERSION; }

void festina_set_timing_events(void *score_begin, void *score_end, void *pairs_begin, void *pairs_end) {
  t_events[0] = static_cast<hipEvent_t>(score_begin);
  t_events[1] = static_cast<hipEvent_t>(score_end);
  t_events[2] = static_cast<hipEvent_t>(pairs_begin);
  t_events[3] = static_cast<hipEvent_t>(pairs_end);
}

const char *festina_status_string(festina_status s) {
  switch (s) {
    case FESTINA_OK: return "ok";
    case FESTINA_ERR_INVALID: return "invalid argument (null pointer, bad size or workspace too small)";
    case FESTINA_ERR_DEVICE: return "HIP device error";
    case FESTINA_ERR_UNSUPPORTED: return "shape not supported by the kernels";
    case FESTINA_ERR_TOO_LARGE:
      return "input needs more workspace than the library's fixed device scratch holds";
  }
  return "unknown status";
}

size_t festina_placements_workspace_bytes(const festina_lut *lut, const festina_gpus *gpus,
                                          const festina_requests *req) {
  PlaceLayout lay;
  if (!place_layout(lut, gpus, req, &lay)) return 0;
  return lay.total;
}

}  // extern "C"

namespace {

// Checks of a placement call that need no workspace; on success `lay` holds the workspace
// layout.  FESTINA_OK with n_requests == 0 means there is nothing to launch.
festina_status place_args(const festina_lut *L, const festina_gpus *G, const festina_requests *Q,
                          const festina_placements *out, PlaceLayout *lay) {
  if (!place_shapes_ok(L, G, Q) || !out) return FESTINA_ERR_INVALID;
  const long long C = (long long)L->n_sm * L->n_freq;
  if (C > FESTINA_MAX_CELLS) return FESTINA_ERR_UNSUPPORTED;
  if (!L->sm_level || !L->freq_level || !L->pf || !L->dc) return FESTINA_ERR_INVALID;
  if (!G->batch || !G->k_dyn_w || !G->resident) return FESTINA_ERR_INVALID;
  if (!place_layout(L, G, Q, lay)) return FESTINA_ERR_INVALID;
  if (Q->n_requests == 0) return FESTINA_OK;
  if (!Q->model || !Q->prompt_tokens || !Q->pred_out_tokens || !Q->slo_ttft_ms || !Q->slo_tbt_ms)
    return FESTINA_ERR_INVALID;
  if (!out->choice || !out->feasible || !out->energy_mj) return FESTINA_ERR_INVALID;
  return FESTINA_OK;
}

// The launches of one placement call on a checked workspace of lay.total bytes.
festina_status place_launch(const festina_lut *L, const festina_gpus *G, const festina_requests *Q,
                            const festina_placements *out, const PlaceLayout &lay, char *ws, void *stream) {
  const long long C = (long long)L->n_sm * L->n_freq;
  PlaceArgs a;
  a.M = L->n_models;
  a.NS = L->n_sm;
  a.NF = L->n_freq;
  a.C = (int32_t)C;
  a.sm_level = L->sm_level;
  a.freq_level = L->freq_level;
  a.pf = L->pf;
  a.dc = L->dc;
  a.p0 = L->p0_w;
  a.G = G->n_gpus;
  a.W = G->n_waves;
  a.words = (L->n_models + 31) / 32;
  a.batch = G->batch;
  a.kdyn = G->k_dyn_w;
  a.resident = G->resident;
  a.cap_pf = G->cap_pf;
  a.cap_dc = G->cap_dc;
  a.has_caps = (G->cap_pf || G->cap_dc) ? 1 : 0;
  a.R = Q->n_requests;
  a.model = Q->model;
  a.wave = Q->wave;
  a.prompt = Q->prompt_tokens;
  a.pred = Q->pred_out_tokens;
  a.slo_ttft = Q->slo_ttft_ms;
  a.slo_tbt = Q->slo_tbt_ms;
  a.choice = out->choice;
  a.feasible = out->feasible;
  a.energy = out->energy_mj;
  a.NB = lay.NB;
  a.tile = lay.tile;
  a.max_tiles = lay.max_tiles;
  a.cnt = reinterpret_cast<int32_t *>(ws + lay.cnt);
  const int nb4 = (lay.NB + 3) & ~3;      // counters padded with zeros to whole int4
  a.bstart = reinterpret_cast<int32_t *>(ws + lay.bstart);
  a.n_tiles = reinterpret_cast<int32_t *>(ws + lay.ntiles);
  a.tiles = reinterpret_cast<int2 *>(ws + lay.tiles);
  a.host_cnt = reinterpret_cast<int32_t *>(ws + lay.host_cnt);
  a.host_list = reinterpret_cast<int32_t *>(ws + lay.host_list);
  a.recs = reinterpret_cast<HostRec *>(ws + lay.recs);
  a.preq = reinterpret_cast<ReqRec *>(ws + lay.preq);
  a.key = reinterpret_cast<int32_t *>(ws + lay.key);
  a.off = reinterpret_cast<int32_t *>(ws + lay.off);

  hipStream_t st = static_cast<hipStream_t>(stream);
  const int zb = (nb4 + 255) / 256;
  k_zero<<<zb < 1024 ? zb : 1024, 256, 0, st>>>(a.cnt, nb4);
  if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  const int nbr = (a.R + kReqPerPrepBlock - 1) / kReqPerPrepBlock;
  const long long nrec = ((long long)a.W * a.G + kPrepBlock - 1) / kPrepBlock;
  k_prep<<<(unsigned)(nbr + a.M + nrec), kPrepBlock, 0, st>>>(a, nbr);
  if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  const bool local = lay.NB <= kHistMax;
  if (!local) {
    k_scan<<<1, 1024, lay.NB <= kScanLds ? sizeof(int) * lay.NB : 0, st>>>(a);
    if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  }
  k_scatter<<<nbr, kPrepBlock, local ? sizeof(int) * lay.NB : 0, st>>>(a);
  if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  const int cpl = C <= 64 ? 1 : (C <= 128 ? 2 : 4);
  const int wpb = lay.waves_per_block;
  size_t lds = sizeof(float) * score_lds_floats((int)C, cpl, wpb);
  if (lay.fast) {
    const size_t f = fast_lds_bytes(wpb);
    lds = f > lds ? f : lds;
  }
  hipError_t e = mark(0, st);
  if (e != hipSuccess) return FESTINA_ERR_DEVICE;
  if (lay.fast) {
    const int grid = (lay.max_tiles + kXcds - 1) / kXcds * kXcds;
    if (wpb == 4)
      k_score_c128<4><<<grid, 4 * kWave, lds, st>>>(a);
    else
      k_score_c128<1><<<grid, kWave, lds, st>>>(a);
    e = hipGetLastError();
  } else if (cpl == 1)
    e = launch_score<1>(a, lay.max_tiles, wpb, lds, st);
  else if (cpl == 2)
    e = launch_score<2>(a, lay.max_tiles, wpb, lds, st);
  else
    e = launch_score<4>(a, lay.max_tiles, wpb, lds, st);
  if (e == hipSuccess) e = mark(1, st);
  return e == hipSuccess ? FESTINA_OK : FESTINA_ERR_DEVICE;
}

// Workspace of the allocation-free placement entry point: one array per GPU, held by the
// library for the life of the process.  In host code `scratch` names a host-side stand-in;
// the array's device address on each GPU comes from hipGetSymbolAddress, looked up once per
// device (on the first call with that device current) and kept in scratch_dev.
constexpr size_t kScratchBytes = FESTINA_NOALLOC_WORKSPACE_BYTES;
static_assert(kScratchBytes % 256 == 0, "the scratch size is a multiple of the workspace alignment");
__device__ __align__(256) char scratch[kScratchBytes];
constexpr int kScratchDevices = 64;
std::atomic<char *> scratch_dev[kScratchDevices];
std::mutex scratch_mu;

// Device address of the current device's scratch array, or nullptr on a HIP error.
char *scratch_for_current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kScratchDevices) return nullptr;
  char *p = scratch_dev[dev].load(std::memory_order_acquire);
  if (p) return p;
  std::lock_guard<std::mutex> lock(scratch_mu);
  p = scratch_dev[dev].load(std::memory_order_relaxed);
  if (!p) {
    void *addr = nullptr;
    if (hipGetSymbolAddress(&addr, HIP_SYMBOL(scratch)) != hipSuccess || !addr) return nullptr;
    p = static_cast<char *>(addr);
    scratch_dev[dev].store(p, std::memory_order_release);
  }
  return p;
}

}  // namespace

extern "C" {

festina_status festina_score_placements(const festina_lut *L, const festina_gpus *G,
                                        const festina_requests *Q, festina_placements *out,
                                        void *workspace, size_t workspace_bytes, void *stream) {
  PlaceLayout lay;
  const festina_status s = place_args(L, G, Q, out, &lay);
  if (s != FESTINA_OK || Q->n_requests == 0) return s;
  if (!workspace || workspace_bytes < lay.total || (((uintptr_t)workspace) & 255) != 0)
    return FESTINA_ERR_INVALID;
  return place_launch(L, G, Q, out, lay, static_cast<char *>(workspace), stream);
}

festina_status festina_score_placements_noalloc(const festina_lut *L, const festina_gpus *G,
                                                const festina_requests *Q, festina_placements *out,
                                                void *stream) {
  PlaceLayout lay;
  const festina_status s = place_args(L, G, Q, out, &lay);
  if (s != FESTINA_OK || Q->n_requests == 0) return s;
  if (lay.total > kScratchBytes) return FESTINA_ERR_TOO_LARGE;
  char *ws = scratch_for_current_device();
  if (!ws) return FESTINA_ERR_DEVICE;
  return place_launch(L, G, Q, out, lay, ws, stream);
}

static bool mig_shapes_ok(const festina_lut *L, const festina_fleet *F) {
  if (!L || !F) return false;
  if (L->n_models < 1 || L->n_rows != kRows || L->n_sm < 1 || L->n_freq < 1) return false;
  if (F->n_gpus < 2 || F->max_inst < 1) return false;
  if ((long long)F->n_gpus * F->max_inst > INT_MAX) return false;
  return true;
}

size_t festina_migrations_workspace_bytes(const festina_lut *lut, const festina_fleet *fleet) {
  if (!mig_shapes_ok(lut, fleet)) return 0;
  return align256((size_t)32 * fleet->n_gpus);      // one 32-byte destination record per GPU
}

festina_status festina_score_migrations(const festina_lut *L, const festina_fleet *F,
                                        festina_migrations *out, void *workspace,
                                        size_t workspace_bytes, void *stream) {
  if (!mig_shapes_ok(L, F) || !out) return FESTINA_ERR_INVALID;
  if (L->n_freq > FESTINA_MAX_FREQ_MIG) return FESTINA_ERR_UNSUPPORTED;
  if (!L->freq_level || !L->pf || !L->dc) return FESTINA_ERR_INVALID;
  if (!F->n_inst || !F->inst_model || !F->inst_prompt_tokens || !F->inst_batch || !F->inst_sm ||
      !F->inst_slo_ttft_ms || !F->inst_slo_tbt_ms || !F->hbm_mib || !F->sm_permille || !F->util ||
      !F->k_dyn_w)
    return FESTINA_ERR_INVALID;
  if (!out->best_dst || !out->saving_w || !out->freq_level) return FESTINA_ERR_INVALID;
  const size_t need = festina_migrations_workspace_bytes(L, F);
  if (!workspace || workspace_bytes < need || (((uintptr_t)workspace) & 255) != 0) return FESTINA_ERR_INVALID;
  MigArgs a;
  a.M = L->n_models;
  a.NS = L->n_sm;
  a.NF = L->n_freq;
  a.C = L->n_sm * L->n_freq;
  a.freq_level = L->freq_level;
  a.pf = L->pf;
  a.dc = L->dc;
  a.p0 = L->p0_w;
  a.G = F->n_gpus;
  a.K = F->max_inst;
  a.n_inst = F->n_inst;
  a.inst_model = F->inst_model;
  a.inst_prompt = F->inst_prompt_tokens;
  a.inst_batch = F->inst_batch;
  a.inst_sm = F->inst_sm;
  a.inst_slo_ttft = F->inst_slo_ttft_ms;
  a.inst_slo_tbt = F->inst_slo_tbt_ms;
  a.hbm = F->hbm_mib;
  a.smpm = F->sm_permille;
  a.util = F->util;
  a.kdyn = F->k_dyn_w;
  a.hbm_cap = F->hbm_cap_mib;
  a.sm_cap = F->sm_cap_permille;
  a.best_dst = out->best_dst;
  a.saving = out->saving_w;
  a.level = out->freq_level;
  char *ws = static_cast<char *>(workspace);
  a.drec = reinterpret_cast<v4i *>(ws);
  hipStream_t st = static_cast<hipStream_t>(stream);
  k_fleet<<<(a.G + 3) / 4, 256, 0, st>>>(a);
  if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  if (mark(2, st) != hipSuccess) return FESTINA_ERR_DEVICE;
  k_migrate<<<(a.G + kMigSrcPerBlock - 1) / kMigSrcPerBlock, 256, 0, st>>>(a);
  if (hipGetLastError() != hipSuccess || mark(3, st) != hipSuccess) return FESTINA_ERR_DEVICE;
  return FESTINA_OK;
}

}  // extern "C"
