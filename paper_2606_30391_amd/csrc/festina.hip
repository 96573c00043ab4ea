// festina.hip -- MI355X (gfx950) kernels and C-ABI host dispatch of the batched
// energy-aware placement and migration search (Festina, Sec. 3.3 and Sec. 3.5).
//
// Placement pipeline (one call, four launches on the caller's stream, five with k_scan):
//   k_init      clear the bucket counters; the table minima (least entry of each prefill
//                 row, its least nonzero magnitude, least decode entry of each model)
//   k_prep      requests: validity, bucket key (wave, model, has-prompt), the bucket count
//                 and the request's position within its bucket; hosts: per-model list of
//                 hosting GPUs in ascending order (for 8 x 16 tables sorted by SM-cap class
//                 within chunks); GPU records: per (wave, GPU) the post-admission batch row,
//                 k_g * u_g and the SM caps
//   k_scan      one block: bucket offsets and the tile table (only with more buckets than
//                 an LDS histogram holds)
//   k_scatter   bucket offsets and the tile table (each block scans the counts itself),
//                 request records (5% output pad, prompt bucket, SLOs) grouped by bucket
//   k_score_r16 (8 x 16 tables) / k_score (any shape): workgroups of tiles of one bucket's
//                 requests: the model's decode table is staged in LDS, lanes span the
//                 (SM level, frequency level) cells, and the per-request argmin with the
//                 lowest-index tie-break is fused; only 9 bytes per request reach HBM
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
constexpr int kNS8 = 8;
constexpr int kClasses = kNS8 * kNS8;            // (cap_pf, cap_dc) pairs of 8 SM levels
constexpr int kHcap = 128;                       // host records staged in LDS per chunk
// A prompt latency at least this large keeps a normal value when divided by any Lout up to
// 2^40 (2^-86 * 2^-40 = 2^-126, the least normal float).
constexpr float kTinyLatency = 0x1p-86f;
constexpr int kPrepBlock = 256;
static_assert(kHcap <= kPrepBlock, "a chunk's class sort takes one host per thread");
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
  int32_t NB;                    // buckets = 2 * W * M, in groups of gw (see bucket_of)
  int32_t gw, ng;                // buckets per group, groups (ng * gw = NB)
  int32_t tile;                  // requests per tile
  int32_t max_tiles;
  int32_t gpad;                  // tiles per workgroup of the 8 x 16 kernel: the tiles of each
                                 // (model, prompt kind) group are padded to a multiple of it
                                 // with empty tiles (1: no padding)
  int32_t scan_local;            // k_scatter scans the bucket counts itself (else k_scan)
  int32_t *cnt;                  // [NB4] counters
  int32_t *bstart;               // [NB + 1]
  int32_t *n_tiles;              // [1]
  int2 *tiles;                   // [max_tiles] {bucket, first position}; bucket -1: empty tile
  int32_t *gscan;                // [2][ng + 1] group tile prefixes and padded group starts (k_scan)
  int32_t *host_cnt;             // [M]
  int32_t *host_list;            // [M][G]
  HostRec *recs;                 // [W][G]
  ReqRec *preq;                  // [R] request records in bucket order
  int32_t *key;                  // [R]
  int32_t *off;                  // [R] position of request r within its bucket
  // 8 x 16 tables: per model, its host list in chunks of kHcap hosts, each chunk grouped
  // by SM-cap class
  int32_t fast;
  int32_t nch;                   // chunks per model, ceil(G / kHcap)
  int32_t *host_pos;             // [M][G] slot of host i within its chunk's class order
  int32_t *cls_tab;              // [M][nch][kClasses + 1] the chunk's non-empty classes
  // table minima (for requests that no candidate can serve)
  float *pf_rowmin;              // [M][32] least prefill entry of each row (NaN ignored)
  float *pf_rowtiny;             // [M][32] least nonzero magnitude in each prefill row
  float *dc_min;                 // [M] least decode entry of each model
};

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

// A fresh copy of a wave-uniform value: whatever is computed from it (addresses, tests) is
// computed where it is used, not kept in scalar registers from an earlier computation.
__device__ __forceinline__ int fresh_s(int v) {
  asm volatile("" : "+s"(v));
  return v;
}

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

// Buckets: the requests of one (wave, model, prompt kind).  The buckets of a group are
// consecutive, so a group's tiles are contiguous in the tile table.
// The arrival waves form ng / 2M slabs of gw consecutive waves; a group is one (slab, model,
// prompt kind) and its gw buckets, one per wave of the slab, are consecutive: bucket =
// ((slab * 2M + 2 m + prompt-less) * gw + wave within the slab).  Groups are numbered slab
// first, so the XCD that takes a contiguous range of groups writes the results of the
// requests of a few arrival waves (request ids that share cache lines), not of all.
__device__ __forceinline__ int bucket_of(const PlaceArgs &a, int w, int m, bool noprompt) {
  const int sl = w / a.gw;
  return (sl * 2 * a.M + ((m << 1) | (noprompt ? 1 : 0))) * a.gw + (w - sl * a.gw);
}
struct BucketId {
  int w, m;
  bool noprompt;
};
__device__ __forceinline__ BucketId bucket_id(const PlaceArgs &a, int bucket) {
  const int q = bucket / a.gw;                    // the group: slab * 2M + 2 m + prompt-less
  const int sl = q / (2 * a.M), g = q - sl * 2 * a.M;
  return BucketId{sl * a.gw + (bucket - q * a.gw), g >> 1, (g & 1) != 0};
}

// ------------------------------------------------------------------ prologue kernels
// Inclusive prefix sum over a wavefront.
// Inclusive prefix sum over the wavefront's 64 lanes with DPP moves (no LDS permutes):
// shifts by 1, 2, 4 and 8 lanes within each row of 16 (a lane shifted in from outside its
// row adds 0), then row_bcast:15 adds row 0's total to row 1 and row 2's to row 3, and
// row_bcast:31 adds the total of rows 0-1 to rows 2 and 3.
__device__ __forceinline__ int wave_scan(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);   // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);   // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);   // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);   // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);   // row_bcast:15, rows 1 and 3
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);   // row_bcast:31, rows 2 and 3
  return v;
}

__device__ __forceinline__ float wave_minf(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float o = __shfl_xor(v, off, kWave);
    v = o < v ? o : v;
  }
  return v;
}

// Blocks [0, zb): clear the bucket counters.  Blocks [zb, zb + 8M): four prefill-table rows
// each, one per wavefront: the least entry (NaN ignored) and the least nonzero magnitude.
// Blocks [zb + 8M, zb + 9M): the least entry of one model's decode table.
__global__ void __launch_bounds__(256) k_init(PlaceArgs a, int32_t zb, int32_t nb4) {
  const int b = blockIdx.x;
  if (b < zb) {
    for (int i = b * 256 + (int)threadIdx.x; i < nb4; i += zb * 256) a.cnt[i] = 0;
    return;
  }
  const int lane = threadIdx.x & (kWave - 1);
  if (b < zb + 8 * a.M) {
    const int row = (b - zb) * 4 + (int)(threadIdx.x >> 6);        // m * 32 + prompt row
    const float *p = a.pf + (size_t)row * a.C;
    float mn = kInf, tiny = kInf;
    constexpr int U = FESTINA_MAX_CELLS / kWave;                   // the row's loads together
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = lane + u * kWave < a.C ? p[lane + u * kWave] : kInf;
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const float av = fabsf(v[u]);
      mn = v[u] < mn ? v[u] : mn;
      tiny = av > 0.f && av < tiny ? av : tiny;
    }
    mn = wave_minf(mn);
    tiny = wave_minf(tiny);
    if (lane == 0) {
      a.pf_rowmin[row] = mn;
      a.pf_rowtiny[row] = tiny;
    }
    return;
  }
  __shared__ float part[256 / kWave];
  const int m = b - zb - 8 * a.M;
  const float *p = a.dc + (size_t)m * kRows * a.C;
  float mn = kInf;
  constexpr int U = 8;                                             // loads in flight per thread
  for (int c0 = threadIdx.x; c0 < kRows * a.C; c0 += U * 256) {
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = c0 + u * 256 < kRows * a.C ? p[c0 + u * 256] : kInf;
#pragma unroll
    for (int u = 0; u < U; ++u) mn = v[u] < mn ? v[u] : mn;
  }
  mn = wave_minf(mn);
  if (lane == 0) part[threadIdx.x >> 6] = mn;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < 256 / kWave; ++i) mn = part[i] < mn ? part[i] : mn;
    a.dc_min[m] = mn;
  }
}

// The fields of request r that decide its bucket.
struct ReqKeyFields {
  int m, w, pt, pr;
  float st, sb;
};
__device__ __forceinline__ ReqKeyFields load_key_fields(const PlaceArgs &a, int r) {
  return ReqKeyFields{a.model[r], a.wave ? a.wave[r] : 0, a.prompt[r], a.pred[r], a.slo_ttft[r], a.slo_tbt[r]};
}

// Prompt bucket of a token count: min(ceil(tokens / 256), 32) - 1 (unsigned: no overflow for
// any int32 count; 0 tokens give -1, the decode batch row).
__device__ __forceinline__ int prompt_row(int pt) {
  return pt == 0 ? -1 : (min((int)(((unsigned)pt + 255u) >> 8), kRows) - 1);
}

// Validity and bucket key (wave, model, has-prompt) of request r from its fields.  Returns
// the key, or -1 (and writes the infeasible result) for an invalid request and for one that
// no candidate can serve: no entry of its model's decode table is below its TBT SLO, or no
// entry of its prefill row is below its TTFT SLO (the SLO test of every candidate reads one
// of those entries, so none can pass).  The stored key carries kKeyTiny when the 8 x 16
// kernel must not divide the request's prompt row by Lout (see make_req_rec).
constexpr int kKeyTiny = 1 << 30;                 // bucket numbers stay below 2^30
// The table minima a request's test reads: loaded for every request (at model 0 / row 0 for
// an invalid one), so that the loads of several requests issue together, before any test.
struct ReqMins {
  float dmin, pmin, ptiny;
};
__device__ __forceinline__ ReqMins load_req_mins(const PlaceArgs &a, const ReqKeyFields &f) {
  const bool mv = f.m >= 0 && f.m < a.M;
  const int m = mv ? f.m : 0, row = f.pt > 0 ? prompt_row(f.pt) : 0;
  return ReqMins{a.dc_min[m], a.pf_rowmin[m * kRows + row], a.pf_rowtiny[m * kRows + row]};
}
__device__ __forceinline__ int prep_request(const PlaceArgs &a, int r, const ReqKeyFields &f, const ReqMins &mn) {
  bool ok = f.m >= 0 && f.m < a.M && f.w >= 0 && f.w < a.W && f.pt >= 0 && f.pr >= 0;
  bool tiny = false;
  if (ok) {
    const int row = prompt_row(f.pt);
    ok = mn.dmin < f.sb && (row < 0 || mn.pmin < f.st);
    tiny = a.fast && row >= 0 && mn.ptiny < kTinyLatency;
  }
  if (!ok) {
    a.key[r] = -1;
    a.choice[r] = -1;
    a.feasible[r] = 0;
    a.energy[r] = kInf;
    return -1;
  }
  const int k = bucket_of(a, f.w, f.m, f.pt == 0);
  __builtin_nontemporal_store(k | (tiny ? kKeyTiny : 0), &a.key[r]);   // read by the next kernel
  return k;
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

// SM-cap class of GPU g for the 8 x 16 chunk sort: caps outside [0, 7] (a GPU without
// candidates) are clamped; absent cap arrays mean 7.  The loads are unconditional (an
// absent array reads kNoCap), so that a caller's loads of several GPUs issue together.
__device__ const int8_t kNoCap = 0;                // read in place of absent cap arrays
__device__ __forceinline__ int host_class(const PlaceArgs &a, int g) {
  const int8_t cpv = *(a.cap_pf ? a.cap_pf + g : &kNoCap);
  const int8_t cdv = *(a.cap_dc ? a.cap_dc + g : &kNoCap);
  const int cp = a.cap_pf ? min(max((int)cpv, 0), kNS8 - 1) : kNS8 - 1;
  const int cd = a.cap_dc ? min(max((int)cdv, 0), kNS8 - 1) : kNS8 - 1;
  return class_id(cp, cd);
}

// Model m's host list, in chunks of kHcap hosts, grouped by SM-cap class within each chunk
// (8 x 16 tables): host_pos[m][i] = slot of host i within its chunk, and per chunk the list
// of non-empty classes in ascending class number, each as cap_pf * 8 + cap_dc | first slot
// << 6 | end slot << 15, with the count at [kClasses].  One block of kPrepBlock threads;
// `cnt` is LDS scratch of kClasses ints; `keys` holds the class of each of the first nkeys
// hosts in list order (LDS), the others are looked up.
__device__ void sort_host_chunks(const PlaceArgs &a, int m, int hcnt, int *cnt, const int *keys, int nkeys) {
  const int t = threadIdx.x;
  for (int c0 = 0, ch = 0; c0 < hcnt; c0 += kHcap, ++ch) {
    __syncthreads();                      // the host list is written; the counts are free
    if (t < kClasses) cnt[t] = 0;
    __syncthreads();
    const int i = c0 + t;
    int key = -1, rank = 0;
    if (t < kHcap && i < hcnt) {
      key = i < nkeys ? keys[i] : host_class(a, a.host_list[(size_t)m * a.G + i]);
      rank = atomicAdd(&cnt[key], 1);
    }
    __syncthreads();
    int *tab = a.cls_tab + ((size_t)m * a.nch + ch) * (kClasses + 1);
    if (t < kWave) {                      // exclusive prefix over the 64 classes, compact list
      const int n = cnt[t];
      const int inc = wave_scan(n);
      const unsigned long long ne = __ballot(n > 0);
      const int pos = __popcll(ne & ((1ull << t) - 1ull));
      if (n > 0) tab[pos] = class_caps(t) | ((inc - n) << 6) | (inc << 15);
      if (t == kWave - 1) tab[kClasses] = __popcll(ne);
      cnt[t] = inc - n;
    }
    __syncthreads();
    if (key >= 0) a.host_pos[(size_t)m * a.G + i] = cnt[key] + rank;
  }
}

// The LDS histogram's flush: each non-empty slot's count is added to its bucket's global
// counter, and the returned old value (this block's base within the bucket) replaces it.
// Slot h = w * 2M + g holds the bucket of wave w = sl * gw + wr and 2 m + prompt-less = g;
// (sl, wr, g) advance with h by constant steps (two divisions per thread, none per slot),
// and the KF slots of a round have their atomics issued together (one round trip to the
// counters per round, not per slot).  Called by the whole block between two barriers.
template <int KF>
__device__ __forceinline__ void flush_hist(const PlaceArgs &a, int *hist) {
  const int NG = 2 * a.M;
  const int dw = kPrepBlock / NG, dg = kPrepBlock - dw * NG;
  const int dsl = dw / a.gw, dwr = dw - dsl * a.gw;
  const int w0 = (int)threadIdx.x / NG;
  int g = (int)threadIdx.x - w0 * NG, sl = w0 / a.gw, wr = w0 - sl * a.gw;
  for (int h0 = threadIdx.x; h0 < a.NB; h0 += KF * kPrepBlock) {
    int cv[KF], bk[KF];
#pragma unroll
    for (int u = 0; u < KF; ++u) {
      const int h = h0 + u * kPrepBlock;
      cv[u] = h < a.NB ? hist[h] : 0;
      bk[u] = (sl * NG + g) * a.gw + wr;
      g += dg;                            // next slot: w += dw (sl += dsl, wr += dwr), g += dg
      sl += dsl;
      wr += dwr;
      if (g >= NG) {
        g -= NG;
        ++wr;
      }
      if (wr >= a.gw) {                   // wr < 2 gw here: dwr < gw, plus at most one carry
        wr -= a.gw;
        ++sl;
      }
    }
    int base[KF];
#pragma unroll
    for (int u = 0; u < KF; ++u) base[u] = cv[u] ? atomicAdd(&a.cnt[bk[u]], cv[u]) : 0;
#pragma unroll
    for (int u = 0; u < KF; ++u)
      if (cv[u]) hist[h0 + u * kPrepBlock] = base[u];
  }
}

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
    // The LDS histogram is indexed wave-major, h = w * 2M + (2 m + prompt-less): requests that
    // arrive together share w and spread over consecutive words (banks), where the bucket
    // numbers, W apart, would all fall on one bank.
    // the table minima of all U requests in one round trip, then the tests
    ReqMins mn[U];
#pragma unroll
    for (int u = 0; u < U; ++u) mn[u] = load_req_mins(a, f[u]);
    int key[U], pos[U], hk[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int r = b * kReqPerPrepBlock + u * kPrepBlock + threadIdx.x;
      key[u] = r < a.R ? prep_request(a, r, f[u], mn[u]) : -1;
      hk[u] = f[u].w * (2 * a.M) + ((f[u].m << 1) | (f[u].pt == 0 ? 1 : 0));
    }
    // the LDS histogram and the global counters in separate loops: an atomic through a
    // pointer that may be either would be a flat atomic, waited for like a global one
    if (local) {
#pragma unroll
      for (int u = 0; u < U; ++u) pos[u] = key[u] >= 0 ? atomicAdd(&hist[hk[u]], 1) : 0;
    } else {
#pragma unroll
      for (int u = 0; u < U; ++u) pos[u] = key[u] >= 0 ? atomicAdd(&a.cnt[key[u]], 1) : 0;
    }
    if (local) {
      __syncthreads();
      // KF slots per thread per round (all slots of the histogram in one round up to 16 per
      // thread; four per round for small histograms, whose extra slots would only cost the walk)
      if (a.NB > 4 * kPrepBlock)
        flush_hist<16>(a, hist);
      else
        flush_hist<4>(a, hist);
      __syncthreads();
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (key[u] >= 0) pos[u] += hist[hk[u]];
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (key[u] >= 0) __builtin_nontemporal_store(pos[u], &a.off[b * kReqPerPrepBlock + u * kPrepBlock + threadIdx.x]);
    return;
  }
  if (b < nbr + a.M) {
    // ascending list of GPUs whose resident mask has bit m, kHostU chunks of kPrepBlock GPUs
    // per round with their mask words (and SM caps) requested together; with the 8 x 16
    // tables each listed GPU's SM-cap class goes to LDS for the chunk sort
    constexpr int kHostU = 4;
    const int m = b - nbr;
    __shared__ int wsum[kHostU][kPrepBlock / kWave];
    const int lane = threadIdx.x & (kWave - 1), wv = threadIdx.x >> 6;
    int *keys = hist + kClasses;                   // classes of the first nkeys listed hosts
    const int nkeys = kHistMax - kClasses;
    int base = 0;
    for (int G0 = 0; G0 < a.G; G0 += kHostU * kPrepBlock) {
      bool has[kHostU];
      int key[kHostU];
#pragma unroll
      for (int u = 0; u < kHostU; ++u) {
        const int g = G0 + u * kPrepBlock + threadIdx.x;
        const int gc = min(g, a.G - 1);
        const uint32_t word = a.resident[(size_t)gc * a.words + (m >> 5)];   // loads unconditional
        const int cls = host_class(a, gc);
        has[u] = g < a.G && ((word >> (m & 31)) & 1u);
        key[u] = a.fast ? cls : 0;
      }
      int before[kHostU];
#pragma unroll
      for (int u = 0; u < kHostU; ++u) {
        const unsigned long long bal = __ballot(has[u]);
        before[u] = __popcll(bal & ((1ull << lane) - 1ull));
        if (lane == 0) wsum[u][wv] = __popcll(bal);
      }
      __syncthreads();
      int off = base;
#pragma unroll
      for (int u = 0; u < kHostU; ++u) {
        int tot = 0, mine = off;
        for (int i = 0; i < kPrepBlock / kWave; ++i) {
          if (i < wv) mine += wsum[u][i];
          tot += wsum[u][i];
        }
        if (has[u]) {
          const int g = G0 + u * kPrepBlock + threadIdx.x;
          a.host_list[(size_t)m * a.G + mine + before[u]] = g;
          if (mine + before[u] < nkeys) keys[mine + before[u]] = key[u];
        }
        off += tot;
      }
      base = off;
      __syncthreads();                            // wsum is rewritten next round
    }
    if (threadIdx.x == 0) a.host_cnt[m] = base;
    if (a.fast) sort_host_chunks(a, m, base, hist, keys, nkeys);
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

// Group padding: the ng groups each end with (gP[g] - gP[g + 1]) mod gpad empty tiles.  gP
// holds the unpadded tile index of each group's first bucket, with the tile total at [ng];
// the scan writes pp[g] = the padded index of group g's first tile (gP[g] plus the pads of
// the groups before it), pp[ng] = the padded total.  The whole block takes part;
// s_a is LDS scratch of blockDim / 64 ints that no thread still reads; ends with a barrier.
template <typename P>
__device__ void scan_group_pads(const PlaceArgs &a, P gP, P pp, int *s_a) {
  const int NG = a.ng, T = blockDim.x, gm = a.gpad - 1;
  const int per = (NG + T - 1) / T;
  const int lo = min((int)threadIdx.x * per, NG), hi = min(lo + per, NG);
  int s = 0;
  for (int g = lo; g < hi; ++g) s += (gP[g] - gP[g + 1]) & gm;
  const int is = wave_scan(s);
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & (kWave - 1);
  if (lane == kWave - 1) s_a[wv] = is;
  __syncthreads();
  int p = is - s, tot = 0;
  for (int i = 0; i < T / kWave; ++i) {
    if (i < wv) p += s_a[i];
    tot += s_a[i];
  }
  for (int g = lo; g < hi; ++g) {
    pp[g] = gP[g] + p;
    p += (gP[g] - gP[g + 1]) & gm;
  }
  if (threadIdx.x == 0) pp[NG] = gP[NG] + tot;
  __syncthreads();
}

// Table entries of bucket i (n requests from position pc; its first tile at index t): one per
// tile of a.tile requests.
__device__ __forceinline__ void put_tiles(const PlaceArgs &a, int i, int n, int pc, int t) {
  const int nt = (n + a.tile - 1) >> __builtin_ctz((unsigned)a.tile);
  for (int k = 0; k < nt; ++k) a.tiles[t + k] = make_int2(i, pc + k * a.tile);
}

// Scan body over bucket counts `cnt` (LDS copy or the global counters themselves).
template <typename P>
__device__ __forceinline__ void scan_buckets(const PlaceArgs &a, P cnt, int *s_cnt, int *s_til) {
  const int T = blockDim.x;
  const int per = (a.NB + T - 1) / T;
  const int lo = min((int)threadIdx.x * per, a.NB);
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
  int pc0 = ic - c, pt0 = it - t;                // exclusive prefix within the wave
  int tot_c = 0, tot_t = 0;
  for (int i = 0; i < T / kWave; ++i) {
    if (i < wv) {
      pc0 += s_cnt[i];
      pt0 += s_til[i];
    }
    tot_c += s_cnt[i];
    tot_t += s_til[i];
  }
  const bool pad = a.gpad > 1;
  int *gP = a.gscan, *pp = a.gscan + a.ng + 1;
  const int g0 = lo / a.gw, w0 = lo - g0 * a.gw;
  {
    int pc = pc0, pt = pt0, g = g0, wi = w0;
    for (int i = lo; i < hi; ++i) {
      const int n = cnt[i];
      a.bstart[i] = pc;
      if (!pad)
        put_tiles(a, i, n, pc, pt);
      else if (wi == 0)
        gP[g] = pt;
      pc += n;
      pt += (n + a.tile - 1) / a.tile;
      if (++wi == a.gw) {
        wi = 0;
        ++g;
      }
    }
  }
  int pads = 0;
  if (pad) {
    if (threadIdx.x == 0) gP[a.ng] = tot_t;
    __syncthreads();
    scan_group_pads(a, gP, pp, s_cnt);
    int pc = pc0, pt = pt0, g = g0, wi = w0;
    for (int i = lo; i < hi; ++i) {
      const int n = cnt[i];
      const int nt = (n + a.tile - 1) / a.tile;
      put_tiles(a, i, n, pc, pt - gP[g] + pp[g]);
      if (wi == a.gw - 1)                 // the group's empty tiles follow its last bucket
        for (int k = pt + nt - gP[g] + pp[g]; k < pp[g + 1]; ++k) a.tiles[k] = make_int2(-1, 0);
      pc += n;
      pt += nt;
      if (++wi == a.gw) {
        wi = 0;
        ++g;
      }
    }
    pads = pp[a.ng] - tot_t;
  }
  if (threadIdx.x == 0) {
    a.bstart[a.NB] = tot_c;
    *a.n_tiles = tot_t + pads;
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
// [1, 2^40]), and the SLOs.  The 8 x 16 kernel scores prompt latencies divided by Lout: only
// while every entry of the prompt row keeps a normal value after the division (or is zero);
// for a row with a smaller nonzero entry k_prep flags the key (kKeyTiny) and take_key sets
// the reciprocal to 0, which sends the request's tile to the generic code.
__device__ __forceinline__ ReqRec make_req_rec(const PlaceArgs &a, int r) {
  const int pt = a.prompt[r];
  ReqRec q;
  q.r = r;
  q.row = prompt_row(pt);
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
// before the first use; the counter array is padded to a multiple of 4 with zeros.  Every
// block scans all buckets (a few KB from L2); the global bucket starts are written by the
// grid from LDS after the block's last barrier (one bucket per thread), the tile table by
// every thread of the grid (one entry each, its bucket found by a binary search over the
// buckets' first tiles in LDS), and block 0 writes the totals.
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

// LDS of block_scan_buckets (ints): [NB4] bucket starts, [NB4 + 4] first tile of each bucket
// and the tile total (NB4 = NB rounded up to 4, so both arrays take 16-byte stores), then
// with group padding [2][ng + 1] group tables.
__host__ __device__ constexpr long long block_scan_ints(long long NB, long long NG, bool pad) {
  return 2 * ((NB + 3) & ~3LL) + 4 + (pad ? 2 * (NG + 1) : 0);
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
  int pc0 = ic - c, pt0 = it - t;
  int tot_c = 0, tot_t = 0;
  for (int i = 0; i < kPrepBlock / kWave; ++i) {
    if (i < wv) {
      pc0 += s_c[i];
      pt0 += s_t[i];
    }
    tot_c += s_c[i];
    tot_t += s_t[i];
  }
  const bool pad = a.gpad > 1;
  const int NB4 = (a.NB + 3) & ~3;
  int *ts = start + NB4;                             // [NB + 1] unpadded first tile of each bucket
  int *gP = ts + NB4 + 4, *pp = gP + a.ng + 1;       // [ng + 1] each, with group padding
  const int g0 = lo / a.gw, w0 = lo - g0 * a.gw;
  {
    // a thread's buckets are 4-aligned and contiguous: each chunk of 4 starts goes to LDS as
    // one 16-byte store per array (a chunk past NB holds zero counts, so its entries past NB
    // repeat the totals, and ts[NB] gets the tile total)
    int pc = pc0, pt = pt0, g = g0, wi = w0;
#pragma unroll
    for (int q = 0; q < V; ++q)
      if (lo + 4 * q < hi) {
        v4i sv, tv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int n = v[q][e];
          sv[e] = pc;
          tv[e] = pt;
          if (lo + 4 * q + e < hi) {
            if (pad && wi == 0) gP[g] = pt;
            if (++wi == a.gw) {
              wi = 0;
              ++g;
            }
          }
          pc += n;
          pt += (n + a.tile - 1) >> tsh;
        }
        *reinterpret_cast<v4i *>(start + lo + 4 * q) = sv;
        *reinterpret_cast<v4i *>(ts + lo + 4 * q) = tv;
      }
  }
  if (threadIdx.x == 0) ts[a.NB] = tot_t;
  int total = tot_t;
  if (pad) {
    if (threadIdx.x == 0) gP[a.ng] = tot_t;
    __syncthreads();
    scan_group_pads(a, gP, pp, s_c);
    total = pp[a.ng];
  } else {
    __syncthreads();
  }
  // the global bucket starts, copied from LDS after the last barrier (a global store before
  // a barrier holds the barrier until the store is acknowledged); block b writes buckets
  // b * 256 + t, (b + grid) * 256 + t, ...
  for (int i = blockIdx.x * kPrepBlock + threadIdx.x; i < a.NB; i += gridDim.x * kPrepBlock) a.bstart[i] = start[i];
  // Padded tile k: its group g (pp[g] <= k < pp[g + 1]; an empty group's range is empty), its
  // unpadded index u within the group's tiles, and the bucket l of the group with ts[l] <= u <
  // ts[l + 1]; u past the group's tiles is one of its empty tiles.  Without padding the
  // bucket is searched among all buckets.
  for (int k = blockIdx.x * kPrepBlock + threadIdx.x; k < total; k += gridDim.x * kPrepBlock) {
    int u = k, l = 0, h = a.NB;                      // ts[l] <= u < ts[h]
    bool empty = false;
    if (pad) {
      int gl = 0, gh = a.ng;                         // pp[gl] <= k < pp[gh]
      while (gh - gl > 1) {
        const int mid = (gl + gh) >> 1;
        if (pp[mid] <= k)
          gl = mid;
        else
          gh = mid;
      }
      u = k - pp[gl] + gP[gl];
      empty = u >= gP[gl + 1];
      l = gl * a.gw;
      h = l + a.gw;
    }
    if (!empty) {
      while (h - l > 1) {
        const int mid = (l + h) >> 1;
        if (ts[mid] <= u)
          l = mid;
        else
          h = mid;
      }
    }
    const int off = u - ts[l];
    const int n = (l + 1 < a.NB ? start[l + 1] : tot_c) - start[l];
    a.tiles[k] = !empty && off < ((n + a.tile - 1) >> tsh) ? make_int2(l, start[l] + off * a.tile) : make_int2(-1, 0);
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    a.bstart[a.NB] = tot_c;
    *a.n_tiles = total;
  }
}

// Requests grouped by bucket: request r goes to its bucket's start plus its position from
// k_prep.  With a.scan_local (at most kHistMax buckets, and the group tables fit beside the
// starts in kScanLds ints of LDS) each block scans the bucket counts itself; otherwise k_scan
// has written the bucket starts and the tile table.
constexpr int kScatterU = kReqPerPrepBlock / kPrepBlock;

// A request record written with streaming (nontemporal) stores: the next kernel reads it on
// any XCD, so it is not kept in this XCD's L2 to be written back when the kernel ends.
__device__ __forceinline__ void store_rec_nt(ReqRec *p, const ReqRec &r) {
  const v4i lo = v4i{r.r, r.row, __float_as_int(r.lout), __float_as_int(r.slo_ttft)};
  const v4i hi = v4i{__float_as_int(r.slo_tbt), __float_as_int(r.rlout), 0, 0};
  __builtin_nontemporal_store(lo, reinterpret_cast<v4i *>(p));
  __builtin_nontemporal_store(hi, reinterpret_cast<v4i *>(p) + 1);
}

// Request u of this thread: stored key (-1: none), position and record.  Every load is issued
// before the first use; a thread past the last request reads the last one (R >= 1) and drops
// it, and an invalid request's position (never written) is not used.  take_key then splits
// the key into the bucket and the prompt-row flag.
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

__device__ __forceinline__ void take_key(int (&key)[kScatterU], ReqRec (&rec)[kScatterU]) {
#pragma unroll
  for (int u = 0; u < kScatterU; ++u)
    if (key[u] >= 0) {
      if (key[u] & kKeyTiny) rec[u].rlout = 0.f;
      key[u] &= kKeyTiny - 1;
    }
}

__global__ void __launch_bounds__(kPrepBlock) k_scatter(PlaceArgs a) {
  extern __shared__ __align__(16) int start[];   // block_scan_ints(NB, ng, padded) ints
  int key[kScatterU], pos[kScatterU];
  ReqRec rec[kScatterU];
  if (a.scan_local) {
    // the bucket counts are requested together with the request fields: one round trip
    v4i cv[kScanChunks];
    load_scan_counts(a, cv);
    scatter_loads(a, key, pos, rec);
    __builtin_amdgcn_sched_barrier(0);   // no use of a loaded value is scheduled before a load
    block_scan_buckets(a, start, cv);    // the bucket starts are complete on return
    take_key(key, rec);
#pragma unroll
    for (int u = 0; u < kScatterU; ++u)
      if (key[u] >= 0) store_rec_nt(a.preq + start[key[u]] + pos[u], rec[u]);
  } else {
    scatter_loads(a, key, pos, rec);
    take_key(key, rec);
#pragma unroll
    for (int u = 0; u < kScatterU; ++u)
      if (key[u] >= 0) store_rec_nt(a.preq + a.bstart[key[u]] + pos[u], rec[u]);
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

// The scoring loop of score_requests_generic for one kind of tile: MODE 0 prompt-less
// requests, 1 GPUs without SM caps, 2 capped GPUs (one loop per kind keeps the kind's branch
// out of the loop body).
template <int CPL, int MODE, int FNF>
__device__ void generic_loop(const PlaceArgs &a, int m, int w, int beg, int end, int stride, float *lds) {
  const int C = FNF ? kNS8 * FNF : a.C, NF = FNF ? FNF : a.NF;
  float *dcs = lds;
  float *pds = lds + kRows * C + kWave * CPL;
  float *rows = pds + C;

  const int wv = uniform(threadIdx.x >> 6);
  const int lane = threadIdx.x & (kWave - 1);
  float *myrows = rows + (size_t)wv * kQ * C;
  const int hcnt = ro(a.host_cnt)[m];
  // the model's host list and the wave's records are addressed afresh for each GPU (a few
  // scalar instructions) instead of holding both 64-bit bases through the request loop
  const auto hl = [&](int i) { return ro(a.host_list)[(size_t)fresh_s(m) * (unsigned)a.G + i]; };
  const auto rw = [&]() { return ro(a.recs + (size_t)fresh_s(w) * (unsigned)a.G); };
  const float p0 = a.p0;

  int cj[CPL], ck[CPL];
  int livev[CPL];                 // 1: a cell of the table, 0: a slot past the last cell
  float pdl[CPL];
#pragma unroll
  for (int u = 0; u < CPL; ++u) {
    const int c = lane * CPL + u;
    livev[u] = c < C ? 1 : 0;
    const int cc = c < C ? c : 0;
    cj[u] = cc / NF;
    ck[u] = cc - cj[u] * NF;
    pdl[u] = pds[cc];
  }

  for (int base = beg; base < end; base += stride) {
    int rq[kQ];
    float lo[kQ], st[kQ], sb[kQ];
    int prw[kQ];
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const int pos = base + q;
      const ReqRec rr = load_req_lane(a, pos < end ? pos : beg);   // in VGPRs: frees scalar registers
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

    if constexpr (MODE == 0) {
      // TTFT from the prefill table at the decode batch row (global, L2-resident)
      const float *pfm = a.pf + (size_t)m * kRows * C;
      for (int i = 0; i < hcnt; ++i) {
        const int g = hl(i);
        const HostRec rec = load_rec(rw(), g);
        if (rec.row_off < 0) continue;
        const int cp = rec.caps & 0xff, cd = (rec.caps >> 8) & 0xff;
        // the cell tests are remade per GPU from vector values, not held as lane masks in
        // scalar registers across the loop
        int lv[CPL];
#pragma unroll
        for (int u = 0; u < CPL; ++u) {
          lv[u] = livev[u];
          asm volatile("" : "+v"(lv[u]));
        }
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
            const bool ok = lv[u] != 0 && ttft < st[q] && tbt < sb[q] && E < be[q][u];
            be[q][u] = ok ? E : be[q][u];
            bg[q][u] = ok ? g : bg[q][u];
          }
        }
      }
    } else if constexpr (MODE == 1) {
      // uncapped: the request's TTFT cells stay in registers, masked by its TTFT SLO
      float tt[kQ][CPL];
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
        const float *pr = a.pf + ((size_t)m * kRows + prw[q]) * C;
#pragma unroll
        for (int u = 0; u < CPL; ++u) {
          const float v = (rq[q] >= 0 && livev[u] != 0) ? pr[lane * CPL + u] : kInf;
          tt[q][u] = v < st[q] ? v : kMask;
        }
      }
      for (int i = 0; i < hcnt; ++i) {
        const int g = hl(i);
        const HostRec rec = load_rec(rw(), g);
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
        const int g = hl(i);
        const HostRec rec = load_rec(rw(), g);
        if (rec.row_off < 0) continue;
        const int cp = rec.caps & 0xff, cd = (rec.caps >> 8) & 0xff;
        // the cell tests are remade per GPU from vector values, not held as lane masks in
        // scalar registers across the loop
        int lv[CPL];
#pragma unroll
        for (int u = 0; u < CPL; ++u) {
          lv[u] = livev[u];
          asm volatile("" : "+v"(lv[u]));
        }
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
            const bool ok = lv[u] != 0 && tbt < sb[q] && E < be[q][u];
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

// Requests [beg, end) of bucket positions, read by this wavefront kQ at a time from beg with
// step `stride`, of model m and arrival wave w (both wave-uniform; beg = end: no requests).
// The whole workgroup calls it (it stages the model's decode table in LDS).
// FNF = 16: the 8 x 16 tables (their sizes known when compiled), 0: any.
template <int CPL, int FNF = 0>
__device__ void score_requests_generic(const PlaceArgs &a, int m, bool noprompt, int w, int beg, int end,
                                       int stride, float *lds) {
  const int C = FNF ? kNS8 * FNF : a.C, NF = FNF ? FNF : a.NF;
  float *dcs = lds;                                   // [32 * C + pad] decode table of the tile's model
  float *pds = lds + kRows * C + kWave * CPL;         // [C] s_j * f_k^3, then per wavefront
                                                      // [Q][C] prompt rows (capped GPUs)

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
  if (noprompt)
    generic_loop<CPL, 0, FNF>(a, m, w, beg, end, stride, lds);
  else if (a.has_caps == 0)
    generic_loop<CPL, 1, FNF>(a, m, w, beg, end, stride, lds);
  else
    generic_loop<CPL, 2, FNF>(a, m, w, beg, end, stride, lds);
}

// Tile t of the tile table: its bucket's requests [first, first + tile), wavefront v taking
// kQ of them at positions first + v * kQ + i * waves * kQ.
template <int CPL>
__device__ void score_tile_generic(const PlaceArgs &a, int t, float *lds) {
  const auto tp = ro(reinterpret_cast<const int32_t *>(a.tiles));
  const int bucket = tp[2 * t];
  const BucketId id = bucket_id(a, bucket);
  const int first = tp[2 * t + 1];
  const int end = min(first + a.tile, ro(a.bstart)[bucket + 1]);
  const int nwaves = blockDim.x / kWave;
  const int wv = uniform(threadIdx.x >> 6);
  score_requests_generic<CPL>(a, id.m, id.noprompt, id.w, first + wv * kQ, end, nwaves * kQ, lds);
}

template <int CPL>
__global__ void __launch_bounds__(256) k_score(PlaceArgs a) {
  extern __shared__ __align__(16) float lds[];
  if ((int)blockIdx.x >= *ro(a.n_tiles)) return;
  score_tile_generic<CPL>(a, blockIdx.x, lds);
}

// ------------------------------------------------------------------ helpers of the 8 x 16 kernel
constexpr int kXcds = 8;                         // MI355X: 8 XCDs, each with its own L2

typedef float v2f __attribute__((ext_vector_type(2)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef unsigned int v2u __attribute__((ext_vector_type(2)));

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

// DPP lane moves within rows of 16 lanes (every source lane exists).
constexpr int kDppRor8 = 0x128;        // row_ror:8: lane i reads lane i ^ 8 of its row
constexpr int kDppHalfMirror = 0x141;  // lane i reads lane 7 - i of its group of 8
constexpr int kDppQuad2301 = 0x4E;     // lane i reads lane i ^ 2 of its quad
constexpr int kDppQuad1032 = 0xB1;     // lane i reads lane i ^ 1 of its quad

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}

// ------------------------------------------------------------------ 8 x 16 scoring kernel
// Tables of 8 SM levels x 16 frequency levels (128 cells).  A workgroup takes a tile of
// WPB * kR requests of one (wave, model) bucket; each wavefront scores its kR = 16
// requests against every GPU hosting the model.
//
// A candidate's key is its energy divided by the request's Lout (Eq. energy, Sec. 3.3):
//   key = Pp * (TTFT / Lout) + Pd * TBT,  Pp = P0 + k_g u_g s_jp f_k^3,  Pd = P0 + k_g u_g s_jd f_k^3,
// one FMA once the request term x = TTFT / Lout is staged; Lout is one positive scale per
// request, so its keys order as its energies (up to rounding) and its energy is Lout times
// its least key.
//
// Lane l owns one cell of each of two ranges of SM levels, (j, k) = (l / 16, l % 16) in
// range A (levels 0-3) and (4 + l / 16, l % 16) in range B (levels 4-7), and keeps the
// request terms of both cells for the 16 requests in registers (xA, xB; NaN where TTFT misses
// the SLO).  Pass 1 runs range A, then range B, over the tile's GPUs, which k_prep grouped by
// SM-cap class (cap_pf, cap_dc) in ascending m = max(cap_pf, cap_dc); a GPU's cells above
// level m repeat its level-m cells at a higher index, so they need no work.  Per class the
// lanes fetch the capped request terms x(q, min(j, cap_pf), k) from xA / xB (ds_bpermute)
// and the power factors; per GPU a lane reads one TBT value and forms Pp and Pd * TBT, shared
// by its 16 requests: 16 FMA and 8 v_min3 per GPU for 16 candidates.  A class with one or two
// levels in the range packs 4 or 2 GPUs per step (lane row l / 16 = GPU slot and level), and
// the partial minima are folded back onto the level's own lanes when the group ends.
//
// Pass 2: K* = the request's least key (a transposing wavefront reduction over both ranges);
// its tied cells are the lanes whose minimum equals K*, lowest first.  For each such cell the
// lanes take (request l / 4, host 4 i + l % 4) and recompute the key with the operations of
// pass 1 (hence bit-identical) in ascending host order; the first host reaching K* has the
// lowest GPU id, giving the index g * 128 + cell, and the least index over tied cells wins:
// the (key, index) lexicographic minimum.  The energy written is Lout * K*.
//
// Tiles whose requests mix TBT SLOs, or whose Lout or prompt latencies would lose precision
// in the division (a request record with a zero reciprocal), run the generic kernel's tile
// code instead; NaN is the mask value: a multiply or FMA with NaN stays NaN, v_min ignores it
// and == never matches it.
constexpr int kR = 16;                           // requests per wavefront
constexpr int kRowPad = 130 * 4;                 // bytes per decode-table row in LDS
// Workgroup LDS: the model's decode table, the power factors, the chunk's class list and the
// class-order slot of each host; then per wavefront its arrival wave's GPU records (class
// order) and the pass-2 tables.
constexpr uint32_t kL_dcs = 0;                                  // [32][130] decode table
constexpr uint32_t kL_pd = kRows * kRowPad;                     // [128] s_j * f_k^3
constexpr uint32_t kL_cls = kL_pd + 128 * 4;                    // [kClasses + 1] class list
constexpr uint32_t kL_hpos = kL_cls + (kClasses + 1) * 4 + 12;  // [kHcap] slot of chunk host i
constexpr uint32_t kL_W = kL_hpos + kHcap * 4;                  // per wavefront, kLw bytes each:
constexpr uint32_t kLw_rec = 0;                                 //   [kHcap] records, class order
constexpr uint32_t kLw_T = kHcap * 16;                          //   [kR][8] pass-2 terms
constexpr uint32_t kLw_Q = kLw_T + kR * 8 * 4;                  //   [kR] {K*, tied cell}
constexpr uint32_t kLw_M = kLw_Q + kR * 8;                      //   [kR] K*, [kR] index: the merge of
constexpr uint32_t kLw = kLw_M + kR * 8;                        //   a tile split over wavefronts
static_assert(kL_W % 16 == 0 && kLw % 16 == 0, "per-wave tables start 16-byte aligned");
__host__ __device__ constexpr size_t r16_lds_bytes(int wpb) { return kL_W + (size_t)wpb * kLw; }

__device__ __forceinline__ float bperm(uint32_t addr, float v) {
  return __int_as_float(__builtin_amdgcn_ds_bpermute((int)addr, __float_as_int(v)));
}

// The key of one candidate; pass 1 and pass 2 both evaluate exactly these operations.
__device__ __forceinline__ float r16_key(float kap, float pdp, float pdd, float tbt, float x, float p0) {
  const float Pp = fmaf(kap, pdp, p0);
  const float Y = fmaf(kap, pdd, p0) * tbt;
  return fmaf(Pp, x, Y);
}

// Request terms and power factors of one class for this lane: level jl of the lane (range
// start JB plus its row within the GPU's levels), capped at cap_pf for the prefill term and
// power and at cap_dc for the decode latency and power; a level above max(cap_pf, cap_dc)
// gets NaN power.
struct R16Class {
  float x[kR];
  float pdp, pdd;
  uint32_t mD;                   // byte offset of the decode cell within a table row
};

template <int JB>
__device__ __forceinline__ void r16_class(const char *L, int jl, int kf, int cp, int cd, const float (&xA)[kR],
                                          const float (&xB)[kR], R16Class &c) {
  const int jp = min(jl, cp), jd = min(jl, cd);
  c.pdp = jl > max(cp, cd) ? kMask : *reinterpret_cast<const float *>(L + kL_pd + (jp * 16 + kf) * 4);
  c.pdd = *reinterpret_cast<const float *>(L + kL_pd + (jd * 16 + kf) * 4);
  c.mD = (uint32_t)(jd * 16 + kf) * 4u;
  const uint32_t src = (uint32_t)((jp & 3) * 16 + kf) * 4u;
  if (JB == 0 || cp < 4) {               // the capped level lies in range A (uniform per class)
#pragma unroll
    for (int q = 0; q < kR; ++q) c.x[q] = bperm(src, xA[q]);
  } else {
#pragma unroll
    for (int q = 0; q < kR; ++q) c.x[q] = bperm(src, xB[q]);
  }
}

// One GPU's shared terms for this lane: Pp and Pd * TBT (TBT premasked: NaN above the SLO).
__device__ __forceinline__ void r16_gpu(const char *L, v4u r, const R16Class &c, float p0, float &Pp, float &Y) {
  const float kap = __uint_as_float(r.y);
  const float t = *reinterpret_cast<const float *>(L + r.x + c.mD);
  Pp = fmaf(kap, c.pdp, p0);
  Y = fmaf(kap, c.pdd, p0) * t;
}

// Pass 1 over the records [cs, ce) of one class, H GPUs per step (lane row / (4 / H) = slot).
template <int H>
__device__ __forceinline__ void r16_steps(const char *L, const char *Rw, int cs, int ce, int slot, const R16Class &c,
                                          float p0, float (&acc)[kR]) {
  constexpr bool ONE = H == 1;
  if (ONE) slot = 0;
  int i = cs;
  for (; i + H < ce; i += 2 * H) {
    const int h1 = i + H + slot;
    const v4u r0 = *reinterpret_cast<const v4u *>(Rw + (i + slot) * 16);
    v4u r1 = *reinterpret_cast<const v4u *>(Rw + (ONE ? h1 : min(h1, ce - 1)) * 16);
    if (!ONE) r1.y = h1 < ce ? r1.y : __float_as_uint(kMask);
    float Pp0, Y0, Pp1, Y1;
    r16_gpu(L, r0, c, p0, Pp0, Y0);
    r16_gpu(L, r1, c, p0, Pp1, Y1);
#pragma unroll
    for (int q = 0; q < kR; ++q) acc[q] = vmin3(acc[q], fmaf(Pp0, c.x[q], Y0), fmaf(Pp1, c.x[q], Y1));
  }
  if (i < ce) {
    const int h0 = i + slot;
    v4u r0 = *reinterpret_cast<const v4u *>(Rw + (ONE ? h0 : min(h0, ce - 1)) * 16);
    if (!ONE) r0.y = h0 < ce ? r0.y : __float_as_uint(kMask);
    float Pp0, Y0;
    r16_gpu(L, r0, c, p0, Pp0, Y0);
#pragma unroll
    for (int q = 0; q < kR; ++q) acc[q] = vmin(acc[q], fmaf(Pp0, c.x[q], Y0));
  }
}

// Pass 1 over the classes [k, ncls) of one chunk that have n levels in range JB..JB+3, where n
// = 1 (H = 4 GPUs per step), 2 (H = 2) or at least 3 (H = 1); returns the first other class.
template <int JB, int H, int S>
__device__ __forceinline__ int r16_group(const char *L, const char *Rw, int k, int ncls, int sp, const float (&xA)[kR],
                                         const float (&xB)[kR], float p0, float (&acc)[kR]) {
  constexpr int LP = 4 / H;                       // levels per GPU in a step
  const int lane = __lane_id();
  const int row = lane >> 4, kf = lane & 15;
  const int jl = JB + row % LP;
  const int slot = row / LP;
  const int *cls = reinterpret_cast<const int *>(L + kL_cls);
  for (; k < ncls; ++k) {
    const int packed = uniform(cls[k]);
    const int cp = (packed >> 3) & 7, cd = packed & 7;
    const int c0 = (packed >> 6) & 511, c1 = (packed >> 15) & 511;
    const int n = max(cp, cd) - JB + 1;           // levels of the range this class needs
    if ((H == 4 && n != 1) || (H == 2 && n != 2)) break;
    // this wavefront's part sp of the class's GPUs (S parts)
    const int cs = S == 1 ? c0 : c0 + (c1 - c0) * sp / S, ce = S == 1 ? c1 : c0 + (c1 - c0) * (sp + 1) / S;
    if (cs == ce) continue;
    R16Class c;
    r16_class<JB>(L, jl, kf, cp, cd, xA, xB, c);
    r16_steps<H>(L, Rw, cs, ce, slot, c, p0, acc);
  }
  return k;
}

// Folds a packed group's partial minima onto the lanes of the levels they belong to: with
// H = 4 rows 0-3 all hold level JB (row 0 takes the minimum of the four), with H = 2 rows
// {0, 2} and {1, 3} hold levels JB and JB + 1 (rows 0 and 1 take the pairs' minima); the
// other rows restart from +inf.  The other rows' values come by ds_bpermute (LDS pipe), so
// a fold costs 2-3 VALU instructions per accumulator.
template <int H>
__device__ __forceinline__ void r16_fold(float (&acc)[kR]) {
  const int row = __lane_id() >> 4;
#pragma unroll
  for (int q = 0; q < kR; ++q) {
    float v = acc[q];
    if (H == 4) {
      const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
      v = vmin(__uint_as_float(r[0]), __uint_as_float(r[1]));
    }
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = vmin(__uint_as_float(r[0]), __uint_as_float(r[1]));
    acc[q] = row < 4 / H ? v : kInf;
  }
}

// Pass 1 of one chunk over range JB..JB+3 (classes in ascending m, so the groups come in the
// order n = 1, 2, then more; classes with no level in the range come first and are skipped).
// The packed groups need the accumulators of the rows they borrow at +inf, which holds in
// the first chunk only: a fold takes the minimum over rows into the level's own row and
// resets the others, so in a later chunk it would move the earlier chunks' minima of the
// other levels onto the wrong cells.  Later chunks therefore score every class one GPU per
// step (a level above a class's caps gets NaN power and never wins).
template <int JB, int S>
__device__ __forceinline__ void r16_range(const char *L, const char *Rw, int ncls, int sp, const float (&xA)[kR],
                                          const float (&xB)[kR], float p0, float (&acc)[kR], bool first_chunk) {
  const int *cls = reinterpret_cast<const int *>(L + kL_cls);
  int k = 0;
  if (JB > 0)
    while (k < ncls) {
      const int packed = uniform(cls[k]);
      if (max((packed >> 3) & 7, packed & 7) >= JB) break;
      ++k;
    }
  if (first_chunk) {
    const int k1 = r16_group<JB, 4, S>(L, Rw, k, ncls, sp, xA, xB, p0, acc);
    if (k1 > k) r16_fold<4>(acc);
    k = r16_group<JB, 2, S>(L, Rw, k1, ncls, sp, xA, xB, p0, acc);
    if (k > k1) r16_fold<2>(acc);
  }
  r16_group<JB, 1, S>(L, Rw, k, ncls, sp, xA, xB, p0, acc);
}

// One value per request for the 16 requests at once: the reduction (OP) over the wavefront's
// lanes of v[q], returned in lane l for request l / 4.  Each exchange halves the values a lane
// holds: permlane32 pairs requests q and q + 8 (lanes 0-31 keep q, 32-63 keep q + 8),
// permlane16 pairs q and q + 4 (row r keeps request 4r + q), a row rotation by 8 pairs q and
// q + 2 (lane bit 3), the row half mirror pairs q and q + 1 (lane bit 2); two quad
// permutations finish each group of 4.
struct OpMinF {
  __device__ static float f(float x, float y) { return vmin(x, y); }
};
struct OpMinI {
  __device__ static int f(int x, int y) { return min(x, y); }
};
struct OpMaxI {
  __device__ static int f(int x, int y) { return max(x, y); }
};
template <typename T>
__device__ __forceinline__ unsigned bits_of(T x) {
  unsigned u;
  __builtin_memcpy(&u, &x, 4);
  return u;
}
template <typename T>
__device__ __forceinline__ T from_bits(unsigned u) {
  T x;
  __builtin_memcpy(&x, &u, 4);
  return x;
}
template <typename T>
__device__ __forceinline__ T dpp_t(T x, int) = delete;
template <int CTRL, typename T>
__device__ __forceinline__ T dppv(T x) {
  return from_bits<T>((unsigned)__builtin_amdgcn_update_dpp(0, (int)bits_of(x), CTRL, 0xf, 0xf, false));
}
template <typename OP, typename T>
__device__ __forceinline__ T wave_red16(const T (&v)[kR]) {
  T u[8], w[4], c[2];
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    const auto r = __builtin_amdgcn_permlane32_swap(bits_of(v[p]), bits_of(v[p + 8]), false, false);
    u[p] = OP::f(from_bits<T>(r[0]), from_bits<T>(r[1]));
  }
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const auto r = __builtin_amdgcn_permlane16_swap(bits_of(u[p]), bits_of(u[p + 4]), false, false);
    w[p] = OP::f(from_bits<T>(r[0]), from_bits<T>(r[1]));
  }
  const int lane = __lane_id();
  const bool b3 = (lane & 8) != 0, b2 = (lane & 4) != 0;
#pragma unroll
  for (int p = 0; p < 2; ++p) c[p] = OP::f(b3 ? w[p + 2] : w[p], dppv<kDppRor8>(b3 ? w[p] : w[p + 2]));
  T d = OP::f(b2 ? c[1] : c[0], dppv<kDppHalfMirror>(b2 ? c[0] : c[1]));
  d = OP::f(d, dppv<kDppQuad2301>(d));
  d = OP::f(d, dppv<kDppQuad1032>(d));
  return d;
}

// K* of the 16 requests: the minimum over both ranges' accumulators (lane l: request l / 4).
__device__ __forceinline__ float wave_min16(const float (&a)[kR], const float (&b)[kR]) {
  float v[kR];
#pragma unroll
  for (int q = 0; q < kR; ++q) v[q] = vmin(a[q], b[q]);
  return wave_red16<OpMinF>(v);
}

// Cell value meaning "no tied cell left" (cells are 0-127).
constexpr int kNoCell = 128;

// Wave-level LDS barrier: stores by any lane of the wavefront are visible to its loads after.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}


// A fresh copy of the lane id: a test made on it is made where it is used, not kept as a lane
// mask in scalar registers across a loop.
__device__ __forceinline__ int lane_fresh() {
  int l = __lane_id();
  asm volatile("" : "+v"(l));
  return l;
}

// Lanes 4q store request q's {K*, cell} at Qi + 8q, for the lanes' broadcast reads.
__device__ __forceinline__ void r16_store_q(char *L, uint32_t Qi, float Kl, int cellv) {
  const int lane = lane_fresh();
  if ((lane & 3) == 0) *reinterpret_cast<v2u *>(L + Qi + (lane >> 2) * 8) = v2u{__float_as_uint(Kl), (unsigned)cellv};
  wave_sync();
}

// For each request q, its least tied cell above its previous one (the cell stored at Qi + 8q;
// -1 before the first round): among the cells whose minimum equals K* (lane l of range A is
// cell l, of range B cell 64 + l), the least one above it, for every request at once by a
// wavefront min-reduction of (tied ? cell : kNoCell); an infeasible request has NaN stored as
// its K*, which no minimum equals, so it gets kNoCell.  `more` tells whether some request has
// a tied cell above the one returned (a max-reduction of the same cells).  Returns the cell in
// every lane of request q's quad.  K* and the previous cell come from LDS as broadcast reads,
// so that no per-request value occupies a scalar register.
__device__ __forceinline__ int r16_next_cells(const char *L, uint32_t Qi, const float (&accA)[kR],
                                              const float (&accB)[kR], bool &more) {
  const int lane = __lane_id();
  int lo[kR], hi[kR];
#pragma unroll
  for (int q = 0; q < kR; ++q) {
    const v2u qi = *reinterpret_cast<const v2u *>(L + Qi + q * 8);
    const float K = __uint_as_float(qi.x);
    const int pv = (int)qi.y;
    const int ca = accA[q] == K && lane > pv ? lane : kNoCell;
    const int cb = accB[q] == K && 64 + lane > pv ? 64 + lane : kNoCell;
    lo[q] = min(ca, cb);
    hi[q] = max(ca == kNoCell ? -1 : ca, cb == kNoCell ? -1 : cb);
  }
  const int c = wave_red16<OpMinI>(lo);
  const int top = wave_red16<OpMaxI>(hi);
  more = __ballot(c < kNoCell && top > c) != 0ull;
  return c;
}

constexpr int kWpb16 = 4;                        // wavefronts per workgroup of the 8 x 16 kernel

// S = wavefronts per tile: with S > 1 (small request counts, too few tiles to fill the chip)
// the S wavefronts of a tile split each SM-cap class's GPUs into S parts in pass 1, merge the
// least key per request through LDS, each finds the lowest index reaching it among its own
// tied cells (over all GPUs), and the least index is merged the same way.
template <int S>
__global__ void __launch_bounds__(kWpb16 * 64) k_score_r16(PlaceArgs a) {
  constexpr int WPB = kWpb16, TPB = WPB / S;     // tiles per workgroup
  extern __shared__ __align__(16) float lds[];
  __shared__ int s_ok[WPB];
  char *L = reinterpret_cast<char *>(lds);
  constexpr int T = WPB * 64;
  // Workgroup t takes tiles [TPB t, TPB t + TPB) of the table, all of one (model, prompt
  // kind) group: the tiles of a group are contiguous and padded to a multiple of TPB, so the
  // first is never empty.  Wavefront v scores part v % S of tile TPB t + v / S: up to kR
  // requests of one (arrival wave, model) bucket.
  // XCD-aware order: workgroups are dealt to the 8 XCDs round-robin, so XCD x takes the
  // contiguous range [x * per, (x + 1) * per) -- the same models -- instead of every eighth.
  const int nblk = *ro(a.n_tiles) / TPB;
  const int per = (nblk + kXcds - 1) / kXcds;
  const int idx = blockIdx.x / kXcds;
  const int t = (blockIdx.x % kXcds) * per + idx;
  if (idx >= per || t >= nblk) return;
  const auto tp = ro(reinterpret_cast<const int32_t *>(a.tiles));
  const int beg = tp[2 * TPB * t + 1];    // the workgroup's first request
  const int b0 = tp[2 * TPB * t];         // the workgroup's first bucket
  const BucketId grp = bucket_id(a, b0);
  const int m = grp.m;
  const int wv = uniform(threadIdx.x >> 6);
  const int ti = wv / S, sp = wv - ti * S;  // this wavefront's tile and part
  const int bk = tp[2 * (TPB * t + ti)];  // the tile's bucket (-1: an empty tile)
  const int q0 = bk >= 0 ? tp[2 * (TPB * t + ti) + 1] : beg;
  const int nq = bk >= 0 ? min(kR, ro(a.bstart)[bk + 1] - q0) : 0;
  const int w = bk >= 0 ? grp.w + (bk - b0) : 0;   // the group's buckets are consecutive waves
  if (grp.noprompt) {                     // prompt-less requests: TTFT from the batch row
    score_requests_generic<2, 16>(a, m, true, w, q0 + sp * kQ, q0 + nq, S * kQ, lds);
    return;
  }
  // Staging waits on memory and barriers while other workgroups' pass 1 keeps the VALU busy:
  // at a raised wavefront priority its instructions issue first.
  __builtin_amdgcn_s_setprio(2);
  const int lane = threadIdx.x & (kWave - 1);
  // One round trip for everything that needs only the model and the tile entries, all loads
  // into registers before any LDS store (a store between loads would order them): the
  // model's decode table, the power factors, the first host chunk's GPU ids and class slots
  // (kHk per lane: this wavefront's part of its tile's records), the chunk's class list and
  // the requests.  Lane l holds the fields of request l / 4, read at the tile's position
  // clamped into the request array (a missing request is masked below).
  constexpr int kDcV = kRows * 128 / 4 / T;        // float4 of the decode table per thread
  constexpr int kHk = kHcap >= S * kWave ? kHcap / (S * kWave) : 1;   // chunk hosts per lane
  const float *dsrc = a.dc + (size_t)m * kRows * 128;
  const bool dc_al = (((uintptr_t)dsrc) & 15) == 0;
  float4 dcv[kDcV];
  if (dc_al) {
#pragma unroll
    for (int u = 0; u < kDcV; ++u) dcv[u] = reinterpret_cast<const float4 *>(dsrc)[threadIdx.x + u * T];
  }
  const float pdv = a.sm_level[(threadIdx.x >> 4) & 7] * cube(a.freq_level[threadIdx.x & 15]);   // cell tid % 128
  int hl[kHk], hp[kHk];
#pragma unroll
  for (int k = 0; k < kHk; ++k) {
    const int i = (k * S + sp) * kWave + lane;     // chunk-0 host of this lane
    hl[k] = i < a.G ? a.host_list[(size_t)m * (unsigned)a.G + i] : 0;
    hp[k] = i < a.G ? a.host_pos[(size_t)m * (unsigned)a.G + i] : 0;
  }
  const int clsv = a.cls_tab[(size_t)m * a.nch * (kClasses + 1) + min((int)threadIdx.x, kClasses)];
  const bool has = (lane >> 2) < nq;
  const ReqRec rq = load_req_lane(a, min(q0 + (lane >> 2), a.R - 1));
  float lo_has = has ? rq.lout : 0.f;
  // the request's prompt-row offset, TTFT SLO and 1 / Lout for the request-term staging
  // (a missing request: row 0, SLO -inf, so every term is masked)
  v4u stage_rec = v4u{(unsigned)((m * kRows + (has ? rq.row : 0)) * 128),
                      has ? __float_as_uint(rq.slo_ttft) : __float_as_uint(-kInf),
                      has ? __float_as_uint(rq.rlout) : __float_as_uint(1.f), 0u};
  // made here, not at their uses: the lane mask `has` is then dead before pass 1
  asm volatile("" : "+v"(lo_has), "+v"(stage_rec));
  const ReqRec r0 = load_req(a, beg);     // the workgroup's first request (scalar)
  {
    const bool ok = !has || (rq.rlout > 0.f && __float_as_int(rq.slo_tbt) == __float_as_int(r0.slo_tbt));
    const unsigned long long bad = __ballot(!ok);
    if (lane == 0) s_ok[wv] = bad == 0ull;
  }
  __syncthreads();
  bool tile_ok = true;
#pragma unroll
  for (int v = 0; v < WPB; ++v) tile_ok = tile_ok && s_ok[v];
  if (!tile_ok) {                         // mixed TBT SLOs or an unscalable request
    score_requests_generic<2, 16>(a, m, false, w, q0 + sp * kQ, q0 + nq, S * kQ, lds);
    return;
  }
  const float tsb = r0.slo_tbt;           // every request of the workgroup has this TBT SLO
  const int hcnt = ro(a.host_cnt)[m];
  const int n0 = min(kHcap, hcnt);

  float xA[kR], xB[kR];
  const uint32_t Wb = kL_W + (uint32_t)wv * kLw;   // this wavefront's tables
  const uint32_t Tw = Wb + kLw_T;
  const uint32_t Wt = kL_W + (uint32_t)(ti * S) * kLw;   // the tile's shared tables
  const char *Rw = L + Wt + kLw_rec;
  float *Km = reinterpret_cast<float *>(L + Wt + kLw_M);   // merged K* of the tile's requests
  int *Bm = reinterpret_cast<int *>(L + Wt + kLw_M + kR * 4);   // merged least index
  // Second round trip: the request terms x = TTFT / Lout (NaN where TTFT misses the SLO) at
  // this lane's cell of each range for the 16 requests, each request's row offset, SLO and
  // 1 / Lout taken from its lane by ds_bpermute; and the GPU records of the chunk's hosts.
  HostRec hr0[kHk];
  if (nq > 0) {
#pragma unroll
    for (int q = 0; q < kR; ++q) {
      const unsigned off = (unsigned)__builtin_amdgcn_ds_bpermute(q * 16, (int)stage_rec.x);
      xA[q] = a.pf[off + lane];
      xB[q] = a.pf[off + 64 + lane];
    }
#pragma unroll
    for (int k = 0; k < kHk; ++k) {
      const int i = (k * S + sp) * kWave + lane;
      if (i < n0) hr0[k] = a.recs[(size_t)w * (unsigned)a.G + hl[k]];
    }
#pragma unroll
    for (int q = 0; q < kR; ++q) {
      const float st = bperm(q * 16, __uint_as_float(stage_rec.y)), rl = bperm(q * 16, __uint_as_float(stage_rec.z));
      xA[q] = xA[q] < st ? xA[q] * rl : kMask;
      xB[q] = xB[q] < st ? xB[q] * rl : kMask;
    }
  }
  // LDS: the power factors, the decode table (rows padded to kRowPad bytes, NaN where TBT
  // misses the SLO), the chunk's class list and host slots, the tile's records (class order)
  // (the thread-index tests below are made here, on a fresh copy, not kept as lane masks)
  int tid = (int)threadIdx.x;
  asm volatile("" : "+v"(tid));
  if (tid < 128) *reinterpret_cast<float *>(L + kL_pd + tid * 4) = pdv;
  if ((((uintptr_t)(a.dc + (size_t)fresh_s(m) * kRows * 128)) & 15) == 0) {   // dc_al, decided afresh
#pragma unroll
    for (int u = 0; u < kDcV; ++u) {
      const int i = threadIdx.x + u * T;
      const float4 v = dcv[u];
      v2f *d = reinterpret_cast<v2f *>(L + kL_dcs + (i >> 5) * kRowPad + (i & 31) * 16);
      d[0] = v2f{v.x < tsb ? v.x : kMask, v.y < tsb ? v.y : kMask};
      d[1] = v2f{v.z < tsb ? v.z : kMask, v.w < tsb ? v.w : kMask};
    }
  } else {
    for (int i = threadIdx.x; i < kRows * 128; i += T) {
      const float v = dsrc[i];
      *reinterpret_cast<float *>(L + kL_dcs + (i >> 7) * kRowPad + (i & 127) * 4) = v < tsb ? v : kMask;
    }
  }
  if (tid <= kClasses) reinterpret_cast<int *>(L + kL_cls)[tid] = clsv;
#pragma unroll
  for (int k = 0; k < kHk; ++k) {
    const int i = (k * S + sp) * kWave + lane;
    if (ti == 0 && i < n0) reinterpret_cast<int *>(L + kL_hpos)[i] = hp[k];
    if (nq > 0 && i < n0) {
      v4u e;
      e.x = kL_dcs + (uint32_t)(max(hr0[k].row_off, 0) / 128) * kRowPad;
      e.y = __float_as_uint(hr0[k].kappa);
      e.z = (uint32_t)hl[k];
      e.w = (uint32_t)hr0[k].caps;
      *reinterpret_cast<v4u *>(L + Wt + kLw_rec + hp[k] * 16) = e;
    }
  }
  if (S > 1 && sp == 0 && lane < kR) {    // made ready before the first pass-1 barrier
    Km[lane] = kInf;
    Bm[lane] = INT_MAX;
  }

  float accA[kR], accB[kR];
#pragma unroll
  for (int q = 0; q < kR; ++q) accA[q] = accB[q] = kInf;
  const float p0 = a.p0;
  for (int c0 = 0, ch = 0; c0 < hcnt; c0 += kHcap, ++ch) {
    const int n = min(kHcap, hcnt - c0);
    if (ch > 0) {                         // later chunks (more than kHcap GPUs host the model)
      __syncthreads();                    // the previous chunk's records are no longer read
      __builtin_amdgcn_s_setprio(2);
      const size_t mg = (size_t)fresh_s(m) * (unsigned)a.G + c0, wg = (size_t)fresh_s(w) * (unsigned)a.G;
      for (int i = threadIdx.x; i < n; i += T)   // class-order slot of each chunk host
        reinterpret_cast<int *>(L + kL_hpos)[i] = a.host_pos[mg + i];
      if (nq > 0)
        for (int i = sp * kWave + lane; i < n; i += S * kWave) {   // the tile's GPU records, class order
          const int g = a.host_list[mg + i];
          const int pos = a.host_pos[mg + i];
          const HostRec h = a.recs[wg + g];
          v4u e;
          e.x = kL_dcs + (uint32_t)(max(h.row_off, 0) / 128) * kRowPad;
          e.y = __float_as_uint(h.kappa);
          e.z = (uint32_t)g;
          e.w = (uint32_t)h.caps;
          *reinterpret_cast<v4u *>(L + Wt + kLw_rec + pos * 16) = e;
        }
      for (int i = threadIdx.x; i <= kClasses; i += T)
        reinterpret_cast<int *>(L + kL_cls)[i] = a.cls_tab[((size_t)fresh_s(m) * a.nch + ch) * (kClasses + 1) + i];
    }
    __syncthreads();
    __builtin_amdgcn_s_setprio(0);
    if (nq > 0) {
      const int ncls = uniform(reinterpret_cast<const int *>(L + kL_cls)[kClasses]);
      r16_range<0, S>(L, Rw, ncls, sp, xA, xB, p0, accA, ch == 0);
      r16_range<4, S>(L, Rw, ncls, sp, xA, xB, p0, accB, ch == 0);
    }
  }
  if (S == 1 && nq == 0) return;          // (with S > 1 every wavefront meets the barriers below)

  // pass 2: per request the least key K* and, per tied cell in ascending order, the first host
  // (ascending GPU id) reaching it
  float Kl = wave_min16(accA, accB);                // request lane / 4
  if (S > 1) {                            // K* over the tile's S parts
    if (nq > 0 && (lane_fresh() & 3) == 0) atomicMin(&Km[lane >> 2], Kl);
    __syncthreads();
    Kl = Km[lane >> 2];
  }
  // Lout of request lane / 4, 0 for a missing request (tested as a vector value so that no
  // lane mask stays live in scalar registers across pass 1)
  const float lo_l = lo_has;
  const float Ks = lo_l > 0.f && Kl < kInf && lo_l * Kl < kInf ? Kl : kMask;   // NaN: infeasible
  const bool recs_in_lds = hcnt <= kHcap;                     // T[q][j] at Tw + (8q + j) * 4
  const uint32_t Qi = Wb + kLw_Q;                             // {K*, cell} of request q at Qi + 8q
  int best = INT_MAX;                                         // lanes of request q: its least index
  bool more;
  r16_store_q(L, Qi, Ks, -1);
  int cellv = r16_next_cells(L, Qi, accA, accB, more);
  while (nq > 0 && __ballot(cellv < kNoCell) != 0ull) {
    r16_store_q(L, Qi, Ks, cellv);
    // T[q][j] = request q's term at level j and its tied cell's frequency level: lanes j < 8
    // read lane (j % 4) * 16 + k of xA[q] (j < 4) or xB[q]; every request at once.  The
    // cell comes from lane 4q by readlane and every permute is issued before the first store
    // (a cell read back from LDS would wait behind the previous request's store).
    float tv[kR];
#pragma unroll
    for (int q = 0; q < kR; ++q) {
      const int ck = __builtin_amdgcn_readlane(cellv, 4 * q) & 15;
      const uint32_t src = (uint32_t)((lane & 3) * 16 + ck) * 4u;
      const float xa = bperm(src, xA[q]), xb = bperm(src, xB[q]);
      tv[q] = lane < 4 ? xa : xb;
    }
    if (lane < 8) {
#pragma unroll
      for (int q = 0; q < kR; ++q) *reinterpret_cast<float *>(L + Tw + (q * 8 + lane) * 4) = tv[q];
    }
    wave_sync();
    // Lanes take 64 hosts at a time in ascending order; each pending request is evaluated at
    // its tied cell on all of them (four requests at a time, their LDS reads together), and
    // its first matching lane is its lowest GPU id, so a request is done at the first block
    // with a match.
    unsigned long long pend = __ballot((lane_fresh() & 3) == 0 && cellv < kNoCell);   // bit 4q: request q
    for (int b0 = 0; b0 < hcnt && pend != 0ull; b0 += kWave) {
      asm volatile("" ::: "memory");      // per-request values are reloaded in every block
      const int i = b0 + lane;
      const bool valid = i < hcnt;
      const int ic = valid ? i : hcnt - 1;
      uint32_t rowB;
      float kap;
      int g, caps;
      if (recs_in_lds) {
        const int slot = reinterpret_cast<const int *>(L + kL_hpos)[ic];
        const v4u r = *reinterpret_cast<const v4u *>(Rw + slot * 16);
        rowB = r.x;
        kap = __uint_as_float(r.y);
        g = (int)r.z;
        caps = (int)r.w;
      } else {
        g = a.host_list[(size_t)fresh_s(m) * (unsigned)a.G + ic];
        const HostRec hr = a.recs[(size_t)fresh_s(w) * (unsigned)a.G + g];
        rowB = kL_dcs + (uint32_t)(max(hr.row_off, 0) / 128) * kRowPad;
        kap = hr.kappa;
        caps = hr.caps;
      }
      const int cp = caps & 0xff, cd = (caps >> 8) & 0xff, mx = max(cp, cd);
#pragma unroll
      for (int q0 = 0; q0 < kR; q0 += 4) {
        if (((pend >> (4 * q0)) & 0x1111ull) == 0ull) continue;
        unsigned long long mk[4];
        int cq[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int q = q0 + t;
          // request q's K* and tied cell, wave-uniform: read from its lane into scalar
          // registers, so the cell's level, frequency and offsets are scalar arithmetic
          const float K = __uint_as_float(__builtin_amdgcn_readlane(__float_as_uint(Ks), 4 * q));
          const int c = __builtin_amdgcn_readlane(cellv, 4 * q);
          cq[t] = c;
          const int cj = c >> 4, ck4 = (c & 15) * 4;
          const int jp = min(cj, cp), jd = min(cj, cd);
          const float pdp = *reinterpret_cast<const float *>(L + kL_pd + ck4 + jp * 64);
          const float pdd = *reinterpret_cast<const float *>(L + kL_pd + ck4 + jd * 64);
          const float tbt = *reinterpret_cast<const float *>(L + rowB + (uint32_t)(ck4 + jd * 64));
          const float x = *reinterpret_cast<const float *>(L + Tw + (uint32_t)(q * 32 + jp * 4));
          // a cell above max(cap_pf, cap_dc) repeats a lower cell of the same GPU: pass 1 gave
          // it NaN power, so it never matches; the ballot is taken here, from the compares'
          // own masks
          mk[t] = __ballot(valid && cj <= mx && r16_key(kap, pdp, pdd, tbt, x, p0) == K);
        }
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int q = q0 + t;
          if (((pend >> (4 * q)) & 1ull) && mk[t] != 0ull) {
            const int first = __builtin_ctzll(mk[t]);
            const int gw = __builtin_amdgcn_readlane(g, first);
            // the lane test on a fresh lane id: made here, not kept as 16 lane masks in
            // scalar registers through pass 2
            best = (lane_fresh() >> 2) == q ? min(best, gw * 128 + cq[t]) : best;
            pend &= ~(1ull << (4 * q));
          }
        }
      }
    }
    if (!more) break;
    cellv = r16_next_cells(L, Qi, accA, accB, more);
    wave_sync();                          // T is rewritten next round
  }
  if (S > 1) {                            // the least index over the tile's S parts
    if (nq > 0 && (lane_fresh() & 3) == 0 && best != INT_MAX) atomicMin(&Bm[lane >> 2], best);
    __syncthreads();
    best = Bm[lane >> 2];
  }
  // fresh copies of the lane id and Lout: tests on them are made here, not kept as lane masks
  // in scalar registers through pass 2
  const int ln = lane_fresh();
  float lo_w = lo_l;
  asm volatile("" : "+v"(lo_w));
  if (sp == 0 && (ln & 3) == 0 && lo_w > 0.f) {
    const bool found = best != INT_MAX;
    a.choice[rq.r] = found ? best : -1;
    a.feasible[rq.r] = found ? 1 : 0;
    a.energy[rq.r] = found ? lo_l * Kl : kInf;
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
  size_t cnt, bstart, ntiles, tiles, gscan, host_cnt, host_list, recs, preq, key, off;
  size_t host_pos, cls_tab, pf_rowmin, pf_rowtiny, dc_min, total;
  int32_t NB, tile, max_tiles, waves_per_block, nch, gpad;
  int32_t gw, ng;                // buckets per group and groups
  int32_t split;                 // 8 x 16 kernel: wavefronts per tile (1, 2 or 4)
  bool fast;                     // 8 SM x 16 frequency levels: the specialised kernel
  bool scan_local;               // k_scatter scans the bucket counts (no k_scan launch)
  size_t scatter_lds;            // dynamic LDS bytes of k_scatter
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
  // arrival-wave slabs: the largest divisor of W up to kXcds, gw waves each
  int slabs = 1;
  for (int d = kXcds; d > 1; --d)
    if (W % d == 0) {
      slabs = d;
      break;
    }
  const long long gw = W / slabs, ng = 2 * M * slabs;
  if (NB > INT_MAX / 2 - 4 || Gn * C > INT_MAX || W * Gn > INT_MAX || M * Gn > INT_MAX) return false;
  // tile size: large tiles amortise the table staging, small ones fill the chip
  const bool fast = L->n_sm == 8 && L->n_freq == 16;
  int wpb = 4, tile, split = 1;
  if (fast) {                    // tiles of kR requests, S wavefronts each
    tile = kR;
    wpb = kWpb16;
    // too few tiles for four wavefronts per SIMD: split each tile's GPUs over 2 or 4
    const long long tiles = (R + kR - 1) / kR;
    split = tiles <= 1024 ? 4 : (tiles <= 2048 ? 2 : 1);
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
  // the 8 x 16 kernel's workgroups take wpb / split tiles of one (model, prompt kind) group:
  // each of the ng groups is padded with fewer empty tiles than that
  const int gpad = fast ? wpb / split : 1;
  const long long max_tiles = (R + tile - 1) / tile + NB + (long long)(gpad - 1) * ng;
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
  o->gscan = take(sizeof(int32_t) * (gpad > 1 ? 2 * (ng + 1) : 1));
  o->host_cnt = take(sizeof(int32_t) * M);
  o->host_list = take(sizeof(int32_t) * M * Gn);
  o->recs = take(sizeof(HostRec) * W * Gn);
  o->preq = take(sizeof(ReqRec) * (R > 0 ? R : 1));
  o->key = take(sizeof(int32_t) * (R > 0 ? R : 1));
  o->off = take(sizeof(int32_t) * (R > 0 ? R : 1));
  const long long nch = fast ? (Gn + kHcap - 1) / kHcap : 0;
  o->host_pos = take(sizeof(int32_t) * (fast ? M * Gn : 1));
  o->cls_tab = take(sizeof(int32_t) * (fast ? M * nch * (kClasses + 1) : 1));
  o->pf_rowmin = take(sizeof(float) * M * kRows);
  o->pf_rowtiny = take(sizeof(float) * M * kRows);
  o->dc_min = take(sizeof(float) * M);
  o->total = off;
  o->nch = (int32_t)nch;
  o->NB = (int32_t)NB;
  o->gw = (int32_t)gw;
  o->ng = (int32_t)ng;
  static_assert((kR & (kR - 1)) == 0 && (kQ & (kQ - 1)) == 0, "tile sizes are powers of two");
  o->tile = tile;                       // a power of two: the bucket scans shift by its log2
  o->max_tiles = (int32_t)max_tiles;
  o->waves_per_block = wpb;
  o->gpad = gpad;
  o->split = split;
  const long long scan_ints = block_scan_ints(NB, ng, gpad > 1);
  o->scan_local = NB <= kHistMax && scan_ints <= kScanLds;
  o->scatter_lds = o->scan_local ? sizeof(int32_t) * (size_t)scan_ints : 0;
  return true;
}

// A caller's event recorded on the stream (the timed entry points); nullptr: nothing.
hipError_t mark(void *ev, hipStream_t st) {
  return ev ? hipEventRecord(static_cast<hipEvent_t>(ev), st) : hipSuccess;
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

// The launches of one placement call on a checked workspace of lay.total bytes; ev_begin /
// ev_end (the timed entry point, else nullptr) are recorded around the scoring kernel.
festina_status place_launch(const festina_lut *L, const festina_gpus *G, const festina_requests *Q,
                            const festina_placements *out, const PlaceLayout &lay, char *ws, void *stream,
                            void *ev_begin = nullptr, void *ev_end = nullptr) {
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
  a.gw = lay.gw;
  a.ng = lay.ng;
  a.tile = lay.tile;
  a.max_tiles = lay.max_tiles;
  a.gpad = lay.gpad;
  a.scan_local = lay.scan_local ? 1 : 0;
  a.cnt = reinterpret_cast<int32_t *>(ws + lay.cnt);
  const int nb4 = (lay.NB + 3) & ~3;      // counters padded with zeros to whole int4
  a.bstart = reinterpret_cast<int32_t *>(ws + lay.bstart);
  a.n_tiles = reinterpret_cast<int32_t *>(ws + lay.ntiles);
  a.tiles = reinterpret_cast<int2 *>(ws + lay.tiles);
  a.gscan = reinterpret_cast<int32_t *>(ws + lay.gscan);
  a.host_cnt = reinterpret_cast<int32_t *>(ws + lay.host_cnt);
  a.host_list = reinterpret_cast<int32_t *>(ws + lay.host_list);
  a.recs = reinterpret_cast<HostRec *>(ws + lay.recs);
  a.preq = reinterpret_cast<ReqRec *>(ws + lay.preq);
  a.key = reinterpret_cast<int32_t *>(ws + lay.key);
  a.off = reinterpret_cast<int32_t *>(ws + lay.off);
  a.fast = lay.fast ? 1 : 0;
  a.nch = lay.nch;
  a.host_pos = reinterpret_cast<int32_t *>(ws + lay.host_pos);
  a.cls_tab = reinterpret_cast<int32_t *>(ws + lay.cls_tab);
  a.pf_rowmin = reinterpret_cast<float *>(ws + lay.pf_rowmin);
  a.pf_rowtiny = reinterpret_cast<float *>(ws + lay.pf_rowtiny);
  a.dc_min = reinterpret_cast<float *>(ws + lay.dc_min);

  hipStream_t st = static_cast<hipStream_t>(stream);
  int zb = (nb4 + 255) / 256;
  zb = zb < 1024 ? zb : 1024;
  k_init<<<zb + 9 * a.M, 256, 0, st>>>(a, zb, nb4);
  if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  const int nbr = (a.R + kReqPerPrepBlock - 1) / kReqPerPrepBlock;
  const long long nrec = ((long long)a.W * a.G + kPrepBlock - 1) / kPrepBlock;
  k_prep<<<(unsigned)(nbr + a.M + nrec), kPrepBlock, 0, st>>>(a, nbr);
  if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  if (!lay.scan_local) {
    k_scan<<<1, 1024, lay.NB <= kScanLds ? sizeof(int) * lay.NB : 0, st>>>(a);
    if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  }
  k_scatter<<<nbr, kPrepBlock, lay.scatter_lds, st>>>(a);
  if (hipGetLastError() != hipSuccess) return FESTINA_ERR_DEVICE;
  const int cpl = C <= 64 ? 1 : (C <= 128 ? 2 : 4);
  const int wpb = lay.waves_per_block;
  size_t lds = sizeof(float) * score_lds_floats((int)C, cpl, wpb);
  if (lay.fast) {
    const size_t f = r16_lds_bytes(wpb);
    lds = f > lds ? f : lds;
  }
  hipError_t e = mark(ev_begin, st);
  if (e != hipSuccess) return FESTINA_ERR_DEVICE;
  if (lay.fast) {
    const int blocks = (lay.max_tiles + lay.gpad - 1) / lay.gpad;
    const int grid = (blocks + kXcds - 1) / kXcds * kXcds;
    if (lay.split == 4)
      k_score_r16<4><<<grid, kWpb16 * kWave, lds, st>>>(a);
    else if (lay.split == 2)
      k_score_r16<2><<<grid, kWpb16 * kWave, lds, st>>>(a);
    else
      k_score_r16<1><<<grid, kWpb16 * kWave, lds, st>>>(a);
    e = hipGetLastError();
  } else if (cpl == 1)
    e = launch_score<1>(a, lay.max_tiles, wpb, lds, st);
  else if (cpl == 2)
    e = launch_score<2>(a, lay.max_tiles, wpb, lds, st);
  else
    e = launch_score<4>(a, lay.max_tiles, wpb, lds, st);
  if (e == hipSuccess) e = mark(ev_end, st);
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

festina_status festina_score_placements_timed(const festina_lut *L, const festina_gpus *G,
                                              const festina_requests *Q, festina_placements *out,
                                              void *workspace, size_t workspace_bytes, void *stream,
                                              void *score_begin, void *score_end) {
  PlaceLayout lay;
  const festina_status s = place_args(L, G, Q, out, &lay);
  if (s != FESTINA_OK || Q->n_requests == 0) return s;
  if (!workspace || workspace_bytes < lay.total || (((uintptr_t)workspace) & 255) != 0)
    return FESTINA_ERR_INVALID;
  return place_launch(L, G, Q, out, lay, static_cast<char *>(workspace), stream, score_begin, score_end);
}

festina_status festina_score_placements(const festina_lut *L, const festina_gpus *G,
                                        const festina_requests *Q, festina_placements *out,
                                        void *workspace, size_t workspace_bytes, void *stream) {
  return festina_score_placements_timed(L, G, Q, out, workspace, workspace_bytes, stream, nullptr, nullptr);
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

festina_status festina_score_migrations_timed(const festina_lut *L, const festina_fleet *F,
                                              festina_migrations *out, void *workspace,
                                              size_t workspace_bytes, void *stream, void *pairs_begin,
                                              void *pairs_end) {
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
  if (mark(pairs_begin, st) != hipSuccess) return FESTINA_ERR_DEVICE;
  k_migrate<<<(a.G + kMigSrcPerBlock - 1) / kMigSrcPerBlock, 256, 0, st>>>(a);
  if (hipGetLastError() != hipSuccess || mark(pairs_end, st) != hipSuccess) return FESTINA_ERR_DEVICE;
  return FESTINA_OK;
}

festina_status festina_score_migrations(const festina_lut *L, const festina_fleet *F,
                                        festina_migrations *out, void *workspace,
                                        size_t workspace_bytes, void *stream) {
  return festina_score_migrations_timed(L, F, out, workspace, workspace_bytes, stream, nullptr, nullptr);
}

}  // extern "C"
