// transfer.hip -- MI355X (gfx950) kernels and C-ABI host dispatch of the transfer plan that
// follows a reconfiguration (Festina, App. F): the cost matrix of the device mapping and the
// per-request choice to finish in place or move.
//
// k_transfer_costs  e_uv = Bytes(u -> v) / BW(u, v) for every ordered pair, written as a
//   dense [G][G] float32 matrix (the input of the minimum-cost assignment).  Bytes = u's
//   request state plus the weights of u's resident models that v lacks; e_uu = 0; BW is
//   the intra-node link inside a node, else the inter-node one.  A block owns a stretch of
//   row u (u's residency and state are wave-uniform); each thread makes two groups of four
//   consecutive entries from the set bits of (u's models & ~v's models) and stores each as
//   one 16-byte vector, so the kernel is a coalesced stream of stores.
// k_request_moves   one thread per in-flight request: remaining decode time at the source
//   against token transfer plus the faster of KV-cache transfer and recompute on the
//   destination of the plan.
//
// Exactness: byte counts are integers; times are float64 (bytes * ms_per_byte, with
// ms_per_byte = 1e3 / (GB/s * 1e9) formed on the host), so every comparison is decided on
// the same values as any float64 evaluation in that order, and the costs are those values
// rounded to float32.
#include <hip/hip_runtime.h>

#include <climits>
#include <cstddef>
#include <cstdint>

#include "festina.h"

namespace {

constexpr int kRows = FESTINA_N_ROWS;
constexpr int kCostBlock = 256;
constexpr int kMoveBlock = 256;

struct CostArgs {
  int32_t G, M, words;
  const uint32_t *resident;
  const int32_t *weights, *state, *node;
  double mpb_intra, mpb_inter;           // ms per byte
  float *cost;
};

// Cost of sending u's state (state_mib, residency word pointer ru) to v.
__device__ __forceinline__ float pair_cost(const CostArgs &a, int u, int v, long long state, int node_u,
                                           const uint32_t *ru) {
  if (v == u) return 0.f;
  long long mib = state;
  for (int w = 0; w < a.words; ++w) {
    unsigned bits = ru[w] & ~a.resident[(size_t)v * a.words + w];     // u's models that v lacks
    while (bits) {
      const int m = w * 32 + __builtin_ctz(bits);
      bits &= bits - 1;
      if (m < a.M) mib += a.weights[m];
    }
  }
  const double mpb = a.node[v] == node_u ? a.mpb_intra : a.mpb_inter;
  return (float)((double)(mib * 1048576) * mpb);
}

// Thread t of a block makes entries v = base + 4t .. 4t+3 and base + 4(t + kCostBlock) ..
// of row u: kCostVecs 16-byte stores per thread, each coalesced across the block.
constexpr int kCostVecs = 2;

__global__ void __launch_bounds__(kCostBlock) k_transfer_costs(CostArgs a, int32_t blocks_per_row, int32_t vec) {
  const int u = blockIdx.x / blocks_per_row;
  const int part = blockIdx.x - u * blocks_per_row;
  const long long state = a.state[u];
  const int node_u = a.node[u];
  const uint32_t *ru = a.resident + (size_t)u * a.words;
  float *row = a.cost + (size_t)u * a.G;
  const int base = part * kCostBlock * 4 * kCostVecs;
#pragma unroll
  for (int c = 0; c < kCostVecs; ++c) {
    const int v0 = base + (c * kCostBlock + threadIdx.x) * 4;
    if (v0 >= a.G) break;
    float e[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) e[q] = v0 + q < a.G ? pair_cost(a, u, v0 + q, state, node_u, ru) : 0.f;
    if (vec && v0 + 3 < a.G) {
      *reinterpret_cast<float4 *>(row + v0) = make_float4(e[0], e[1], e[2], e[3]);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (v0 + q < a.G) row[v0 + q] = e[q];
    }
  }
}

// Fleets of at most 32 models with rows of whole 16-byte vectors: u's models are walked as
// a wave-uniform bit loop, and per destination a model costs one bit test, a select and a
// float64 add (byte counts are whole MiB, exact in float64); e = MiB * (2^20 * ms_per_byte),
// the same value as bytes * ms_per_byte since scaling by 2^20 is exact.
__global__ void __launch_bounds__(kCostBlock) k_transfer_costs_w1(CostArgs a, int32_t blocks_per_row) {
  const int u = blockIdx.x / blocks_per_row;
  const int part = blockIdx.x - u * blocks_per_row;
  const double state = (double)a.state[u];
  const int node_u = a.node[u];
  const unsigned cu = __builtin_amdgcn_readfirstlane(a.resident[u]);
  const double mib_intra = a.mpb_intra * 1048576.0, mib_inter = a.mpb_inter * 1048576.0;
  float *row = a.cost + (size_t)u * a.G;
  const int base = part * kCostBlock * 4 * kCostVecs;
#pragma unroll
  for (int c = 0; c < kCostVecs; ++c) {
    const int v0 = base + (c * kCostBlock + threadIdx.x) * 4;
    if (v0 >= a.G) break;
    const uint4 cv = *reinterpret_cast<const uint4 *>(a.resident + v0);
    const int4 nv = *reinterpret_cast<const int4 *>(a.node + v0);
    double acc[4] = {state, state, state, state};
    for (unsigned bits = cu; bits; bits &= bits - 1) {          // u's models, wave-uniform
      const int m = __builtin_ctz(bits);
      if (m >= a.M) break;
      const double w = (double)a.weights[m];
      acc[0] += ((cv.x >> m) & 1u) ? 0.0 : w;
      acc[1] += ((cv.y >> m) & 1u) ? 0.0 : w;
      acc[2] += ((cv.z >> m) & 1u) ? 0.0 : w;
      acc[3] += ((cv.w >> m) & 1u) ? 0.0 : w;
    }
    const int nvv[4] = {nv.x, nv.y, nv.z, nv.w};
    float e[4];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      e[q] = v0 + q == u ? 0.f : (float)(acc[q] * (nvv[q] == node_u ? mib_intra : mib_inter));
    // streaming store: the matrix is written once and not read back by this kernel
    typedef float v4f __attribute__((ext_vector_type(4)));
    __builtin_nontemporal_store(v4f{e[0], e[1], e[2], e[3]}, reinterpret_cast<v4f *>(row + v0));
  }
}

struct MoveArgs {
  int32_t M, NS, NF, C, G, Q;
  const float *pf, *dc;
  const int32_t *node;
  double mpb_intra, mpb_inter;
  const int32_t *dest, *freq_cur, *sm_cur, *batch;
  const int32_t *src, *model, *ctx, *rem, *kv_kib, *tok_kib;
  int32_t *decision;
  float *remaining_ms, *migrate_ms;
};

// ms for `bytes` over the link u -> v, one rounding per operation.
__device__ __forceinline__ double link_ms(long long bytes, double mpb) {
#pragma clang fp contract(off)
  return (double)bytes * mpb;
}

__global__ void __launch_bounds__(kMoveBlock) k_request_moves(MoveArgs a) {
#pragma clang fp contract(off)
  const int q = blockIdx.x * kMoveBlock + threadIdx.x;
  if (q >= a.Q) return;
  int dec = -1;
  double rem_ms = 0.0, mig_ms = 0.0;
  const int u = a.src[q], m = a.model[q];
  const int v = (u >= 0 && u < a.G) ? a.dest[u] : -1;
  if (u >= 0 && u < a.G && m >= 0 && m < a.M && v >= 0 && v < a.G) {
    const int ju = a.sm_cur[u], ku = a.freq_cur[u], jv = a.sm_cur[v], kv = a.freq_cur[v];
    const int Bu = a.batch[u], ctx = a.ctx[q], rem = a.rem[q], kvk = a.kv_kib[q], tok = a.tok_kib[q];
    const bool ok = ju >= 0 && ju < a.NS && ku >= 0 && ku < a.NF && jv >= 0 && jv < a.NS && kv >= 0 && kv < a.NF &&
                    Bu >= 0 && ctx >= 1 && rem >= 0 && kvk >= 0 && tok >= 0;
    if (ok) {
      dec = 0;
      const int bu = Bu + 1 > kRows ? kRows : Bu + 1;
      const int crow = min((int)(((unsigned)ctx + 255u) >> 8), kRows) - 1;
      rem_ms = (double)rem * (double)a.dc[((size_t)m * kRows + (bu - 1)) * a.C + (size_t)ju * a.NF + ku];
      if (v != u) {
        const double mpb = a.node[u] == a.node[v] ? a.mpb_intra : a.mpb_inter;
        const double kv_ms = link_ms((long long)kvk * 1024, mpb);
        const double tok_ms = link_ms((long long)tok * 1024, mpb);
        const double rec_ms = (double)a.pf[((size_t)m * kRows + crow) * a.C + (size_t)jv * a.NF + kv];
        const bool use_kv = kv_ms < rec_ms;
        mig_ms = tok_ms + (use_kv ? kv_ms : rec_ms);
        if (rem_ms > mig_ms) dec = use_kv ? 1 : 2;
      }
    }
  }
  a.decision[q] = dec;
  a.remaining_ms[q] = (float)rem_ms;
  a.migrate_ms[q] = (float)mig_ms;
}

double ms_per_byte(float gbs) { return 1e3 / ((double)gbs * 1e9); }

bool transfer_ok(const festina_transfer *T) {
  if (!T || T->n_gpus < 1 || T->n_models < 1) return false;
  if (!T->resident || !T->weights_mib || !T->state_mib || !T->node) return false;
  if (!(T->bw_intra_gbs > 0.f) || !(T->bw_inter_gbs > 0.f)) return false;
  return true;
}

}  // namespace

extern "C" festina_status festina_transfer_costs(const festina_transfer *T, float *cost, void *stream) {
  if (!transfer_ok(T) || !cost) return FESTINA_ERR_INVALID;
  if ((long long)T->n_gpus * T->n_gpus > (1LL << 40)) return FESTINA_ERR_UNSUPPORTED;
  CostArgs a;
  a.G = T->n_gpus;
  a.M = T->n_models;
  a.words = (T->n_models + 31) / 32;
  a.resident = T->resident;
  a.weights = T->weights_mib;
  a.state = T->state_mib;
  a.node = T->node;
  a.mpb_intra = ms_per_byte(T->bw_intra_gbs);
  a.mpb_inter = ms_per_byte(T->bw_inter_gbs);
  a.cost = cost;
  const int per_block = kCostBlock * 4 * kCostVecs;
  const int bpr = (a.G + per_block - 1) / per_block;
  const long long blocks = (long long)a.G * bpr;
  if (blocks > INT_MAX) return FESTINA_ERR_UNSUPPORTED;
  hipStream_t st = static_cast<hipStream_t>(stream);
  // 16-byte row stores when every row starts 16-byte aligned
  const int vec = (a.G % 4 == 0) && ((reinterpret_cast<uintptr_t>(cost) & 15) == 0);
  const bool aligned_in = ((reinterpret_cast<uintptr_t>(T->resident) & 15) == 0) &&
                          ((reinterpret_cast<uintptr_t>(T->node) & 15) == 0);
  if (vec && a.words == 1 && aligned_in)
    k_transfer_costs_w1<<<(unsigned)blocks, kCostBlock, 0, st>>>(a, bpr);
  else
    k_transfer_costs<<<(unsigned)blocks, kCostBlock, 0, st>>>(a, bpr, vec);
  return hipGetLastError() == hipSuccess ? FESTINA_OK : FESTINA_ERR_DEVICE;
}

extern "C" festina_status festina_request_moves(const festina_lut *L, const festina_transfer *T,
                                                const festina_plan *P, const festina_inflight *Q,
                                                festina_moves *out, void *stream) {
  if (!L || !transfer_ok(T) || !P || !Q || !out || Q->n_requests < 0) return FESTINA_ERR_INVALID;
  if (L->n_models < 1 || L->n_rows != kRows || L->n_sm < 1 || L->n_freq < 1 || !L->pf || !L->dc)
    return FESTINA_ERR_INVALID;
  if ((long long)L->n_sm * L->n_freq > FESTINA_MAX_CELLS) return FESTINA_ERR_UNSUPPORTED;
  if (!P->dest || !P->freq_cur || !P->sm_cur || !P->batch) return FESTINA_ERR_INVALID;
  if (Q->n_requests == 0) return FESTINA_OK;
  if (!Q->src || !Q->model || !Q->context_tokens || !Q->remaining_tokens || !Q->kv_kib || !Q->token_kib)
    return FESTINA_ERR_INVALID;
  if (!out->decision || !out->remaining_ms || !out->migrate_ms) return FESTINA_ERR_INVALID;
  MoveArgs a;
  a.M = L->n_models;
  a.NS = L->n_sm;
  a.NF = L->n_freq;
  a.C = L->n_sm * L->n_freq;
  a.G = T->n_gpus;
  a.Q = Q->n_requests;
  a.pf = L->pf;
  a.dc = L->dc;
  a.node = T->node;
  a.mpb_intra = ms_per_byte(T->bw_intra_gbs);
  a.mpb_inter = ms_per_byte(T->bw_inter_gbs);
  a.dest = P->dest;
  a.freq_cur = P->freq_cur;
  a.sm_cur = P->sm_cur;
  a.batch = P->batch;
  a.src = Q->src;
  a.model = Q->model;
  a.ctx = Q->context_tokens;
  a.rem = Q->remaining_tokens;
  a.kv_kib = Q->kv_kib;
  a.tok_kib = Q->token_kib;
  a.decision = out->decision;
  a.remaining_ms = out->remaining_ms;
  a.migrate_ms = out->migrate_ms;
  hipStream_t st = static_cast<hipStream_t>(stream);
  k_request_moves<<<(a.Q + kMoveBlock - 1) / kMoveBlock, kMoveBlock, 0, st>>>(a);
  return hipGetLastError() == hipSuccess ? FESTINA_OK : FESTINA_ERR_DEVICE;
}
