/*
 * festina.h -- C ABI of the batched energy-aware placement and migration search
 * (Festina, "Energy-Aware Scheduling for Serverless LLM Serving on Shared GPUs").
 *
 * Two calls do the work:
 *   festina_score_placements  -- for every pending request, score every
 *       (GPU, SM-partition level, frequency level) candidate against the offline
 *       profile tables, drop candidates that miss the TTFT/TBT SLO, and pick the
 *       least-energy one (Sec. 3.3, Phase One feasibility and Phase Two
 *       E^k = Power x Latency, argmin over the feasible set; Eq. energy).
 *   festina_score_migrations  -- for consolidation (Sec. 3.5), score every ordered
 *       source -> destination GPU pair for moving the whole source workload, and
 *       return each source's best destination.
 * and, for the per-GPU local schedulers:
 *   festina_sweep_batches     -- the joint SM/frequency sweep of many task batches at
 *       once (Sec. 3.4, runtime resource allocation): per batch, the least-energy
 *       frequency level at which every task meets its deadline on its smallest
 *       sufficient SM share and the shares fit the device.
 * and, as inputs of the consolidation algorithm (App. E, Sec. 3.5.1):
 *   festina_preferred_configs -- every active LLM's preferred configuration: the
 *       least-energy SLO-feasible cell of each phase, then the time-weighted SM share
 *       and energy-weighted frequency (Eq. preferred_sm, Eq. preferred_frequency);
 *   festina_fleet_ewr         -- the fleet's energy waste, optimal energy and energy
 *       waste ratio (Eq. energy_waste, energy_optimal, energy_waste_ratio);
 * the transfer plan after a reconfiguration (App. F):
 *   festina_transfer_costs    -- the device-mapping cost matrix e_uv = Bytes / BW;
 *   festina_request_moves     -- per in-flight request: finish in place, or move with the
 *       KV cache, or move the tokens and recompute;
 * and the paper's own dispatcher, for comparison with the exhaustive search:
 *   festina_dispatch_requests -- one operating point per GPU (its current frequency),
 *       the 2% stability tie-break, the F_max fallback and scale-out (Sec. 3.3).
 *   festina_dispatch_waves    -- the same over arrival waves, each wave's placements
 *       committed to the GPUs' batch, memory and frequency before the next wave.
 *
 * Conventions shared by every entry point
 *  - All array pointers inside the structs are DEVICE pointers (HIP global memory
 *    of the current device), laid out as structures of arrays, row-major, with the
 *    shapes given beside each field.  The caller owns every buffer, including the
 *    workspace; the library allocates nothing and keeps no pointer after a call.
 *  - Work is enqueued on `stream` (a hipStream_t passed as void*; NULL = the null
 *    stream).  Outputs are valid once the caller has synchronised that stream.
 *    Calls are stateless and reentrant; concurrent calls need distinct workspaces.
 *  - Errors: a NULL required pointer, a non-positive or inconsistent size, or a
 *    workspace smaller than the matching *_workspace_bytes() value returns
 *    FESTINA_ERR_INVALID before anything is launched.  A shape the kernels do not
 *    support returns FESTINA_ERR_UNSUPPORTED before anything is launched.  A HIP
 *    launch or runtime failure returns FESTINA_ERR_DEVICE.
 *  - Bad per-element data never causes an out-of-bounds access: it only makes the
 *    affected request, GPU or pair infeasible (see each struct).
 *  - Units: latency ms, power W, energy mJ (W x ms), saving W.
 */
#ifndef FESTINA_H
#define FESTINA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FESTINA_ABI_VERSION 4
#define FESTINA_N_ROWS 32        /* rows of every profile table */
#define FESTINA_MAX_CELLS 256    /* n_sm * n_freq limit of the placement kernels */
#define FESTINA_MAX_FREQ_MIG 32  /* n_freq limit of the migration kernels (32-bit level masks) */
#define FESTINA_MAX_FREQ_SWEEP 64 /* n_freq limit of the sweep kernel (one lane per level) */
#define FESTINA_MAX_TASKS 64     /* task slots per batch of the sweep kernel */
#define FESTINA_PREFILL 0        /* task phases of the sweep */
#define FESTINA_DECODE 1
#define FESTINA_STATIC_PER_TASK 0    /* sweep energy: static power in every task's Power x Latency */
#define FESTINA_STATIC_PER_BATCH 1   /* sweep energy: static power once, over the batch's longest task */
/* Device scratch that festina_score_placements_noalloc holds per GPU (32 MiB: the
 * 262,144-request, 1,024-GPU, 64-wave placement search needs 11.3 MiB of it). */
#define FESTINA_NOALLOC_WORKSPACE_BYTES ((size_t)32 << 20)

typedef enum {
  FESTINA_OK = 0,
  FESTINA_ERR_INVALID = 1,
  FESTINA_ERR_DEVICE = 2,
  FESTINA_ERR_UNSUPPORTED = 3,
  FESTINA_ERR_TOO_LARGE = 4     /* input exceeds the fixed scratch of an allocation-free entry point */
} festina_status;

/* Offline profile look-up table (Sec. 3.2.1: latency per model under each frequency,
 * SM share and input length / batch).  Power is the closed form
 *   P(s, f, u) = p0_w + k_g * s * f^3 * u
 * (static power plus dynamic power cubic in frequency, Sec. 3.5.1), so it needs no table.
 *   pf[m][row][j][k]: prefill latency (TTFT, ms) of model m for a prompt in 256-token
 *                     bucket `row` (tokens in (256*row, 256*(row+1)]), SM level j,
 *                     frequency level k.
 *   dc[m][row][j][k]: decode-step latency (TBT, ms) at batch row+1.
 * NaN or +inf entries are never feasible. */
typedef struct festina_lut {
  int32_t n_models;          /* M >= 1 */
  int32_t n_rows;            /* must be FESTINA_N_ROWS */
  int32_t n_sm;              /* NS >= 1 */
  int32_t n_freq;            /* NF >= 1; NS*NF <= FESTINA_MAX_CELLS */
  const float *sm_level;     /* [NS] SM share s_j in (0, 1] */
  const float *freq_level;   /* [NF] normalised frequency f_k */
  const float *pf;           /* [M][32][NS][NF] */
  const float *dc;           /* [M][32][NS][NF] */
  float p0_w;                /* static power P0, W */
} festina_lut;

/* GPU state summaries (Sec. 3.3 Phase One: what each local scheduler reports).
 * A request admitted to GPU g in wave w runs at batch b = min(batch[w][g] + 1, 32)
 * and utilisation u = b / 32.  A GPU whose batch is negative (in that wave) or
 * whose SM cap lies outside [0, NS-1] has no candidates. */
typedef struct festina_gpus {
  int32_t n_gpus;            /* G >= 1 */
  int32_t n_waves;           /* W >= 1 independent snapshots (arrival waves) */
  const int32_t *batch;      /* [W][G] current batch B_g */
  const float *k_dyn_w;      /* [G] dynamic-power coefficient k_g, W */
  const uint32_t *resident;  /* [G][(M+31)/32] bit m set = model m resident on g */
  const int8_t *cap_pf;      /* [G] or NULL: prefill runs at SM level min(j, cap_pf[g]) */
  const int8_t *cap_dc;      /* [G] or NULL: decode runs at SM level min(j, cap_dc[g]) */
} festina_gpus;

/* Pending requests (Sec. 3.3 Phase One: input length, predicted output length, SLOs).
 * The library applies the 5% output-length safety pad, Lout = ceil(1.05 * pred)
 * (Sec. 3.2.2), and buckets the prompt, row = min(ceil(tokens/256), 32) - 1; a request
 * with 0 prompt tokens reads its TTFT from the decode batch row instead.  A model id
 * outside [0, M), a wave outside [0, W), or negative token counts make the request
 * infeasible. */
typedef struct festina_requests {
  int32_t n_requests;              /* R >= 0 */
  const int32_t *model;            /* [R] */
  const int32_t *wave;             /* [R] snapshot index, or NULL (all wave 0) */
  const int32_t *prompt_tokens;    /* [R] */
  const int32_t *pred_out_tokens;  /* [R] predicted output tokens (before the pad) */
  const float *slo_ttft_ms;        /* [R] */
  const float *slo_tbt_ms;         /* [R] */
} festina_requests;

/* Placement results, one entry per request (device memory, written by the call):
 *   choice    = (g * NS + j) * NF + k of the least-energy feasible candidate; among
 *               candidates of exactly equal energy the lowest index; -1 if none;
 *   feasible  = 1 if a candidate was chosen, else 0 (the caller scales out,
 *               Sec. 3.3 Phase Three);
 *   energy_mj = Pp * TTFT + Lout * Pd * TBT of the choice (float32), +inf if none.
 * A candidate is feasible when TTFT < slo_ttft and TBT < slo_tbt (strict). */
typedef struct festina_placements {
  int32_t *choice;
  uint8_t *feasible;
  float *energy_mj;
} festina_placements;

/* Bytes of device workspace festina_score_placements needs for these shapes
 * (reads only the scalar fields).  Returns 0 for invalid shapes. */
size_t festina_placements_workspace_bytes(const festina_lut *lut, const festina_gpus *gpus,
                                          const festina_requests *req);

/* Score all requests (Sec. 3.3 Phases One-Two; Eq. energy).  `workspace` is device
 * memory of at least festina_placements_workspace_bytes() bytes, 256-byte aligned;
 * its contents on entry do not matter and are clobbered. */
festina_status festina_score_placements(const festina_lut *lut, const festina_gpus *gpus,
                                        const festina_requests *req, festina_placements *out,
                                        void *workspace, size_t workspace_bytes, void *stream);

/* For callers that time the scoring kernel alone (a measurement, not part of the search):
 * festina_score_placements, with `score_begin` recorded on `stream` immediately before
 * the scoring kernel and `score_end` immediately after it, so that hipEventElapsedTime of
 * the two is that kernel's duration.  Each is a hipEvent_t passed as void*, created by the
 * caller on the current device; NULL leaves that point unrecorded (both NULL: exactly
 * festina_score_placements).  Same arguments, checks, outputs and errors otherwise; a
 * failing record returns FESTINA_ERR_DEVICE.  Each recorded event costs a few microseconds
 * of stream time. */
festina_status festina_score_placements_timed(const festina_lut *lut, const festina_gpus *gpus,
                                              const festina_requests *req, festina_placements *out,
                                              void *workspace, size_t workspace_bytes, void *stream,
                                              void *score_begin, void *score_end);

/* For callers that cannot allocate device memory -- code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc: festina_score_placements with its
 * workspace taken from a fixed device array of FESTINA_NOALLOC_WORKSPACE_BYTES that the
 * library holds on every GPU it runs on until the process ends.  The call allocates
 * nothing; the caller passes inputs and outputs as for festina_score_placements, and gets
 * the same outputs.  The array's address on the current device is looked up on the first
 * call made with that device current.  Shapes whose festina_placements_workspace_bytes()
 * exceeds FESTINA_NOALLOC_WORKSPACE_BYTES return FESTINA_ERR_TOO_LARGE before anything is
 * launched.  Every call on one GPU shares that GPU's array: calls that overlap in time on
 * one GPU (on different streams or from different host threads) race and their results
 * are undefined; calls ordered on one stream are safe, since each call clears what it
 * needs cleared with a kernel (no memset) before it uses it. */
festina_status festina_score_placements_noalloc(const festina_lut *lut, const festina_gpus *gpus,
                                                const festina_requests *req, festina_placements *out,
                                                void *stream);

/* Consolidation fleet (Sec. 3.5.2; App. E): every GPU holds 1..max_inst resident
 * model instances.  Instance i of GPU g meets its SLOs at frequency level k when
 *   pf[model][prompt row][inst_sm][k] < slo_ttft  and  dc[model][batch row][inst_sm][k] < slo_tbt
 * (rows as for requests: prompt bucket, or the batch row for 0 prompt tokens; batch row
 * = min(inst_batch + 1, 32) - 1).  One frequency is shared by the whole GPU (Sec. 2.2),
 * so a GPU is feasible at k when all of its instances are.  An n_inst outside
 * [1, max_inst] or any instance field out of range makes the GPU infeasible. */
typedef struct festina_fleet {
  int32_t n_gpus;                    /* G >= 2 */
  int32_t max_inst;                  /* instance slots per GPU, >= 1 */
  const int32_t *n_inst;             /* [G] */
  const int32_t *inst_model;         /* [G][max_inst] */
  const int32_t *inst_prompt_tokens; /* [G][max_inst] */
  const int32_t *inst_batch;         /* [G][max_inst] */
  const int32_t *inst_sm;            /* [G][max_inst] SM level index the instance runs at */
  const float *inst_slo_ttft_ms;     /* [G][max_inst] */
  const float *inst_slo_tbt_ms;      /* [G][max_inst] */
  const int32_t *hbm_mib;            /* [G] resident memory footprint, MiB */
  const int32_t *sm_permille;        /* [G] SM demand (utilisation), per-mille */
  const float *util;                 /* [G] utilisation u_g used in the power model */
  const float *k_dyn_w;              /* [G] k_g, W */
  int32_t hbm_cap_mib;               /* memory budget of one GPU (with any safety margin) */
  int32_t sm_cap_permille;           /* SM budget, per-mille */
} festina_fleet;

/* Migration results, one entry per source GPU s (device memory):
 *   best_dst   = destination d != s maximising saving_w; lowest d on exact ties; -1 if none;
 *   saving_w   = P0 - k_d * (f[k*]^3 * (u_s + u_d) - f[kd0]^3 * u_d) (float32), -inf if none:
 *                the source's static power freed minus the destination's added dynamic
 *                power; may be negative (whether to move is the caller's decision);
 *   freq_level = k*, the lowest level at which every instance of s and d meets its SLOs
 *                (kd0 = d's own lowest such level); -1 if none.
 * A pair is feasible when hbm_s + hbm_d <= hbm_cap, sm_s + sm_d <= sm_cap (inclusive)
 * and such a k* exists. */
typedef struct festina_migrations {
  int32_t *best_dst;
  float *saving_w;
  int32_t *freq_level;
} festina_migrations;

size_t festina_migrations_workspace_bytes(const festina_lut *lut, const festina_fleet *fleet);

/* Score all ordered pairs and reduce per source (Sec. 3.5; capacity check Sec. 3.5.2).
 * Requires n_freq <= FESTINA_MAX_FREQ_MIG.  Workspace as for placements. */
festina_status festina_score_migrations(const festina_lut *lut, const festina_fleet *fleet,
                                        festina_migrations *out, void *workspace,
                                        size_t workspace_bytes, void *stream);

/* festina_score_migrations with `pairs_begin` / `pairs_end` recorded around its
 * pair-scoring kernel (k_migrate), as festina_score_placements_timed does around the
 * placement scoring kernel. */
festina_status festina_score_migrations_timed(const festina_lut *lut, const festina_fleet *fleet,
                                              festina_migrations *out, void *workspace,
                                              size_t workspace_bytes, void *stream, void *pairs_begin,
                                              void *pairs_end);

/* Task batches of the local schedulers (Sec. 3.4): batch b holds n_tasks[b] tasks in
 * slots 0..n_tasks[b]-1 of its max_tasks slots.  A task is a prefill unit (phase
 * FESTINA_PREFILL: latency from pf at the prompt bucket of task_tokens, rows as for
 * requests) or one decode step (phase FESTINA_DECODE: latency from dc at batch size
 * task_tokens, row = min(task_tokens, 32) - 1), and must finish strictly within
 * task_slack_ms, the remaining time to its SLO deadline.  SM level j takes sm_units[j]
 * of the device (e.g. per-mille: 125 per eighth); the shares of a batch must sum to
 * strictly less than sm_budget (Sec. 3.4: below 100% of the SMs).  A model id outside
 * [0, M), task_tokens < 1, an unknown phase, or n_tasks outside [0, max_tasks] makes
 * the batch infeasible. */
typedef struct festina_batches {
  int32_t n_batches;                 /* B >= 0 */
  int32_t max_tasks;                 /* task slots per batch, 1..FESTINA_MAX_TASKS */
  const int32_t *n_tasks;            /* [B] */
  const int32_t *task_model;         /* [B][max_tasks] */
  const int32_t *task_phase;         /* [B][max_tasks] FESTINA_PREFILL or FESTINA_DECODE */
  const int32_t *task_tokens;        /* [B][max_tasks] prompt tokens (prefill) or batch size (decode) */
  const float *task_slack_ms;        /* [B][max_tasks] */
  const float *k_dyn_w;              /* [B] dynamic-power coefficient of the batch's GPU, W */
  const float *util;                 /* [B] utilisation u of the batch's GPU in the power model */
  const int32_t *sm_units;           /* [NS] integer SM share of each level */
  int32_t sm_budget;                 /* shares must sum to < sm_budget */
  int32_t static_power;              /* FESTINA_STATIC_PER_TASK or FESTINA_STATIC_PER_BATCH */
} festina_batches;

/* Sweep results (device memory, written by the call):
 *   freq_level[b] = least-energy usable frequency level, lowest on exact ties; -1 if none;
 *   feasible[b]   = 1 if a level was chosen, else 0;
 *   energy_mj[b]  = at that level, with FESTINA_STATIC_PER_TASK the sum over tasks of
 *                   (P0 + k_dyn * s_j * f^3 * u) * latency, with FESTINA_STATIC_PER_BATCH
 *                   P0 * (the longest task's latency) + the sum over tasks of
 *                   k_dyn * s_j * f^3 * u * latency (float32); +inf if none;
 *   task_sm[b][t] = SM level of task t at that level (the smallest whose latency is below
 *                   the slack); -1 for slots t >= n_tasks[b] and for infeasible batches. */
typedef struct festina_sweep_result {
  int32_t *freq_level;
  uint8_t *feasible;
  float *energy_mj;
  int32_t *task_sm;
} festina_sweep_result;

/* Sweep every batch (Sec. 3.4, runtime resource allocation: per frequency, the minimum SM
 * share per task that meets its deadline, the device SM budget, the least predicted
 * energy).  Needs no workspace.  Requires n_freq <= FESTINA_MAX_FREQ_SWEEP,
 * n_sm <= FESTINA_MAX_CELLS and max_tasks <= FESTINA_MAX_TASKS.  One kernel launch on
 * `stream`.  The paper does not say how the tasks' energies combine; static_power selects
 * the reading (FESTINA_STATIC_PER_TASK, Power x Latency per task as the placement search
 * charges it per request, or FESTINA_STATIC_PER_BATCH, the device's static power once over
 * the batch's longest task since the partitions run side by side); any other value is
 * FESTINA_ERR_INVALID. */
festina_status festina_sweep_batches(const festina_lut *lut, const festina_batches *batches,
                                     festina_sweep_result *out, void *stream);

/* Active LLM instances (App. E: per LLM, the average input/output lengths over the last
 * window; Sec. 3.5.2 Phase One).  Slot i of GPU g is an instance when i < n_inst[g].  Its
 * prefill phase lasts TTFT = pf[model][prompt row of avg_in_tokens][j][k], its decode phase
 * avg_out_tokens x TBT with TBT = dc[model][batch row][j][k] (batch row =
 * min(batch + 1, 32) - 1); each must be strictly below its SLO.  Power is
 * p0_w + k_dyn_w[g] * s_j * f_k^3 * u with u = min(batch + 1, 32) / 32.  A model id out of
 * range, batch < 0, avg_in_tokens < 1, avg_out_tokens < 0, or n_inst outside
 * [0, max_inst] makes the instance infeasible. */
typedef struct festina_llms {
  int32_t n_gpus;                    /* G >= 0 */
  int32_t max_inst;                  /* K >= 1 slots per GPU */
  const int32_t *n_inst;             /* [G] */
  const int32_t *model;              /* [G][K] */
  const int32_t *avg_in_tokens;      /* [G][K] */
  const int32_t *avg_out_tokens;     /* [G][K] */
  const int32_t *batch;              /* [G][K] current decode batch B */
  const float *slo_ttft_ms;          /* [G][K] */
  const float *slo_tbt_ms;           /* [G][K] */
  const float *k_dyn_w;              /* [G] */
} festina_llms;

/* Preferred configurations, [G][K] each (device memory, written by the call):
 *   sm_p, f_p / sm_d, f_d = SM and frequency level of the least-energy feasible cell of
 *       the prefill / decode phase (energy = power x duration; lowest cell j*NF + k on
 *       exact ties); -1 when the phase has no feasible cell;
 *   t_p_ms, p_p_w / t_d_ms, p_d_w = that cell's duration and power (0 when none);
 *   t_ms = t_p_ms + t_d_ms, the instance's execution time t_l of Eq. energy_waste;
 *   sm_pref = (s_p t_p + s_d t_d) / (t_p + t_d)                    (Eq. preferred_sm),
 *   f_pref  = (P_p t_p f_p + P_d t_d f_d) / (P_p t_p + P_d t_d)    (Eq. preferred_frequency),
 *       as SM share and normalised frequency, NaN unless both phases have a cell;
 *   feasible = 1 when both phases have a cell. */
typedef struct festina_preferred {
  int32_t *sm_p, *f_p, *sm_d, *f_d;
  float *t_p_ms, *t_d_ms, *p_p_w, *p_d_w;
  float *t_ms;
  float *sm_pref, *f_pref;
  uint8_t *feasible;
} festina_preferred;

/* Preferred configuration of every instance slot (App. E).  Needs no workspace; requires
 * n_sm * n_freq <= FESTINA_MAX_CELLS.  One kernel launch on `stream`. */
festina_status festina_preferred_configs(const festina_lut *lut, const festina_llms *llms,
                                         festina_preferred *out, void *stream);

/* Energy waste of a fleet (Sec. 3.5.1), device memory written by the call:
 *   f_gpu[g]     = F_g, the highest preferred frequency among GPU g's instances (0 if none);
 *   waste_gpu[g] = sum over its instances of t_l * (F_g^3 - F_l^3), float64;
 *   totals[0]    = E_waste = sum of waste_gpu; totals[1] = E_optimal = sum of t_l * F_l^3;
 *   totals[2]    = EWR = E_waste / E_optimal. */
typedef struct festina_ewr {
  float *f_gpu;
  double *waste_gpu;
  double *totals;
} festina_ewr;

/* Bytes of device workspace festina_fleet_ewr needs (0 for n_gpus < 1). */
size_t festina_ewr_workspace_bytes(int32_t n_gpus);

/* EWR of the fleet whose instance slots [n_gpus][max_inst] hold preferred frequencies
 * f_pref and execution times t_ms (device pointers; e.g. festina_preferred_configs'
 * f_pref and t_ms).  Slots past n_inst[g], and slots whose frequency or time is
 * not finite, are left out.  Workspace 256-byte aligned, contents clobbered; one kernel
 * launch on `stream` up to 16,384 GPUs, two beyond; the totals are summed in a fixed
 * order (deterministic). */
festina_status festina_fleet_ewr(int32_t n_gpus, int32_t max_inst, const int32_t *n_inst,
                                 const float *f_pref, const float *t_ms, festina_ewr *out,
                                 void *workspace, size_t workspace_bytes, void *stream);

/* The paper's own dispatcher (Sec. 3.3): each GPU offers one operating point, its current
 * frequency level freq_cur and the SMs free once the request's memory is available.  Its
 * local scheduler reports a free-memory profile of n_steps steps: from t_avail_ms[g][s] on
 * (non-decreasing in s), mem_free_mib[g][s] MiB and SM level sm_free[g][s] (-1 = none) are
 * free.  A request needs Req_mem = kv_kib_per_token[model] * (prompt + Lout) KiB (Lout the
 * padded output); T_avail and SM_free come from the first step whose memory holds it.  A GPU
 * with a negative batch, not hosting the model, or without such a step is no candidate.
 * n_gpus must be below 2^24 and n_sm * n_freq at most FESTINA_MAX_CELLS. */
typedef struct festina_gpu_avail {
  int32_t n_gpus;                    /* G >= 1 */
  int32_t n_steps;                   /* S >= 1 */
  const int32_t *freq_cur;           /* [G] current frequency level F_curr */
  const int32_t *batch;              /* [G] current batch B (b = min(B+1, 32), u = b/32) */
  const float *k_dyn_w;              /* [G] */
  const uint32_t *resident;          /* [G][(M+31)/32] */
  const float *t_avail_ms;           /* [G][S] */
  const int32_t *mem_free_mib;       /* [G][S] */
  const int32_t *sm_free;            /* [G][S] SM level index, -1 = none */
  const int32_t *kv_kib_per_token;   /* [M] KV-cache KiB per token of each model */
  float k_new_w;                     /* k of a newly activated GPU */
} festina_gpu_avail;

/* Dispatch results, one entry per request (device memory, written by the call):
 *   phase 1 (Phase Two): among the GPUs whose point meets both SLOs (T_avail + TTFT <
 *     slo_ttft, TBT < slo_tbt at (SM_free, freq_cur)), every one with energy
 *     E = (P0 + k*s*f^3*u) * (TTFT + Lout*TBT) within 2% of the least (E <= E_min + 0.02|E_min|)
 *     ties, and the one with the most free memory, then the most free SMs, then the
 *     lowest id wins;
 *   phase 2 (Phase Three): no such GPU; the earliest-available GPU (then lowest id) whose
 *     point meets the SLOs at the top frequency level;
 *   phase 3 (scale-out): a new GPU (batch 1, every SM, available now, k = k_new_w) at its
 *     least-energy feasible level (lowest on ties); gpu = -1;
 *   phase 0: nothing feasible (also for an invalid request); gpu, levels -1, energy +inf.
 * Energies are evaluated in float64, each operation rounded in the order written above,
 * and returned as float32. */
typedef struct festina_dispatches {
  int32_t *gpu, *freq_level, *sm_level;
  uint8_t *phase;
  float *energy_mj;
} festina_dispatches;

size_t festina_dispatch_workspace_bytes(const festina_lut *lut, const festina_gpu_avail *avail);

/* Dispatch every request against one snapshot of the GPUs' answers (Sec. 3.3, Phases One
 * to Three; requests' wave field is ignored).  Workspace as for placements; two kernel
 * launches on `stream`. */
festina_status festina_dispatch_requests(const festina_lut *lut, const festina_gpu_avail *avail,
                                         const festina_requests *req, festina_dispatches *out,
                                         void *workspace, size_t workspace_bytes, void *stream);

/* The GPUs' state that a wave-by-wave dispatch carries from one wave to the next (device
 * memory written by the call; the arrays may be avail's own, which are then updated in
 * place).  On return it is the state after the last wave. */
typedef struct festina_gpu_state {
  int32_t *freq_cur;                 /* [G] current frequency level */
  int32_t *batch;                    /* [G] decode batch */
  int32_t *mem_free_mib;             /* [G][S] free-memory profile */
} festina_gpu_state;

size_t festina_dispatch_waves_workspace_bytes(const festina_lut *lut, const festina_gpu_avail *avail);

/* The dispatcher over arrival waves (Sec. 3.3 decides each request on the state the local
 * schedulers report; here one wave of requests shares a snapshot and the waves follow one
 * another).  Requests are ordered by wave: wave w is requests wave_start[w] ..
 * wave_start[w+1]-1 (wave_start: HOST array of n_waves + 1 entries, wave_start[0] = 0,
 * non-decreasing, wave_start[n_waves] = n_requests; requests' wave field is ignored).
 * The state starts as avail's freq_cur, batch and mem_free_mib.  Each wave is dispatched
 * exactly as festina_dispatch_requests would on the current state, then each of its
 * requests placed on a GPU of the table (phase 1 or 2) is committed to that GPU: the batch
 * grows by one; ceil(Req_mem / 1024) MiB are taken from every profile step at or after the
 * one that admitted it (a step left short reads -1 MiB); a phase-2 (F_max) placement leaves
 * the GPU at the top frequency level.  Profile times, free SM levels, k and residency stay
 * as given; a scale-out (phase 3) commits nothing.  Workspace from
 * festina_dispatch_waves_workspace_bytes (256-byte aligned, clobbered).  One kernel launch
 * per non-empty wave plus three (two without requests) on `stream`, nothing allocated or
 * synchronised. */
festina_status festina_dispatch_waves(const festina_lut *lut, const festina_gpu_avail *avail,
                                      const festina_requests *req, int32_t n_waves, const int32_t *wave_start,
                                      festina_gpu_state *state, festina_dispatches *out, void *workspace,
                                      size_t workspace_bytes, void *stream);

/* Transfer plan after a reconfiguration (App. F).  A GPU's state is its resident models'
 * weights plus its request state selected for migration.  Sending GPU u's state to GPU v
 * moves state_mib[u] plus the weights of u's resident models that v does not hold; it
 * runs at bw_intra_gbs between GPUs of one node (equal node ids), else at bw_inter_gbs. */
typedef struct festina_transfer {
  int32_t n_gpus;                    /* G >= 1 */
  int32_t n_models;                  /* M >= 1 */
  const uint32_t *resident;          /* [G][(M+31)/32] models resident now */
  const int32_t *weights_mib;        /* [M] */
  const int32_t *state_mib;          /* [G] */
  const int32_t *node;               /* [G] */
  float bw_intra_gbs, bw_inter_gbs;  /* GB/s, > 0 */
} festina_transfer;

/* Device-mapping cost matrix: cost[u][v] = e_uv = Bytes(u -> v) / BW(u, v) in ms (float32,
 * row-major [G][G], device memory written by the call), e_uu = 0; Bytes in bytes (MiB =
 * 2^20 B), time = bytes * 1e3 / (GB/s * 1e9) evaluated in float64 and rounded once.  This
 * is the input of the minimum-cost assignment (Kuhn-Munkres), which this library does not
 * solve.  One kernel launch on `stream`. */
festina_status festina_transfer_costs(const festina_transfer *transfer, float *cost, void *stream);

/* The plan: dest[u] = the GPU that receives GPU u's state (u itself: it stays), and each
 * GPU's operating point (SM level, frequency level) and decode batch. */
typedef struct festina_plan {
  const int32_t *dest, *freq_cur, *sm_cur, *batch;   /* [G] */
} festina_plan;

/* In-flight requests whose GPU is being reconfigured. */
typedef struct festina_inflight {
  int32_t n_requests;                /* Q >= 0 */
  const int32_t *src;                /* [Q] GPU now serving the request */
  const int32_t *model;              /* [Q] */
  const int32_t *context_tokens;     /* [Q] prompt plus tokens generated so far, >= 1 */
  const int32_t *remaining_tokens;   /* [Q] tokens still to generate (predicted) */
  const int32_t *kv_kib;             /* [Q] KV-cache size */
  const int32_t *token_kib;          /* [Q] token state (prompt and generated ids) */
} festina_inflight;

/* Per request (device memory, written by the call):
 *   remaining_ms = remaining_tokens * TBT at the source (dc at its batch row and point);
 *   migrate_ms   = token transfer + the faster of KV transfer and recompute (pf at the
 *                  context's prompt bucket at the destination's point), 0 when the
 *                  source's state stays (dest[src] == src);
 *   decision     = 1 move with the KV cache, 2 move the tokens and recompute, when
 *                  remaining_ms > migrate_ms; 0 finish in place (or the state stays);
 *                  -1 invalid request (GPU, model, level or token count out of range).
 * Times evaluated in float64 and rounded once to float32. */
typedef struct festina_moves {
  int32_t *decision;
  float *remaining_ms, *migrate_ms;
} festina_moves;

festina_status festina_request_moves(const festina_lut *lut, const festina_transfer *transfer,
                                     const festina_plan *plan, const festina_inflight *req,
                                     festina_moves *out, void *stream);

/* Static, NUL-terminated description of a status code. */
const char *festina_status_string(festina_status status);

/* FESTINA_ABI_VERSION of the loaded library. */
int32_t festina_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FESTINA_H */
