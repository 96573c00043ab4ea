/*
 * festina_oracle.c -- plain, slow, obviously-correct CPU oracle of the batched
 * energy-aware placement and migration search.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and the
 * benchmark's CPU-baseline leg may load or call this library.  The product path
 * (the HIP library) never links it, includes it, or falls back to it, and the two
 * share no code: this file re-declares everything it needs.
 *
 * Arithmetic is float64 throughout (inputs are float32 and are promoted).  Every
 * SLO test compares a float32 table entry with a float32 SLO, so promoting does not
 * change its outcome.  Loops run in the order of the plain definitions:
 *
 *   placement (Sec. 3.3, Phase One and Phase Two; energy = power x time, Eq. energy):
 *     for every request r, every GPU g hosting r's model, every SM level j and
 *     frequency level k: the candidate is feasible when its prefill latency (TTFT)
 *     is strictly below the TTFT SLO and its decode-step latency (TBT) is strictly
 *     below the TBT SLO (Phase One: "complete before its SLO deadline");
 *     its energy is
 *        E = Pp * TTFT + Lout * Pd * TBT,   P = P0 + k_g * s * f^3 * u_g
 *     (Phase Two's E^k = Power x Latency, split into the prefill phase and Lout decode
 *     steps, each at its own SM level); the chosen candidate is the least-energy
 *     feasible one (Phase Two argmin), exact ties going to the lowest linear index
 *     idx = (g*NS + j)*NF + k.  No feasible candidate -> flagged, not placed
 *     (Phase Three: the caller scales out).
 *
 *   migration (Sec. 3.5.2 capacity check; Sec. 1 "saved idle power"; one device-wide
 *   operating point shared by co-located models, Sec. 2.2 / 3.5.1):
 *     for every ordered pair s != d: the merged GPU must fit the HBM and SM budgets
 *     (inclusive) and some frequency level must let every instance of s and of d meet
 *     both SLOs at its own SM level; it then runs at the lowest such level k*;
 *     saving = P0 - k_d * (f[k*]^3 * (u_s + u_d) - f[kd0]^3 * u_d), where kd0 is d's own
 *     lowest feasible level.  Per source: the largest saving, lowest d on exact ties.
 *
 *   local SM/frequency sweep (Sec. 3.4, runtime resource allocation):
 *     for every batch of tasks and every frequency level k: each task takes the smallest
 *     SM level whose latency (PF row for a prefill unit, DC row for a decode step) is
 *     strictly below its slack; k is usable when every task has one and the integer SM
 *     shares sum to strictly less than the device budget; energy at k =
 *        sum over tasks of (P0 + k_dyn * s_j * f_k^3 * u) * latency
 *     (Power x Latency per task, the placement power model); the least-energy usable k
 *     wins, the lowest k on exact ties.
 *
 *   preferred configuration (App. E) and energy waste ratio (Sec. 3.5.1):
 *     per LLM instance, the least-energy SLO-feasible cell of the prefill phase
 *     (duration TTFT at the average prompt's bucket) and of the decode phase (duration
 *     avg_out x TBT at the batch row), then SM_l = (s_p T_p + s_d T_d) / (T_p + T_d) and
 *     F_l = (P_p T_p f_p + P_d T_d f_d) / (P_p T_p + P_d T_d); per GPU F_g = max F_l,
 *     E_waste = sum t_l (F_g^3 - F_l^3), E_optimal = sum t_l F_l^3, EWR = their ratio.
 *
 *   current-frequency dispatch (Sec. 3.3 as the paper runs it, Phases One to Three with
 *   the 2% stability tie-break and the F_max fallback), on one snapshot of the GPUs or
 *   over arrival waves with each wave committed to the GPUs' state before the next: see
 *   the section at the end.
 *
 *   transfer plan (App. F): the cost matrix e_uv = Bytes(u -> v) / BW(u, v) of the
 *   minimum-cost device mapping, and the per-request choice to finish in place or move
 *   (with the KV cache or a recompute of it): see the section at the end.
 *
 * Request pre-processing (Sec. 3.2.1 input-length axis 256..8192; Sec. 3.2.2 / 3.3 the
 * 5% output-length safety pad):
 *   Lout = ceil(1.05 * predicted_out)            (integer: (105*L + 99) / 100)
 *   prompt row = min(ceil(prompt_tokens / 256), 32) - 1; no prompt (0 tokens) -> the
 *   decode batch row is used for the TTFT lookup as well.
 * GPU state (Sec. 3.3 Phase One, post-admission): b = min(B + 1, 32), u = b / 32.
 *
 * Invalid per-element data (model id out of range, negative batch / tokens, wave out
 * of range, SM cap outside [0, NS-1], instance fields out of range) never causes an
 * out-of-bounds read: the request / GPU / pair simply becomes infeasible.
 * A candidate is eligible only when its energy rounded to float32 is below +inf
 * (so NaN and overflowing energies are never chosen); a pair only when its saving
 * rounded to float32 is above -inf.
 *
 * Build: gcc -O2 -ffp-contract=off -fPIC -shared (no fast-math).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define OR_ROWS 32
#define OR_ROW_TOKENS 256

/* ---------------------------------------------------------------- oracle's own records */
typedef struct {
  int32_t n_models, n_rows, n_sm, n_freq;
  const float *sm_level, *freq_level, *pf, *dc;
  double p0_w;
} or_lut;

typedef struct {
  int32_t n_gpus, n_waves;
  const int32_t *batch;       /* [W][G] */
  const float *k_dyn_w;       /* [G] */
  const uint32_t *resident;   /* [G][(M+31)/32] */
  const int8_t *cap_pf, *cap_dc; /* [G] or NULL */
} or_gpus;

typedef struct {
  int32_t n_requests;
  const int32_t *model, *wave, *prompt_tokens, *pred_out_tokens;
  const float *slo_ttft_ms, *slo_tbt_ms;
} or_requests;

typedef struct {
  int32_t n_gpus, max_inst;
  const int32_t *n_inst, *inst_model, *inst_prompt_tokens, *inst_batch, *inst_sm;
  const float *inst_slo_ttft_ms, *inst_slo_tbt_ms;
  const int32_t *hbm_mib, *sm_permille;
  const float *util, *k_dyn_w;
  int32_t hbm_cap_mib, sm_cap_permille;
} or_fleet;

/* ---------------------------------------------------------------- pre-processing */
/* -2 invalid, -1 no prompt, else row 0..31 */
static int or_prompt_row(int32_t tokens) {
  if (tokens < 0) return -2;
  if (tokens == 0) return -1;
  int64_t r = ((int64_t)tokens + OR_ROW_TOKENS - 1) / OR_ROW_TOKENS;
  if (r > OR_ROWS) r = OR_ROWS;
  return (int)(r - 1);
}

static int64_t or_padded_out(int32_t predicted) {
  return ((int64_t)predicted * 105 + 99) / 100;
}

int festina_oracle_prompt_row(int32_t tokens) { return or_prompt_row(tokens); }
int64_t festina_oracle_padded_out(int32_t predicted) { return or_padded_out(predicted); }

static double or_cube(double x) { return x * x * x; }

static size_t or_cell(const or_lut *L, int m, int row, int j, int k) {
  return (((size_t)m * OR_ROWS + (size_t)row) * (size_t)L->n_sm + (size_t)j) * (size_t)L->n_freq + (size_t)k;
}

static int or_lut_ok(const or_lut *L) {
  if (!L || L->n_models < 1 || L->n_rows != OR_ROWS || L->n_sm < 1 || L->n_freq < 1) return 0;
  if (!L->sm_level || !L->freq_level || !L->pf || !L->dc) return 0;
  return 1;
}

/* ---------------------------------------------------------------- placement */
/* Energy of candidate idx for request r.  Returns 1 and sets *energy when the candidate
 * exists, hosts the request's model, is SLO-feasible and has an eligible energy. */
static int or_candidate(const or_lut *L, const or_gpus *G, const or_requests *Q,
                        int32_t r, int64_t idx, double *energy) {
  const int NS = L->n_sm, NF = L->n_freq, M = L->n_models;
  if (r < 0 || r >= Q->n_requests) return 0;
  if (idx < 0 || idx >= (int64_t)G->n_gpus * NS * NF) return 0;
  const int g = (int)(idx / ((int64_t)NS * NF));
  const int j = (int)((idx / NF) % NS);
  const int k = (int)(idx % NF);
  const int m = Q->model[r];
  const int w = Q->wave ? Q->wave[r] : 0;
  if (m < 0 || m >= M || w < 0 || w >= G->n_waves) return 0;
  if (Q->pred_out_tokens[r] < 0) return 0;
  const int prow = or_prompt_row(Q->prompt_tokens[r]);
  if (prow == -2) return 0;
  const int words = (M + 31) / 32;
  if (!((G->resident[(size_t)g * words + (size_t)(m / 32)] >> (m % 32)) & 1u)) return 0;
  const int32_t B = G->batch[(size_t)w * G->n_gpus + g];
  if (B < 0) return 0;
  const int b = (B + 1 > OR_ROWS) ? OR_ROWS : B + 1;
  const int cp = G->cap_pf ? G->cap_pf[g] : NS - 1;
  const int cd = G->cap_dc ? G->cap_dc[g] : NS - 1;
  if (cp < 0 || cp >= NS || cd < 0 || cd >= NS) return 0;
  const int jp = j < cp ? j : cp;
  const int jd = j < cd ? j : cd;
  const int row_p = prow >= 0 ? prow : b - 1;
  const float ttft = L->pf[or_cell(L, m, row_p, jp, k)];
  const float tbt = L->dc[or_cell(L, m, b - 1, jd, k)];
  if (!(ttft < Q->slo_ttft_ms[r] && tbt < Q->slo_tbt_ms[r])) return 0;
  const double u = (double)b / 32.0;
  const double f3 = or_cube((double)L->freq_level[k]);
  const double kg = (double)G->k_dyn_w[g];
  const double Pp = L->p0_w + kg * (double)L->sm_level[jp] * f3 * u;
  const double Pd = L->p0_w + kg * (double)L->sm_level[jd] * f3 * u;
  const double Lout = (double)or_padded_out(Q->pred_out_tokens[r]);
  const double E = Pp * (double)ttft + Lout * Pd * (double)tbt;
  if (!((float)E < INFINITY)) return 0;
  *energy = E;
  return 1;
}

int festina_oracle_candidate(const or_lut *L, const or_gpus *G, const or_requests *Q,
                             int32_t r, int64_t idx, double *energy) {
  if (!or_lut_ok(L) || !G || !Q || !energy) return 0;
  return or_candidate(L, G, Q, r, idx, energy);
}

/* Score requests sel[0..n_sel) (all requests when sel == NULL; then n_sel is ignored).
 * Output i belongs to request sel[i].  Returns 0, or 1 on invalid arguments. */
int festina_oracle_score_placements(const or_lut *L, const or_gpus *G, const or_requests *Q,
                                    int32_t n_sel, const int32_t *sel,
                                    int32_t *choice, uint8_t *feasible, double *energy_mj) {
  if (!or_lut_ok(L) || !G || !Q || !choice || !feasible || !energy_mj) return 1;
  if (G->n_gpus < 0 || G->n_waves < 1 || Q->n_requests < 0) return 1;
  const int64_t cells = (int64_t)L->n_sm * L->n_freq;
  const int words = (L->n_models + 31) / 32;
  const int32_t n = sel ? n_sel : Q->n_requests;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t r = sel ? sel[i] : i;
    const int m = (r >= 0 && r < Q->n_requests) ? Q->model[r] : -1;
    int64_t best_idx = -1;
    double best_e = INFINITY;
    for (int32_t g = 0; g < G->n_gpus && m >= 0 && m < L->n_models; ++g) {
      /* GPUs not hosting the model have no candidates: skip them whole */
      if (!((G->resident[(size_t)g * words + (size_t)(m / 32)] >> (m % 32)) & 1u)) continue;
      for (int64_t c = 0; c < cells; ++c) {
        const int64_t idx = (int64_t)g * cells + c; /* ascending (g, j, k) */
        double e;
        if (!or_candidate(L, G, Q, r, idx, &e)) continue;
        if (best_idx < 0 || e < best_e) {
          best_idx = idx;
          best_e = e;
        }
      }
    }
    choice[i] = (int32_t)best_idx;
    feasible[i] = best_idx >= 0 ? 1 : 0;
    energy_mj[i] = best_idx >= 0 ? best_e : INFINITY;
  }
  return 0;
}

/* ---------------------------------------------------------------- migration */
/* Does instance i of GPU g meet both SLOs at frequency level k (at its own SM level)? */
static int or_instance_ok(const or_lut *L, const or_fleet *F, int g, int i, int k) {
  const size_t at = (size_t)g * F->max_inst + (size_t)i;
  const int m = F->inst_model[at];
  const int j = F->inst_sm[at];
  const int32_t B = F->inst_batch[at];
  const int prow = or_prompt_row(F->inst_prompt_tokens[at]);
  if (m < 0 || m >= L->n_models || j < 0 || j >= L->n_sm || B < 0 || prow == -2) return 0;
  const int b = (B + 1 > OR_ROWS) ? OR_ROWS : B + 1;
  const int row_p = prow >= 0 ? prow : b - 1;
  const float ttft = L->pf[or_cell(L, m, row_p, j, k)];
  const float tbt = L->dc[or_cell(L, m, b - 1, j, k)];
  return ttft < F->inst_slo_ttft_ms[at] && tbt < F->inst_slo_tbt_ms[at];
}

/* Do all instances of GPU g meet their SLOs at level k? */
static int or_gpu_ok(const or_lut *L, const or_fleet *F, int g, int k) {
  const int n = F->n_inst[g];
  if (n < 1 || n > F->max_inst) return 0;
  for (int i = 0; i < n; ++i)
    if (!or_instance_ok(L, F, g, i, k)) return 0;
  return 1;
}

static int or_pair(const or_lut *L, const or_fleet *F, int s, int d, int *kstar_out, double *saving) {
  if (s < 0 || d < 0 || s >= F->n_gpus || d >= F->n_gpus || s == d) return 0;
  if ((int64_t)F->hbm_mib[s] + F->hbm_mib[d] > (int64_t)F->hbm_cap_mib) return 0;
  if ((int64_t)F->sm_permille[s] + F->sm_permille[d] > (int64_t)F->sm_cap_permille) return 0;
  int kstar = -1;
  for (int k = 0; k < L->n_freq && kstar < 0; ++k)
    if (or_gpu_ok(L, F, s, k) && or_gpu_ok(L, F, d, k)) kstar = k;
  if (kstar < 0) return 0;
  int kd0 = -1;
  for (int k = 0; k < L->n_freq && kd0 < 0; ++k)
    if (or_gpu_ok(L, F, d, k)) kd0 = k;
  const double us = (double)F->util[s], ud = (double)F->util[d];
  const double kd = (double)F->k_dyn_w[d];
  const double added = or_cube((double)L->freq_level[kstar]) * (us + ud) - or_cube((double)L->freq_level[kd0]) * ud;
  const double sv = L->p0_w - kd * added;
  if (!((float)sv > -INFINITY)) return 0;
  *kstar_out = kstar;
  *saving = sv;
  return 1;
}

int festina_oracle_pair(const or_lut *L, const or_fleet *F, int32_t s, int32_t d,
                        int32_t *kstar, double *saving) {
  if (!or_lut_ok(L) || !F || !kstar || !saving) return 0;
  int k;
  double sv;
  if (!or_pair(L, F, s, d, &k, &sv)) return 0;
  *kstar = k;
  *saving = sv;
  return 1;
}

/* Score sources sel[0..n_sel) (all when sel == NULL).  Output i belongs to source sel[i]. */
int festina_oracle_score_migrations(const or_lut *L, const or_fleet *F, int32_t n_sel, const int32_t *sel,
                                    int32_t *best_dst, double *saving_w, int32_t *freq_level) {
  if (!or_lut_ok(L) || !F || !best_dst || !saving_w || !freq_level) return 1;
  if (F->n_gpus < 0 || F->max_inst < 1) return 1;
  const int32_t n = sel ? n_sel : F->n_gpus;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t s = sel ? sel[i] : i;
    int32_t bd = -1, bk = -1;
    double bs = -INFINITY;
    for (int32_t d = 0; d < F->n_gpus; ++d) {
      int k;
      double sv;
      if (!or_pair(L, F, s, d, &k, &sv)) continue;
      if (bd < 0 || sv > bs) {
        bd = d;
        bs = sv;
        bk = k;
      }
    }
    best_dst[i] = bd;
    saving_w[i] = bd >= 0 ? bs : -INFINITY;
    freq_level[i] = bk;
  }
  return 0;
}

/* ---------------------------------------------------------------- local SM/frequency sweep */
/* Sec. 3.4, "Runtime Resource Allocation": a local scheduler holds a batch of tasks
 * (prefill units and decode steps) and picks one GPU frequency level for the batch.  At
 * each level k, every task takes the smallest SM level whose profiled latency is strictly
 * below the task's remaining slack; the level is usable only when every task has such an
 * SM level and the SM shares sum to strictly less than the device budget ("< 100%");
 * the batch's energy at k is the sum over its tasks of Power x Latency with the same
 * closed-form power model as placement, P = P0 + k_dyn * s * f^3 * u.  The paper leaves
 * open how the tasks' energies combine; static_power selects the reading: 0 charges P0 in
 * every task's term (as placement charges it per request), 1 charges it once, over the
 * longest task (the partitions run side by side on one device), the dynamic terms still
 * per task.  The chosen level is the least-energy usable one, the lowest k on exact
 * ties. */
typedef struct {
  int32_t n_batches, max_tasks;
  const int32_t *n_tasks;        /* [B] */
  const int32_t *task_model;     /* [B][T] */
  const int32_t *task_phase;     /* [B][T] 0 = prefill (PF table), 1 = decode (DC table) */
  const int32_t *task_tokens;    /* [B][T] prompt tokens (prefill) or decode batch size */
  const float *task_slack_ms;    /* [B][T] */
  const float *k_dyn_w;          /* [B] */
  const float *util;             /* [B] */
  const int32_t *sm_units;       /* [NS] integer SM share of each level */
  int32_t sm_budget;
  int32_t static_power;          /* 0: P0 per task, 1: P0 over the longest task */
} or_batches;

/* Table row of task t of batch b, or -1 when the task is invalid.  Prefill rows are the
 * 256-token prompt buckets; decode rows are batch sizes 1..32 (row = size - 1). */
static int or_task_row(const or_lut *L, const or_batches *S, int b, int t) {
  const size_t at = (size_t)b * S->max_tasks + (size_t)t;
  const int m = S->task_model[at], ph = S->task_phase[at];
  const int32_t tok = S->task_tokens[at];
  if (m < 0 || m >= L->n_models || tok < 1) return -1;
  if (ph == 0) return or_prompt_row(tok);
  if (ph == 1) return (tok > OR_ROWS ? OR_ROWS : tok) - 1;
  return -1;
}

static float or_task_latency(const or_lut *L, const or_batches *S, int b, int t, int row, int j, int k) {
  const size_t at = (size_t)b * S->max_tasks + (size_t)t;
  const int m = S->task_model[at];
  const float *tab = S->task_phase[at] == 0 ? L->pf : L->dc;
  return tab[or_cell(L, m, row, j, k)];
}

/* Smallest SM level at which task t meets its slack at frequency level k; -1 if none. */
static int or_min_sm(const or_lut *L, const or_batches *S, int b, int t, int k) {
  const int row = or_task_row(L, S, b, t);
  if (row < 0) return -1;
  const float slack = S->task_slack_ms[(size_t)b * S->max_tasks + (size_t)t];
  for (int j = 0; j < L->n_sm; ++j)
    if (or_task_latency(L, S, b, t, row, j, k) < slack) return j;
  return -1;
}

static int or_batch_ok(const or_lut *L, const or_batches *S, int b) {
  const int n = S->n_tasks[b];
  if (n < 0 || n > S->max_tasks) return 0;
  for (int t = 0; t < n; ++t)
    if (or_task_row(L, S, b, t) < 0) return 0;
  return 1;
}

/* Energy of batch b at frequency level k: 1 and *energy when level k is usable. */
static int or_sweep_level(const or_lut *L, const or_batches *S, int b, int k, double *energy) {
  if (b < 0 || b >= S->n_batches || k < 0 || k >= L->n_freq || !or_batch_ok(L, S, b)) return 0;
  const double f3 = or_cube((double)L->freq_level[k]);
  const double kg = (double)S->k_dyn_w[b], u = (double)S->util[b];
  int64_t units = 0;
  double E = 0.0, longest = 0.0;
  for (int t = 0; t < S->n_tasks[b]; ++t) {
    const int j = or_min_sm(L, S, b, t, k);
    if (j < 0) return 0;
    units += S->sm_units[j];
    const double lat = (double)or_task_latency(L, S, b, t, or_task_row(L, S, b, t), j, k);
    const double dyn = kg * (double)L->sm_level[j] * f3 * u;
    if (S->static_power == 0) {
      E += (L->p0_w + dyn) * lat;
    } else {
      E += dyn * lat;
      if (lat > longest) longest = lat;
    }
  }
  if (S->static_power != 0) E += L->p0_w * longest;
  if (!(units < (int64_t)S->sm_budget)) return 0;
  if (!((float)E < INFINITY)) return 0;
  *energy = E;
  return 1;
}

int festina_oracle_sweep_level(const or_lut *L, const or_batches *S, int32_t b, int32_t k, double *energy) {
  if (!or_lut_ok(L) || !S || !energy) return 0;
  return or_sweep_level(L, S, b, k, energy);
}

int festina_oracle_min_sm(const or_lut *L, const or_batches *S, int32_t b, int32_t t, int32_t k) {
  if (!or_lut_ok(L) || !S || b < 0 || b >= S->n_batches || t < 0 || t >= S->max_tasks) return -1;
  if (k < 0 || k >= L->n_freq) return -1;
  return or_min_sm(L, S, b, t, k);
}

/* Sweep batches sel[0..n_sel) (all when sel == NULL).  Output i belongs to batch sel[i];
 * task_sm is [n][max_tasks]: each task's SM level at the chosen frequency level, -1 for
 * slots past n_tasks and for batches with no usable level. */
int festina_oracle_sweep(const or_lut *L, const or_batches *S, int32_t n_sel, const int32_t *sel,
                         int32_t *freq_level, uint8_t *feasible, double *energy_mj, int32_t *task_sm) {
  if (!or_lut_ok(L) || !S || !freq_level || !feasible || !energy_mj || !task_sm) return 1;
  if (S->n_batches < 0 || S->max_tasks < 1 || !S->sm_units) return 1;
  if (S->static_power != 0 && S->static_power != 1) return 1;
  const int32_t n = sel ? n_sel : S->n_batches;
  for (int32_t i = 0; i < n; ++i) {
    const int32_t b = sel ? sel[i] : i;
    int32_t bk = -1;
    double be = INFINITY;
    for (int k = 0; k < L->n_freq; ++k) {
      double e;
      if (!or_sweep_level(L, S, b, k, &e)) continue;
      if (bk < 0 || e < be) {
        bk = k;
        be = e;
      }
    }
    freq_level[i] = bk;
    feasible[i] = bk >= 0 ? 1 : 0;
    energy_mj[i] = bk >= 0 ? be : INFINITY;
    for (int t = 0; t < S->max_tasks; ++t)
      task_sm[(size_t)i * S->max_tasks + (size_t)t] = (bk >= 0 && t < S->n_tasks[b]) ? or_min_sm(L, S, b, t, bk) : -1;
  }
  return 0;
}

/* ---------------------------------------------------------------- preferred configuration, EWR */
/* App. E, "Determining Preferred Configurations": per active LLM, the least-energy
 * SLO-feasible (SM level, frequency level) of each phase from the look-up table, then
 * Eq. preferred_sm (time-weighted SM share) and Eq. preferred_frequency (energy-weighted
 * frequency).  Sec. 3.5.1, Eq. energy_waste / energy_optimal / energy_waste_ratio: per GPU
 * the operating frequency F_g is the highest preferred frequency among its LLMs. */
typedef struct {
  int32_t n_gpus, max_inst;
  const int32_t *n_inst;           /* [G] */
  const int32_t *model;            /* [G][K] */
  const int32_t *avg_in_tokens;    /* [G][K] */
  const int32_t *avg_out_tokens;   /* [G][K] */
  const int32_t *batch;            /* [G][K] current decode batch B */
  const float *slo_ttft_ms, *slo_tbt_ms;  /* [G][K] */
  const float *k_dyn_w;            /* [G] */
} or_llms;

typedef struct {
  int32_t sm_p, f_p, sm_d, f_d;    /* chosen levels, -1 when the phase has no feasible cell */
  double t_p, t_d, p_p, p_d;       /* phase duration (ms) and power (W) at those levels */
  double sm_pref, f_pref;          /* Eq. preferred_sm, Eq. preferred_frequency */
  int feasible;                    /* both phases have a feasible cell */
} or_pref;

/* Least-energy feasible cell of one phase of instance i of GPU g.  Prefill: duration
 * TTFT = PF[prompt row][j][k] (< SLO), energy P * TTFT.  Decode: duration
 * avg_out * TBT with TBT = DC[batch row][j][k] (< SLO), energy P * duration.  P is the
 * placement power model with u = b / 32, b = min(B + 1, 32).  Returns the linear cell
 * j*NF + k (lowest on exact ties) or -1. */
static int or_phase_best(const or_lut *L, const or_llms *Q, int g, int i, int decode,
                         double *t_out, double *p_out) {
  const size_t at = (size_t)g * Q->max_inst + (size_t)i;
  const int m = Q->model[at];
  const int32_t B = Q->batch[at];
  const int prow = or_prompt_row(Q->avg_in_tokens[at]);
  if (m < 0 || m >= L->n_models || B < 0 || prow < 0 || Q->avg_out_tokens[at] < 0) return -1;
  const int b = (B + 1 > OR_ROWS) ? OR_ROWS : B + 1;
  const double u = (double)b / 32.0;
  const double kg = (double)Q->k_dyn_w[g];
  int best = -1;
  double best_e = INFINITY, best_t = 0.0, best_p = 0.0;
  for (int j = 0; j < L->n_sm; ++j)
    for (int k = 0; k < L->n_freq; ++k) {
      const float lat = decode ? L->dc[or_cell(L, m, b - 1, j, k)] : L->pf[or_cell(L, m, prow, j, k)];
      const float slo = decode ? Q->slo_tbt_ms[at] : Q->slo_ttft_ms[at];
      if (!(lat < slo)) continue;
      const double P = L->p0_w + kg * (double)L->sm_level[j] * or_cube((double)L->freq_level[k]) * u;
      const double t = decode ? (double)Q->avg_out_tokens[at] * (double)lat : (double)lat;
      const double e = P * t;
      if (!((float)e < INFINITY)) continue;
      if (best < 0 || e < best_e) {
        best = j * L->n_freq + k;
        best_e = e;
        best_t = t;
        best_p = P;
      }
    }
  *t_out = best_t;
  *p_out = best_p;
  return best;
}

/* App. E, Eq. preferred_sm: SM_l = (s_p T_p + s_d T_d) / (T_p + T_d), the SM shares of the
 * two phases' cells weighted by their durations; Eq. preferred_frequency:
 * F_l = (E_p f_p + E_d f_d) / (E_p + E_d) with E = P * T, the frequencies weighted by
 * the phases' energies. */
static void or_averages(const or_lut *L, int jp, int kp, int jd, int kd, double tp, double pp, double td,
                        double pd, double *sm_pref, double *f_pref) {
  const double sp = (double)L->sm_level[jp], sd = (double)L->sm_level[jd];
  const double fp = (double)L->freq_level[kp], fd = (double)L->freq_level[kd];
  *sm_pref = (sp * tp + sd * td) / (tp + td);
  *f_pref = (pp * tp * fp + pd * td * fd) / (pp * tp + pd * td);
}

static void or_preferred_one(const or_lut *L, const or_llms *Q, int g, int i, or_pref *o) {
  double tp = 0, pp = 0, td = 0, pd = 0;
  const int cp = or_phase_best(L, Q, g, i, 0, &tp, &pp);
  const int cd = or_phase_best(L, Q, g, i, 1, &td, &pd);
  o->sm_p = cp < 0 ? -1 : cp / L->n_freq;
  o->f_p = cp < 0 ? -1 : cp % L->n_freq;
  o->sm_d = cd < 0 ? -1 : cd / L->n_freq;
  o->f_d = cd < 0 ? -1 : cd % L->n_freq;
  o->t_p = tp;
  o->p_p = pp;
  o->t_d = td;
  o->p_d = pd;
  o->feasible = cp >= 0 && cd >= 0;
  if (o->feasible) {
    or_averages(L, o->sm_p, o->f_p, o->sm_d, o->f_d, tp, pp, td, pd, &o->sm_pref, &o->f_pref);
  } else {
    o->sm_pref = NAN;
    o->f_pref = NAN;
  }
}

/* Preferred configuration of every instance slot [G][K]; slots past n_inst (or a GPU with
 * n_inst outside [0, K]) are infeasible. */
int festina_oracle_preferred(const or_lut *L, const or_llms *Q, or_pref *out) {
  if (!or_lut_ok(L) || !Q || !out || Q->n_gpus < 0 || Q->max_inst < 1) return 1;
  for (int g = 0; g < Q->n_gpus; ++g)
    for (int i = 0; i < Q->max_inst; ++i) {
      or_pref *o = &out[(size_t)g * Q->max_inst + (size_t)i];
      const int n = Q->n_inst[g];
      if (n < 0 || n > Q->max_inst || i >= n) {
        o->sm_p = o->f_p = o->sm_d = o->f_d = -1;
        o->t_p = o->t_d = o->p_p = o->p_d = 0.0;
        o->sm_pref = o->f_pref = NAN;
        o->feasible = 0;
        continue;
      }
      or_preferred_one(L, Q, g, i, o);
    }
  return 0;
}

/* Energy of one phase at a given cell (for checking another implementation's choice):
 * 1 and the duration/power when the cell is feasible. */
int festina_oracle_phase_cell(const or_lut *L, const or_llms *Q, int32_t g, int32_t i, int32_t decode,
                              int32_t j, int32_t k, double *t_out, double *p_out) {
  if (!or_lut_ok(L) || !Q || g < 0 || g >= Q->n_gpus || i < 0 || i >= Q->max_inst) return 0;
  if (j < 0 || j >= L->n_sm || k < 0 || k >= L->n_freq) return 0;
  const size_t at = (size_t)g * Q->max_inst + (size_t)i;
  const int n = Q->n_inst[g];
  if (n < 0 || n > Q->max_inst || i >= n) return 0;
  const int m = Q->model[at];
  const int32_t B = Q->batch[at];
  const int prow = or_prompt_row(Q->avg_in_tokens[at]);
  if (m < 0 || m >= L->n_models || B < 0 || prow < 0 || Q->avg_out_tokens[at] < 0) return 0;
  const int b = (B + 1 > OR_ROWS) ? OR_ROWS : B + 1;
  const float lat = decode ? L->dc[or_cell(L, m, b - 1, j, k)] : L->pf[or_cell(L, m, prow, j, k)];
  const float slo = decode ? Q->slo_tbt_ms[at] : Q->slo_ttft_ms[at];
  if (!(lat < slo)) return 0;
  const double P = L->p0_w + (double)Q->k_dyn_w[g] * (double)L->sm_level[j] * or_cube((double)L->freq_level[k]) *
                                 ((double)b / 32.0);
  const double t = decode ? (double)Q->avg_out_tokens[at] * (double)lat : (double)lat;
  if (!((float)(P * t) < INFINITY)) return 0;
  *t_out = t;
  *p_out = P;
  return 1;
}

/* Eq. energy_waste, energy_optimal, energy_waste_ratio over a fleet of instance slots.
 * Instances with a non-finite preferred frequency or execution time, or past n_inst, are
 * left out.  F_g = the highest preferred frequency on GPU g (0 with no instance);
 * waste_g = sum t_l (F_g^3 - F_l^3); totals[0] = sum waste_g, totals[1] = sum t_l F_l^3,
 * totals[2] = totals[0] / totals[1]. */
int festina_oracle_fleet_ewr(int32_t n_gpus, int32_t max_inst, const int32_t *n_inst, const float *f_pref,
                             const float *t_ms, double *f_gpu, double *waste_gpu, double *totals) {
  if (n_gpus < 0 || max_inst < 1 || !n_inst || !f_pref || !t_ms || !f_gpu || !waste_gpu || !totals) return 1;
  double waste = 0.0, opt = 0.0;
  for (int g = 0; g < n_gpus; ++g) {
    const int n = n_inst[g];
    double fg = 0.0;
    for (int i = 0; i < max_inst; ++i) {
      const size_t at = (size_t)g * max_inst + (size_t)i;
      if (n < 0 || n > max_inst || i >= n || !isfinite(f_pref[at]) || !isfinite(t_ms[at])) continue;
      if ((double)f_pref[at] > fg) fg = (double)f_pref[at];
    }
    double wg = 0.0;
    for (int i = 0; i < max_inst; ++i) {
      const size_t at = (size_t)g * max_inst + (size_t)i;
      if (n < 0 || n > max_inst || i >= n || !isfinite(f_pref[at]) || !isfinite(t_ms[at])) continue;
      const double fl = (double)f_pref[at], t = (double)t_ms[at];
      wg += t * (or_cube(fg) - or_cube(fl));
      opt += t * or_cube(fl);
    }
    f_gpu[g] = fg;
    waste_gpu[g] = wg;
    waste += wg;
  }
  totals[0] = waste;
  totals[1] = opt;
  totals[2] = waste / opt;
  return 0;
}

/* The two averages of instance (g, i) at given cells of each phase (for checking another
 * implementation's near-tie choice): 1 when both cells are feasible. */
int festina_oracle_preferred_at(const or_lut *L, const or_llms *Q, int32_t g, int32_t i, int32_t jp, int32_t kp,
                                int32_t jd, int32_t kd, double *sm_pref, double *f_pref) {
  double tp, pp, td, pd;
  if (!festina_oracle_phase_cell(L, Q, g, i, 0, jp, kp, &tp, &pp)) return 0;
  if (!festina_oracle_phase_cell(L, Q, g, i, 1, jd, kd, &td, &pd)) return 0;
  or_averages(L, jp, kp, jd, kd, tp, pp, td, pd, sm_pref, f_pref);
  return 1;
}

/* ---------------------------------------------------------------- current-frequency dispatch */
/* Sec. 3.3 as the paper runs it: every GPU offers one operating point, its current
 * frequency F_curr and the SMs free when the request's memory becomes available.
 * Phase One: GPU g's local scheduler reports a free-memory profile (from time t_s on,
 * mem_s MiB and SM level sm_s are free; t_s non-decreasing); the request needs
 * Req_mem = kv_kib_per_token[m] * (prompt + Lout) KiB; T_avail is the first t_s whose
 * mem_s covers it and SM_free that step's SM level.  g is feasible when
 * T_avail + TTFT(SM_free, F_curr) < slo_ttft and TBT(SM_free, F_curr) < slo_tbt.
 * Phase Two: E_g = Power(F_curr) x Latency = P * (TTFT + Lout * TBT); the least E wins,
 * but every candidate within 2% of it (E_g <= E_min + 0.02 |E_min|) ties, and among those the most
 * free memory, then the most free SMs, then the lowest GPU id wins.
 * Phase Three: no candidate -> GPUs ordered by T_avail (then id); the first that meets
 * the SLO at F_max (the top level) with its SM_free takes the request.  Else a new GPU
 * (batch 1, every SM, available now, k = k_new) at its least-energy feasible level.
 * Energies are float64 in a fixed order (the kernels use the same order, so both sides
 * take the 2% decision on identical values). */
typedef struct {
  int32_t n_gpus, n_steps;
  const int32_t *freq_cur;         /* [G] */
  const int32_t *batch;            /* [G] */
  const float *k_dyn_w;            /* [G] */
  const uint32_t *resident;        /* [G][words] */
  const float *t_avail_ms;         /* [G][S] */
  const int32_t *mem_free_mib;     /* [G][S] */
  const int32_t *sm_free;          /* [G][S] SM level index, -1 = none */
  const int32_t *kv_kib_per_token; /* [M] */
  float k_new_w;                   /* k of a newly activated GPU */
} or_avail;

typedef struct {
  int32_t gpu, freq_level, sm_level, phase;   /* phase: 1 = Phase Two, 2 = F_max fallback,
                                                 3 = new GPU, 0 = nothing feasible */
  double energy;
} or_dispatch;

#define OR_STABILITY 0.02

/* Energy of the request on one operating point; the order of operations is fixed. */
static double or_dispatch_energy(double p0, double kg, double s, double f, double u, double ttft, double lout,
                                 double tbt) {
  const double P = p0 + kg * s * (f * f * f) * u;
  return P * (ttft + lout * tbt);
}

/* Phase One for GPU g: 1 when g hosts the model and some profile step holds the memory;
 * then the step's time and SM level. */
static int or_avail_step(const or_lut *L, const or_avail *A, int g, int m, int64_t need_kib, double *t_avail,
                         int *sm, int *mem) {
  const int words = (L->n_models + 31) / 32;
  if (!((A->resident[(size_t)g * words + (size_t)(m / 32)] >> (m % 32)) & 1u)) return 0;
  for (int s = 0; s < A->n_steps; ++s) {
    const size_t at = (size_t)g * A->n_steps + (size_t)s;
    if ((int64_t)A->mem_free_mib[at] * 1024 >= need_kib) {
      *t_avail = (double)A->t_avail_ms[at];
      *sm = A->sm_free[at];
      *mem = A->mem_free_mib[at];
      return 1;
    }
  }
  return 0;
}

/* Does the request meet both SLOs on GPU g's point (level j, frequency k, start t_avail)?
 * Sets the energy when it does. */
static int or_point_ok(const or_lut *L, const or_requests *Q, int r, int m, int prow, int b, int j, int k,
                       double t_avail, double kg, double *energy) {
  if (j < 0 || j >= L->n_sm || k < 0 || k >= L->n_freq) return 0;
  const float ttft = L->pf[or_cell(L, m, prow >= 0 ? prow : b - 1, j, k)];
  const float tbt = L->dc[or_cell(L, m, b - 1, j, k)];
  if (!(t_avail + (double)ttft < (double)Q->slo_ttft_ms[r] && tbt < Q->slo_tbt_ms[r])) return 0;
  const double lout = (double)or_padded_out(Q->pred_out_tokens[r]);
  const double e = or_dispatch_energy(L->p0_w, kg, (double)L->sm_level[j], (double)L->freq_level[k],
                                      (double)b / 32.0, (double)ttft, lout, (double)tbt);
  if (!((float)e < INFINITY)) return 0;
  *energy = e;
  return 1;
}

/* Req_mem in KiB: the model's KV cache per token times the prompt and the padded output. */
static int64_t or_request_kib(const or_avail *A, const or_requests *Q, int r) {
  return (int64_t)A->kv_kib_per_token[Q->model[r]] * ((int64_t)Q->prompt_tokens[r] + or_padded_out(Q->pred_out_tokens[r]));
}

static void or_dispatch_one(const or_lut *L, const or_avail *A, const or_requests *Q, int r, or_dispatch *o) {
  o->gpu = o->freq_level = o->sm_level = -1;
  o->phase = 0;
  o->energy = INFINITY;
  const int m = (r >= 0 && r < Q->n_requests) ? Q->model[r] : -1;
  if (m < 0 || m >= L->n_models || Q->pred_out_tokens[r] < 0) return;
  const int prow = or_prompt_row(Q->prompt_tokens[r]);
  if (prow == -2) return;
  const int64_t need = or_request_kib(A, Q, r);
  /* Phase One and the least energy */
  double emin = INFINITY;
  int any = 0;
  for (int g = 0; g < A->n_gpus; ++g) {
    double ta, e;
    int sm, mem;
    if (!or_avail_step(L, A, g, m, need, &ta, &sm, &mem)) continue;
    const int32_t B = A->batch[g];
    if (B < 0) continue;
    const int b = B + 1 > OR_ROWS ? OR_ROWS : B + 1;
    if (!or_point_ok(L, Q, r, m, prow, b, sm, A->freq_cur[g], ta, (double)A->k_dyn_w[g], &e)) continue;
    if (!any || e < emin) emin = e;
    any = 1;
  }
  if (any) {
    /* Phase Two with the stability tie-break */
    const double bound = emin + OR_STABILITY * fabs(emin);
    int bg = -1, bmem = 0, bsm = 0;
    double be = 0.0;
    for (int g = 0; g < A->n_gpus; ++g) {
      double ta, e;
      int sm, mem;
      if (!or_avail_step(L, A, g, m, need, &ta, &sm, &mem)) continue;
      const int32_t B = A->batch[g];
      if (B < 0) continue;
      const int b = B + 1 > OR_ROWS ? OR_ROWS : B + 1;
      if (!or_point_ok(L, Q, r, m, prow, b, sm, A->freq_cur[g], ta, (double)A->k_dyn_w[g], &e)) continue;
      if (!(e <= bound)) continue;
      if (bg < 0 || mem > bmem || (mem == bmem && sm > bsm)) {
        bg = g;
        bmem = mem;
        bsm = sm;
        be = e;
      }
    }
    o->gpu = bg;
    o->freq_level = A->freq_cur[bg];
    o->sm_level = bsm;
    o->phase = 1;
    o->energy = be;
    return;
  }
  /* Phase Three: the earliest available GPU that meets the SLO at F_max */
  const int kmax = L->n_freq - 1;
  int bg = -1, bsm = -1;
  double bt = INFINITY, be = 0.0;
  for (int g = 0; g < A->n_gpus; ++g) {
    double ta, e;
    int sm, mem;
    if (!or_avail_step(L, A, g, m, need, &ta, &sm, &mem)) continue;
    const int32_t B = A->batch[g];
    if (B < 0) continue;
    const int b = B + 1 > OR_ROWS ? OR_ROWS : B + 1;
    if (!or_point_ok(L, Q, r, m, prow, b, sm, kmax, ta, (double)A->k_dyn_w[g], &e)) continue;
    if (bg < 0 || ta < bt) {
      bg = g;
      bt = ta;
      bsm = sm;
      be = e;
    }
  }
  if (bg >= 0) {
    o->gpu = bg;
    o->freq_level = kmax;
    o->sm_level = bsm;
    o->phase = 2;
    o->energy = be;
    return;
  }
  /* scale out: a new GPU, every SM free now, batch 1, its least-energy feasible level */
  int bk = -1;
  for (int k = 0; k < L->n_freq; ++k) {
    double e;
    if (!or_point_ok(L, Q, r, m, prow, 1, L->n_sm - 1, k, 0.0, (double)A->k_new_w, &e)) continue;
    if (bk < 0 || e < be) {
      bk = k;
      be = e;
    }
  }
  if (bk >= 0) {
    o->freq_level = bk;
    o->sm_level = L->n_sm - 1;
    o->phase = 3;
    o->energy = be;
  }
}

int festina_oracle_dispatch(const or_lut *L, const or_avail *A, const or_requests *Q, int32_t n_sel,
                            const int32_t *sel, or_dispatch *out) {
  if (!or_lut_ok(L) || !A || !Q || !out || A->n_gpus < 0 || A->n_steps < 1 || Q->n_requests < 0) return 1;
  const int32_t n = sel ? n_sel : Q->n_requests;
  for (int32_t i = 0; i < n; ++i) or_dispatch_one(L, A, Q, sel ? sel[i] : i, &out[i]);
  return 0;
}

/* The same dispatcher run over arrival waves, each wave committed before the next one is
 * dispatched (Sec. 3.3 decides one request at a time against the state its local
 * schedulers report; here the requests of one wave share a snapshot, and the waves follow
 * one another).  Requests are ordered by wave: wave w is requests wave_start[w] ..
 * wave_start[w+1]-1.  After every request of a wave is decided, each one placed on a GPU of
 * the table (Phase Two, or the F_max fallback) is committed to that GPU:
 *   its decode batch grows by one (B -> B + 1, so the next request sees row b = min(B+2, 32));
 *   it holds its memory from its start on: every profile step from the one that admitted it
 *   loses ceil(Req_mem / 1024) MiB (a step short of memory reads -1 MiB: nothing fits);
 *   an F_max placement leaves the GPU at the top frequency level (it was boosted).
 * Free SM levels and the profile's times stay as reported; a new GPU (Phase Three's scale
 * out) is not a row of the table and commits nothing.  The state after the last wave is
 * returned in freq_out [G], batch_out [G] and mem_out [G][S]. */
int festina_oracle_dispatch_waves(const or_lut *L, const or_avail *A, const or_requests *Q, int32_t n_waves,
                                  const int32_t *wave_start, int32_t *freq_out, int32_t *batch_out,
                                  int32_t *mem_out, or_dispatch *out) {
  if (!or_lut_ok(L) || !A || !Q || !out || !freq_out || !batch_out || !mem_out || A->n_gpus < 0 ||
      A->n_steps < 1 || Q->n_requests < 0 || n_waves < 0 || (n_waves > 0 && !wave_start))
    return 1;
  if (n_waves == 0 ? Q->n_requests != 0 : (wave_start[0] != 0 || wave_start[n_waves] != Q->n_requests)) return 1;
  for (int32_t w = 0; w < n_waves; ++w)
    if (wave_start[w + 1] < wave_start[w]) return 1;
  const int G = A->n_gpus, S = A->n_steps;
  for (int g = 0; g < G; ++g) {
    freq_out[g] = A->freq_cur[g];
    batch_out[g] = A->batch[g];
    for (int s = 0; s < S; ++s) mem_out[(size_t)g * S + s] = A->mem_free_mib[(size_t)g * S + s];
  }
  int32_t *snap = (int32_t *)malloc(sizeof(int32_t) * ((size_t)G * S + 1));
  if (!snap) return 1;
  or_avail now = *A;              /* the state the wave sees */
  now.freq_cur = freq_out;
  now.batch = batch_out;
  now.mem_free_mib = snap;
  for (int32_t w = 0; w < n_waves; ++w) {
    memcpy(snap, mem_out, sizeof(int32_t) * (size_t)G * S);
    for (int32_t r = wave_start[w]; r < wave_start[w + 1]; ++r) or_dispatch_one(L, &now, Q, r, &out[r]);
    /* decisions first (on the snapshot), then the commits */
    int32_t *boost = (int32_t *)calloc((size_t)G + 1, sizeof(int32_t));
    int32_t *grow = (int32_t *)calloc((size_t)G + 1, sizeof(int32_t));
    int64_t *taken = (int64_t *)calloc((size_t)G * S + 1, sizeof(int64_t));
    if (!boost || !grow || !taken) {
      free(boost), free(grow), free(taken), free(snap);
      return 1;
    }
    for (int32_t r = wave_start[w]; r < wave_start[w + 1]; ++r) {
      const int g = out[r].gpu;
      if (out[r].phase != 1 && out[r].phase != 2) continue;
      const int64_t need = or_request_kib(A, Q, r);
      int first = 0;                /* the admitting step: the first whose memory holds Req_mem */
      while ((int64_t)snap[(size_t)g * S + first] * 1024 < need) ++first;
      for (int s = first; s < S; ++s) taken[(size_t)g * S + s] += (need + 1023) / 1024;
      grow[g] += 1;
      if (out[r].phase == 2) boost[g] = 1;
    }
    for (int g = 0; g < G; ++g) {
      batch_out[g] += grow[g];
      if (boost[g]) freq_out[g] = L->n_freq - 1;
      for (int s = 0; s < S; ++s) {
        const int64_t v = (int64_t)mem_out[(size_t)g * S + s] - taken[(size_t)g * S + s];
        mem_out[(size_t)g * S + s] = (int32_t)(v < -1 ? -1 : v);
      }
    }
    free(boost), free(grow), free(taken);
  }
  free(snap);
  return 0;
}

/* ---------------------------------------------------------------- transfer plan (App. F) */
/* "Transmission plan (device mapping)": the cost of sending the state now on GPU u to GPU v
 * is e_uv = Bytes(u -> v) / BW(u, v), the input of the minimum-cost assignment.  Bytes
 * counts the weights of u's resident models that v does not already hold plus u's request
 * state selected for migration; keeping the state in place costs nothing (e_uu = 0).  BW
 * is the intra-node link bandwidth between GPUs of one node, else the inter-node one.
 * Times in ms: e = bytes * ms_per_byte, ms_per_byte = 1e3 / (GB/s * 1e9), in float64.
 * "Selective request migration" and "what to transfer": an in-flight request on source u
 * whose state goes to v = dest[u] moves only when its remaining decode time at u exceeds
 * its migration time; it then moves its tokens plus either its KV cache or a recompute of
 * it on v, whichever is faster. */
typedef struct {
  int32_t n_gpus, words;
  const uint32_t *resident;        /* [G][words] models resident now */
  const int32_t *weights_mib;      /* [M] */
  const int32_t *state_mib;        /* [G] request state selected for migration */
  const int32_t *node;             /* [G] */
  float bw_intra_gbs, bw_inter_gbs;
} or_transfer;

static double or_ms_per_byte(double gbs) { return 1e3 / (gbs * 1e9); }

static double or_link_ms_per_byte(const or_transfer *T, int u, int v) {
  return T->node[u] == T->node[v] ? or_ms_per_byte((double)T->bw_intra_gbs) : or_ms_per_byte((double)T->bw_inter_gbs);
}

int festina_oracle_transfer_costs(const or_transfer *T, int32_t n_models, double *cost) {
  if (!T || !cost || T->n_gpus < 0 || T->words < (n_models + 31) / 32 || n_models < 1) return 1;
  for (int u = 0; u < T->n_gpus; ++u)
    for (int v = 0; v < T->n_gpus; ++v) {
      double e = 0.0;
      if (u != v) {
        int64_t mib = T->state_mib[u];
        for (int m = 0; m < n_models; ++m) {
          const int on_u = (T->resident[(size_t)u * T->words + (size_t)(m / 32)] >> (m % 32)) & 1u;
          const int on_v = (T->resident[(size_t)v * T->words + (size_t)(m / 32)] >> (m % 32)) & 1u;
          if (on_u && !on_v) mib += T->weights_mib[m];
        }
        e = (double)(mib * 1048576) * or_link_ms_per_byte(T, u, v);
      }
      cost[(size_t)u * T->n_gpus + (size_t)v] = e;
    }
  return 0;
}

typedef struct {
  int32_t n_requests;
  const int32_t *src;              /* [Q] source GPU */
  const int32_t *model;            /* [Q] */
  const int32_t *context_tokens;   /* [Q] prompt + generated so far */
  const int32_t *remaining_tokens; /* [Q] predicted tokens still to generate */
  const int32_t *kv_kib;           /* [Q] KV-cache size */
  const int32_t *token_kib;        /* [Q] token state (prompt and generated ids) */
} or_moves;

typedef struct {
  const int32_t *dest;             /* [G] destination of each GPU's state (the plan) */
  const int32_t *freq_cur, *sm_cur, *batch;   /* [G] operating point and decode batch */
} or_plan;

/* decision: 0 = finish on the source (or the state stays), 1 = move with the KV cache,
 * 2 = move the tokens and recompute the KV cache on the destination, -1 = invalid request
 * (GPU, model, level or token count out of range); times 0 unless computed. */
int festina_oracle_request_moves(const or_lut *L, const or_transfer *T, const or_plan *P, const or_moves *Q,
                                 int32_t *decision, double *remaining_ms, double *migrate_ms) {
  if (!or_lut_ok(L) || !T || !P || !Q || !decision || !remaining_ms || !migrate_ms) return 1;
  for (int q = 0; q < Q->n_requests; ++q) {
    decision[q] = -1;
    remaining_ms[q] = 0.0;
    migrate_ms[q] = 0.0;
    const int u = Q->src[q], m = Q->model[q];
    if (u < 0 || u >= T->n_gpus || m < 0 || m >= L->n_models) continue;
    const int v = P->dest[u];
    if (v < 0 || v >= T->n_gpus) continue;
    const int ju = P->sm_cur[u], ku = P->freq_cur[u], jv = P->sm_cur[v], kv = P->freq_cur[v];
    const int32_t Bu = P->batch[u];
    const int crow = or_prompt_row(Q->context_tokens[q]);
    if (ju < 0 || ju >= L->n_sm || ku < 0 || ku >= L->n_freq || jv < 0 || jv >= L->n_sm || kv < 0 ||
        kv >= L->n_freq || Bu < 0 || crow < 0 || Q->remaining_tokens[q] < 0 || Q->kv_kib[q] < 0 || Q->token_kib[q] < 0)
      continue;
    decision[q] = 0;
    const int bu = Bu + 1 > OR_ROWS ? OR_ROWS : Bu + 1;
    const double rem = (double)Q->remaining_tokens[q] * (double)L->dc[or_cell(L, m, bu - 1, ju, ku)];
    remaining_ms[q] = rem;
    if (v == u) continue;                        /* the state stays: nothing to move */
    const double mpb = or_link_ms_per_byte(T, u, v);
    const double kv_ms = (double)((int64_t)Q->kv_kib[q] * 1024) * mpb;
    const double tok_ms = (double)((int64_t)Q->token_kib[q] * 1024) * mpb;
    const double rec_ms = (double)L->pf[or_cell(L, m, crow, jv, kv)];
    const int use_kv = kv_ms < rec_ms;
    const double mig = tok_ms + (use_kv ? kv_ms : rec_ms);
    migrate_ms[q] = mig;
    if (rem > mig) decision[q] = use_kv ? 1 : 2;
  }
  return 0;
}
