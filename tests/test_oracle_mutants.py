"""The oracle's pins must reject plausible mistakes.

Each case plants one mistake in a copy of the oracle's C source (a dropped term, a
wrong sign or index, an inclusive instead of a strict test, a swapped operand),
compiles it on the CPU, and runs the pin suites against that library: they must
fail.  Nothing here touches a GPU or the HIP library.
"""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(ROOT, "oracle", "festina_oracle.c")

PLACEMENT = [
    ("dropped decode term", "const double E = Pp * (double)ttft + Lout * Pd * (double)tbt;",
     "const double E = Pp * (double)ttft;"),
    ("f instead of f^3", "const double f3 = or_cube((double)L->freq_level[k]);\n  const double kg = (double)G->k_dyn_w[g];",
     "const double f3 = (double)L->freq_level[k];\n  const double kg = (double)G->k_dyn_w[g];"),
    ("inclusive SLO test", "if (!(ttft < Q->slo_ttft_ms[r] && tbt < Q->slo_tbt_ms[r])) return 0;",
     "if (!(ttft <= Q->slo_ttft_ms[r] && tbt <= Q->slo_tbt_ms[r])) return 0;"),
    ("pre-admission batch in u", "const double u = (double)b / 32.0;\n  const double f3",
     "const double u = (double)B / 32.0;\n  const double f3"),
    ("TTFT read from the batch row", "L->pf[or_cell(L, m, row_p, jp, k)]", "L->pf[or_cell(L, m, b - 1, jp, k)]"),
    ("decode cap taken from prefill cap", "const int jd = j < cd ? j : cd;", "const int jd = j < cp ? j : cp;"),
    ("highest index wins ties", "if (best_idx < 0 || e < best_e) {", "if (best_idx < 0 || e <= best_e) {"),
    ("floor instead of ceil in the 5% pad", "((int64_t)predicted * 105 + 99) / 100", "((int64_t)predicted * 105) / 100"),
    ("prompt bucket off by one", "((int64_t)tokens + OR_ROW_TOKENS - 1) / OR_ROW_TOKENS",
     "((int64_t)tokens + OR_ROW_TOKENS) / OR_ROW_TOKENS"),
    ("uncapped SM level in prefill power", "const double Pp = L->p0_w + kg * (double)L->sm_level[jp]",
     "const double Pp = L->p0_w + kg * (double)L->sm_level[j]"),
    ("wrong sign of dynamic power", "const double Pd = L->p0_w + kg", "const double Pd = L->p0_w - kg"),
]

MIGRATION = [
    ("destination baseline level from the source", "if (or_gpu_ok(L, F, d, k)) kd0 = k;",
     "if (or_gpu_ok(L, F, s, k)) kd0 = k;"),
    ("strict HBM budget", "> (int64_t)F->hbm_cap_mib) return 0;", ">= (int64_t)F->hbm_cap_mib) return 0;"),
    ("saving sign flipped", "const double sv = L->p0_w - kd * added;", "const double sv = L->p0_w + kd * added;"),
    ("destination SLOs ignored", "if (or_gpu_ok(L, F, s, k) && or_gpu_ok(L, F, d, k)) kstar = k;",
     "if (or_gpu_ok(L, F, s, k)) kstar = k;"),
    ("instance TTFT read from the batch row", "L->pf[or_cell(L, m, row_p, j, k)]",
     "L->pf[or_cell(L, m, b - 1, j, k)]"),
    ("merged load drops u_d", "* (us + ud) - or_cube", "* us - or_cube"),
    ("source may move onto itself", "if (s < 0 || d < 0 || s >= F->n_gpus || d >= F->n_gpus || s == d) return 0;",
     "if (s < 0 || d < 0 || s >= F->n_gpus || d >= F->n_gpus) return 0;"),
]


SWEEP = [
    ("inclusive slack test", "if (or_task_latency(L, S, b, t, row, j, k) < slack) return j;",
     "if (or_task_latency(L, S, b, t, row, j, k) <= slack) return j;"),
    ("inclusive SM budget", "if (!(units < (int64_t)S->sm_budget)) return 0;",
     "if (!(units <= (int64_t)S->sm_budget)) return 0;"),
    ("dropped static power", "E += (L->p0_w + dyn) * lat;", "E += dyn * lat;"),
    ("utilisation dropped", "const double dyn = kg * (double)L->sm_level[j] * f3 * u;",
     "const double dyn = kg * (double)L->sm_level[j] * f3;"),
    ("f instead of f^3", "const double f3 = or_cube((double)L->freq_level[k]);\n  const double kg = (double)S->k_dyn_w[b]",
     "const double f3 = (double)L->freq_level[k];\n  const double kg = (double)S->k_dyn_w[b]"),
    ("decode reads the prefill table", "const float *tab = S->task_phase[at] == 0 ? L->pf : L->dc;",
     "const float *tab = L->pf;"),
    ("largest SM level instead of smallest",
     "for (int j = 0; j < L->n_sm; ++j)\n    if (or_task_latency",
     "for (int j = L->n_sm - 1; j >= 0; --j)\n    if (or_task_latency"),
    ("decode row off by one", "if (ph == 1) return (tok > OR_ROWS ? OR_ROWS : tok) - 1;",
     "if (ph == 1) return tok >= OR_ROWS ? OR_ROWS - 1 : tok;"),
    ("longest task instead of the sum", "      E += (L->p0_w + dyn) * lat;",
     "      E = E > (L->p0_w + dyn) * lat ? E : (L->p0_w + dyn) * lat;"),
    ("per-batch static power over the sum of latencies", "if (lat > longest) longest = lat;", "longest += lat;"),
    ("per-batch static power dropped", "if (S->static_power != 0) E += L->p0_w * longest;", ""),
    ("per-batch reading charges static power per task", "if (S->static_power == 0) {", "if (1) {"),
    ("per-batch dynamic terms of the longest task only", "      E += dyn * lat;\n", "      E = E > dyn * lat ? E : dyn * lat;\n"),
    ("highest level wins ties", "      if (bk < 0 || e < be) {", "      if (bk < 0 || e <= be) {"),
]


PREFERRED = [
    ("inclusive SLO in the phase search", "      if (!(lat < slo)) continue;", "      if (!(lat <= slo)) continue;"),
    ("decode duration without the output length",
     "const double t = decode ? (double)Q->avg_out_tokens[at] * (double)lat : (double)lat;\n      const double e",
     "const double t = (double)lat;\n      const double e"),
    ("time-weighted frequency", "*f_pref = (pp * tp * fp + pd * td * fd) / (pp * tp + pd * td);",
     "*f_pref = (tp * fp + td * fd) / (tp + td);"),
    ("energy-weighted SM share", "*sm_pref = (sp * tp + sd * td) / (tp + td);",
     "*sm_pref = (pp * tp * sp + pd * td * sd) / (pp * tp + pd * td);"),
    ("averages at given cells take the decode cell for both phases",
     "or_averages(L, jp, kp, jd, kd, tp, pp, td, pd, sm_pref, f_pref);",
     "or_averages(L, jd, kd, jd, kd, tp, pp, td, pd, sm_pref, f_pref);"),
    ("averages at given cells swap the phases' durations",
     "or_averages(L, jp, kp, jd, kd, tp, pp, td, pd, sm_pref, f_pref);",
     "or_averages(L, jp, kp, jd, kd, td, pp, tp, pd, sm_pref, f_pref);"),
    ("decode cell tested as a prefill cell", "if (!festina_oracle_phase_cell(L, Q, g, i, 1, jd, kd, &td, &pd)) return 0;",
     "if (!festina_oracle_phase_cell(L, Q, g, i, 0, jd, kd, &td, &pd)) return 0;"),
    ("decode reads the prompt row", "      const float lat = decode ? L->dc[or_cell(L, m, b - 1, j, k)]",
     "      const float lat = decode ? L->dc[or_cell(L, m, prow, j, k)]"),
    ("pre-admission batch in the phase power", "const double u = (double)b / 32.0;\n  const double kg = (double)Q->k_dyn_w[g];",
     "const double u = (double)B / 32.0;\n  const double kg = (double)Q->k_dyn_w[g];"),
    ("highest cell wins phase ties", "      if (best < 0 || e < best_e) {", "      if (best < 0 || e <= best_e) {"),
    ("GPU frequency from the last LLM", "if ((double)f_pref[at] > fg) fg = (double)f_pref[at];", "fg = (double)f_pref[at];"),
    ("optimal energy at the GPU frequency", "opt += t * or_cube(fl);", "opt += t * or_cube(fg);"),
    ("waste without the cube", "wg += t * (or_cube(fg) - or_cube(fl));", "wg += t * (fg - fl);"),
]


DISPATCH = [
    ("no stability margin", "#define OR_STABILITY 0.02", "#define OR_STABILITY 0.0"),
    ("least memory wins the tie", "if (bg < 0 || mem > bmem || (mem == bmem && sm > bsm)) {",
     "if (bg < 0 || mem < bmem || (mem == bmem && sm > bsm)) {"),
    ("free SMs ignored in the tie", "if (bg < 0 || mem > bmem || (mem == bmem && sm > bsm)) {",
     "if (bg < 0 || mem > bmem) {"),
    ("memory demand without the output",
     "((int64_t)Q->prompt_tokens[r] + or_padded_out(Q->pred_out_tokens[r]))", "((int64_t)Q->prompt_tokens[r])"),
    ("waiting time ignored", "if (!(t_avail + (double)ttft < (double)Q->slo_ttft_ms[r]",
     "if (!((double)ttft < (double)Q->slo_ttft_ms[r]"),
    ("fallback at the current frequency", "if (!or_point_ok(L, Q, r, m, prow, b, sm, kmax, ta,",
     "if (!or_point_ok(L, Q, r, m, prow, b, sm, A->freq_cur[g], ta,"),
    ("fallback to the latest GPU", "if (bg < 0 || ta < bt) {", "if (bg < 0 || ta >= bt) {"),
    ("new GPU at full batch", "if (!or_point_ok(L, Q, r, m, prow, 1, L->n_sm - 1, k, 0.0,",
     "if (!or_point_ok(L, Q, r, m, prow, 32, L->n_sm - 1, k, 0.0,"),
    ("first profile step whatever its memory", "if ((int64_t)A->mem_free_mib[at] * 1024 >= need_kib) {",
     "if (1) {"),
    ("dispatch power without utilisation", "const double P = p0 + kg * s * (f * f * f) * u;",
     "const double P = p0 + kg * s * (f * f * f);"),
]


WAVES = [
    ("memory taken from every step", "for (int s = first; s < S; ++s) taken", "for (int s = 0; s < S; ++s) taken"),
    ("batch does not grow", "batch_out[g] += grow[g];", ""),
    ("no boost after an F_max placement", "if (boost[g]) freq_out[g] = L->n_freq - 1;", ""),
    ("a wave sees its own commits", "memcpy(snap, mem_out, sizeof(int32_t) * (size_t)G * S);\n    for (int32_t r = wave_start[w]; r < wave_start[w + 1]; ++r) or_dispatch_one(L, &now, Q, r, &out[r]);",
     "memcpy(snap, mem_out, sizeof(int32_t) * (size_t)G * S);\n    for (int32_t r = wave_start[w]; r < wave_start[w + 1]; ++r) {\n      or_dispatch_one(L, &now, Q, r, &out[r]);\n      if (out[r].phase == 1 || out[r].phase == 2) { batch_out[out[r].gpu] += 1; for (int s = 0; s < S; ++s) snap[(size_t)out[r].gpu * S + s] -= (int32_t)((A->kv_kib_per_token[Q->model[r]] * ((int64_t)Q->prompt_tokens[r] + or_padded_out(Q->pred_out_tokens[r])) + 1023) / 1024); }\n    }"),
    ("memory floor at zero", "(int32_t)(v < -1 ? -1 : v)", "(int32_t)(v < 0 ? 0 : v)"),
    ("demand rounded down", "taken[(size_t)g * S + s] += (need + 1023) / 1024;", "taken[(size_t)g * S + s] += need / 1024;"),
    ("F_max placement not committed", "if (out[r].phase != 1 && out[r].phase != 2) continue;",
     "if (out[r].phase != 1) continue;"),
]


TRANSFER = [
    ("weights the destination already holds", "if (on_u && !on_v) mib += T->weights_mib[m];",
     "if (on_u) mib += T->weights_mib[m];"),
    ("request state not counted", "int64_t mib = T->state_mib[u];", "int64_t mib = 0;"),
    ("link classes swapped", "return T->node[u] == T->node[v] ?", "return T->node[u] != T->node[v] ?"),
    ("cost on the diagonal", "      if (u != v) {\n        int64_t mib", "      if (1) {\n        int64_t mib"),
    ("remaining time at the destination", "L->dc[or_cell(L, m, bu - 1, ju, ku)]", "L->dc[or_cell(L, m, bu - 1, jv, kv)]"),
    ("recompute at the source", "L->pf[or_cell(L, m, crow, jv, kv)]", "L->pf[or_cell(L, m, crow, ju, ku)]"),
    ("always the KV cache", "const int use_kv = kv_ms < rec_ms;", "const int use_kv = 1;"),
    ("token state forgotten", "const double mig = tok_ms + (use_kv ? kv_ms : rec_ms);",
     "const double mig = (use_kv ? kv_ms : rec_ms);"),
    ("move at equal times", "if (rem > mig) decision[q]", "if (rem >= mig) decision[q]"),
]


def _run_pins(tmp_path, name, old, new, suite):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor not unique/present: {name}"
    mut = tmp_path / "mut.c"
    mut.write_text(src.replace(old, new))
    lib = tmp_path / "libmut.so"
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fPIC", "-shared", "-o", str(lib), str(mut), "-lm"],
                   check=True)
    env = dict(os.environ, FESTINA_ORACLE_LIB=str(lib))
    proc = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           os.path.join(HERE, suite)], cwd=ROOT, env=env,
                          stdout=subprocess.PIPE, stderr=subprocess.STDOUT, timeout=600)
    return proc.returncode, proc.stdout.decode()[-400:]


@pytest.mark.parametrize("name,old,new", PLACEMENT, ids=[p[0] for p in PLACEMENT])
def test_placement_pins_reject_mutant(tmp_path, name, old, new):
    rc, tail = _run_pins(tmp_path, name, old, new, "test_oracle_placement_pins.py")
    assert rc != 0, f"pins accepted the mutant '{name}':\n{tail}"


@pytest.mark.parametrize("name,old,new", MIGRATION, ids=[p[0] for p in MIGRATION])
def test_migration_pins_reject_mutant(tmp_path, name, old, new):
    rc, tail = _run_pins(tmp_path, name, old, new, "test_oracle_migration_pins.py")
    assert rc != 0, f"pins accepted the mutant '{name}':\n{tail}"


@pytest.mark.parametrize("name,old,new", SWEEP, ids=[p[0] for p in SWEEP])
def test_sweep_pins_reject_mutant(tmp_path, name, old, new):
    rc, tail = _run_pins(tmp_path, name, old, new, "test_oracle_sweep_pins.py")
    assert rc != 0, f"pins accepted the mutant '{name}':\n{tail}"


@pytest.mark.parametrize("name,old,new", PREFERRED, ids=[p[0] for p in PREFERRED])
def test_preferred_pins_reject_mutant(tmp_path, name, old, new):
    rc, tail = _run_pins(tmp_path, name, old, new, "test_oracle_preferred_pins.py")
    assert rc != 0, f"pins accepted the mutant '{name}':\n{tail}"


@pytest.mark.parametrize("name,old,new", DISPATCH, ids=[p[0] for p in DISPATCH])
def test_dispatch_pins_reject_mutant(tmp_path, name, old, new):
    rc, tail = _run_pins(tmp_path, name, old, new, "test_oracle_dispatch_pins.py")
    assert rc != 0, f"pins accepted the mutant '{name}':\n{tail}"


@pytest.mark.parametrize("name,old,new", TRANSFER, ids=[p[0] for p in TRANSFER])
def test_transfer_pins_reject_mutant(tmp_path, name, old, new):
    rc, tail = _run_pins(tmp_path, name, old, new, "test_oracle_transfer_pins.py")
    assert rc != 0, f"pins accepted the mutant '{name}':\n{tail}"


@pytest.mark.parametrize("name,old,new", WAVES, ids=[p[0] for p in WAVES])
def test_wave_dispatch_pins_reject_mutant(tmp_path, name, old, new):
    rc, tail = _run_pins(tmp_path, name, old, new, "test_oracle_dispatch_waves_pins.py")
    assert rc != 0, f"pins accepted the mutant '{name}':\n{tail}"
