"""Brute-force enumeration for tiny instances (test helper, not collected).

Written independently of the C oracle: request pre-processing uses exact
rationals, every candidate is listed, its energy is the sum over the two phases
of power x time (Eq. energy), and the answer is the minimum of the list under
the (energy, index) order -- no running minimum, no shared code.
"""
from __future__ import annotations

import itertools
import math
from fractions import Fraction

import numpy as np


def padded_out(pred: int) -> int:
    """ceil(1.05 * L) with exact rationals (5% safety pad, Sec. 3.2.2)."""
    return math.ceil(Fraction(105, 100) * pred)


def prompt_row(tokens: int):
    """None for invalid, -1 for no prompt, else the 256-token bucket row (rounded up)."""
    if tokens < 0:
        return None
    if tokens == 0:
        return -1
    return min(math.ceil(Fraction(tokens, 256)), 32) - 1


def power(p0, k, s, f, u):
    """Closed-form power model P0 + k * s * f^3 * u (W)."""
    return p0 + k * s * f ** 3 * u


def placement_candidates(inp, r):
    """All (energy, idx) of SLO-feasible candidates of request r, in float64."""
    lut, gp, rq = inp["lut"], inp["gpus"], inp["requests"]
    M, NS, NF = lut["n_models"], lut["n_sm"], lut["n_freq"]
    G, W = gp["n_gpus"], gp["n_waves"]
    m = int(rq["model"][r])
    w = int(rq["wave"][r]) if rq.get("wave") is not None else 0
    prow = prompt_row(int(rq["prompt_tokens"][r]))
    pred = int(rq["pred_out_tokens"][r])
    if not (0 <= m < M and 0 <= w < W) or prow is None or pred < 0:
        return []
    lout = padded_out(pred)
    out = []
    for g, j, k in itertools.product(range(G), range(NS), range(NF)):
        if not (int(gp["resident"][g, m // 32]) >> (m % 32)) & 1:
            continue
        B = int(gp["batch"][w, g])
        if B < 0:
            continue
        b = min(B + 1, 32)
        cap_p = NS - 1 if gp.get("cap_pf") is None else int(gp["cap_pf"][g])
        cap_d = NS - 1 if gp.get("cap_dc") is None else int(gp["cap_dc"][g])
        if not (0 <= cap_p < NS and 0 <= cap_d < NS):
            continue
        jp, jd = min(j, cap_p), min(j, cap_d)
        ttft = lut["pf"][m, b - 1 if prow < 0 else prow, jp, k]
        tbt = lut["dc"][m, b - 1, jd, k]
        if not (ttft < rq["slo_ttft_ms"][r] and tbt < rq["slo_tbt_ms"][r]):
            continue
        f = float(lut["freq_level"][k])
        u = b / 32
        kg = float(gp["k_dyn_w"][g])
        phases = [(float(lut["sm_level"][jp]), float(ttft)),
                  (float(lut["sm_level"][jd]), lout * float(tbt))]
        e = sum(power(lut["p0_w"], kg, s, f, u) * t for s, t in phases)
        if not np.float32(e) < np.inf:
            continue
        out.append((e, (g * NS + j) * NF + k))
    return out


def brute_placements(inp):
    R = inp["requests"]["n_requests"]
    choice = np.full(R, -1, np.int32)
    energy = np.full(R, np.inf)
    for r in range(R):
        c = placement_candidates(inp, r)
        if c:
            e, idx = min(c)
            choice[r], energy[r] = idx, e
    return choice, (choice >= 0).astype(np.uint8), energy


# ------------------------------------------------------------------ migration
def feasible_levels(inp, g):
    """Set of frequency levels at which every instance of GPU g meets both SLOs."""
    lut, fl = inp["lut"], inp["fleet"]
    NS, NF, M = lut["n_sm"], lut["n_freq"], lut["n_models"]
    n = int(fl["n_inst"][g])
    if not 1 <= n <= fl["max_inst"]:
        return set()
    levels = set(range(NF))
    for i in range(n):
        m = int(fl["inst_model"][g, i])
        j = int(fl["inst_sm"][g, i])
        B = int(fl["inst_batch"][g, i])
        prow = prompt_row(int(fl["inst_prompt_tokens"][g, i]))
        if not (0 <= m < M and 0 <= j < NS and B >= 0) or prow is None:
            return set()
        b = min(B + 1, 32)
        ok = {k for k in range(NF)
              if lut["pf"][m, b - 1 if prow < 0 else prow, j, k] < fl["inst_slo_ttft_ms"][g, i]
              and lut["dc"][m, b - 1, j, k] < fl["inst_slo_tbt_ms"][g, i]}
        levels &= ok
    return levels


def migration_pairs(inp, s):
    """All (saving, d, k_star) of feasible destinations of source s."""
    lut, fl = inp["lut"], inp["fleet"]
    G = fl["n_gpus"]
    fs = feasible_levels(inp, s)
    out = []
    for d in range(G):
        if d == s:
            continue
        if int(fl["hbm_mib"][s]) + int(fl["hbm_mib"][d]) > fl["hbm_cap_mib"]:
            continue
        if int(fl["sm_permille"][s]) + int(fl["sm_permille"][d]) > fl["sm_cap_permille"]:
            continue
        fd = feasible_levels(inp, d)
        both = fs & fd
        if not both:
            continue
        kstar, kd0 = min(both), min(fd)
        f = [float(x) for x in lut["freq_level"]]
        us, ud, kd = float(fl["util"][s]), float(fl["util"][d]), float(fl["k_dyn_w"][d])
        before = kd * f[kd0] ** 3 * ud                     # d's dynamic power alone
        after = kd * f[kstar] ** 3 * (us + ud)             # merged load at the shared level
        saving = lut["p0_w"] - (after - before)            # source's static power freed
        if not np.float32(saving) > -np.inf:
            continue
        out.append((saving, d, kstar))
    return out


def brute_migrations(inp):
    G = inp["fleet"]["n_gpus"]
    best = np.full(G, -1, np.int32)
    sav = np.full(G, -np.inf)
    lev = np.full(G, -1, np.int32)
    for s in range(G):
        p = migration_pairs(inp, s)
        if p:
            # largest saving, then lowest d
            sv, d, k = min(p, key=lambda t: (-t[0], t[1]))
            best[s], sav[s], lev[s] = d, sv, k
    return best, sav, lev


# ------------------------------------------------------------------ local sweep
def task_rows(inp, b):
    """Table and row of each task of batch b, or None when the batch holds an invalid task."""
    lut, bt = inp["lut"], inp["batches"]
    n = int(bt["n_tasks"][b])
    if not 0 <= n <= bt["max_tasks"]:
        return None
    out = []
    for t in range(n):
        m, ph, tok = int(bt["task_model"][b, t]), int(bt["task_phase"][b, t]), int(bt["task_tokens"][b, t])
        if not 0 <= m < lut["n_models"] or tok < 1 or ph not in (0, 1):
            return None
        if ph == 0:
            out.append((lut["pf"], m, prompt_row(tok)))
        else:
            out.append((lut["dc"], m, min(tok, 32) - 1))
    return out


def sweep_levels(inp, b):
    """All (energy, k, assignment) of usable frequency levels of batch b.

    Every SM assignment that meets all slacks is listed; the per-task minimum SM level is
    the componentwise minimum of that list, and the level is usable when that
    assignment's integer SM shares sum to less than the budget.
    """
    lut, bt = inp["lut"], inp["batches"]
    NS, NF = lut["n_sm"], lut["n_freq"]
    rows = task_rows(inp, b)
    if rows is None:
        return []
    n = len(rows)
    out = []
    for k in range(NF):
        ok = [a for a in itertools.product(range(NS), repeat=n)
              if all(tab[m, row, a[t], k] < bt["task_slack_ms"][b, t] for t, (tab, m, row) in enumerate(rows))]
        if not ok:
            continue
        assign = tuple(min(a[t] for a in ok) for t in range(n))
        if not sum(int(bt["sm_units"][j]) for j in assign) < int(bt["sm_budget"]):
            continue
        f = float(lut["freq_level"][k])
        lat = [float(tab[m, row, assign[t], k]) for t, (tab, m, row) in enumerate(rows)]
        if bt.get("static_power", 0) == 0:     # P0 in every task's Power x Latency
            e = sum(power(lut["p0_w"], float(bt["k_dyn_w"][b]), float(lut["sm_level"][assign[t]]), f,
                          float(bt["util"][b])) * lat[t] for t in range(n))
        else:                                  # P0 once, over the longest task
            e = sum(power(0.0, float(bt["k_dyn_w"][b]), float(lut["sm_level"][assign[t]]), f,
                          float(bt["util"][b])) * lat[t] for t in range(n)) + lut["p0_w"] * max(lat, default=0.0)
        if not np.float32(e) < np.inf:
            continue
        out.append((e, k, assign))
    return out


def brute_sweep(inp):
    bt = inp["batches"]
    B, T = bt["n_batches"], bt["max_tasks"]
    lev = np.full(B, -1, np.int32)
    energy = np.full(B, np.inf)
    tsm = np.full((B, T), -1, np.int32)
    for b in range(B):
        c = sweep_levels(inp, b)
        if c:
            e, k, a = min(c)
            lev[b], energy[b] = k, e
            tsm[b, :len(a)] = a
    return lev, (lev >= 0).astype(np.uint8), energy, tsm


# ------------------------------------------------------------------ preferred configuration, EWR
def phase_cells(inp, g, i, decode):
    """All (energy, cell, duration, power) of the SLO-feasible cells of one phase."""
    lut, q = inp["lut"], inp["llms"]
    NS, NF = lut["n_sm"], lut["n_freq"]
    m, B = int(q["model"][g, i]), int(q["batch"][g, i])
    prow = prompt_row(int(q["avg_in_tokens"][g, i]))
    out_tok = int(q["avg_out_tokens"][g, i])
    if not 0 <= m < lut["n_models"] or B < 0 or prow is None or prow < 0 or out_tok < 0:
        return []
    b = min(B + 1, 32)
    res = []
    for j, k in itertools.product(range(NS), range(NF)):
        lat = lut["dc"][m, b - 1, j, k] if decode else lut["pf"][m, prow, j, k]
        slo = q["slo_tbt_ms"][g, i] if decode else q["slo_ttft_ms"][g, i]
        if not lat < slo:
            continue
        p = power(lut["p0_w"], float(q["k_dyn_w"][g]), float(lut["sm_level"][j]), float(lut["freq_level"][k]),
                  b / 32)
        t = out_tok * float(lat) if decode else float(lat)
        if not np.float32(p * t) < np.inf:
            continue
        res.append((p * t, j * NF + k, t, p))
    return res


def brute_preferred(inp):
    q, lut = inp["llms"], inp["lut"]
    G, K, NF = q["n_gpus"], q["max_inst"], lut["n_freq"]
    out = {"sm_p": np.full((G, K), -1, np.int32), "f_p": np.full((G, K), -1, np.int32),
           "sm_d": np.full((G, K), -1, np.int32), "f_d": np.full((G, K), -1, np.int32),
           "sm_pref": np.full((G, K), np.nan), "f_pref": np.full((G, K), np.nan),
           "feasible": np.zeros((G, K), np.uint8)}
    for g in range(G):
        n = int(q["n_inst"][g])
        for i in range(K):
            if not 0 <= n <= K or i >= n:
                continue
            cp, cd = phase_cells(inp, g, i, False), phase_cells(inp, g, i, True)
            if cp:
                _, c, tp, pp = min(cp)
                out["sm_p"][g, i], out["f_p"][g, i] = divmod(c, NF)
            if cd:
                _, c, td, pd = min(cd)
                out["sm_d"][g, i], out["f_d"][g, i] = divmod(c, NF)
            if cp and cd:
                sp, sd = float(lut["sm_level"][out["sm_p"][g, i]]), float(lut["sm_level"][out["sm_d"][g, i]])
                fp, fd = float(lut["freq_level"][out["f_p"][g, i]]), float(lut["freq_level"][out["f_d"][g, i]])
                out["sm_pref"][g, i] = (sp * tp + sd * td) / (tp + td)          # time-weighted SM share
                out["f_pref"][g, i] = (pp * tp * fp + pd * td * fd) / (pp * tp + pd * td)   # energy-weighted
                out["feasible"][g, i] = 1
    return out


def brute_ewr(n_inst, f_pref, t_ms):
    """Per GPU: the highest preferred frequency, the waste sum t (F_g^3 - F_l^3); totals."""
    G, K = f_pref.shape
    fg, wg, opt = np.zeros(G), np.zeros(G), 0.0
    for g in range(G):
        ls = [(float(f_pref[g, i]), float(t_ms[g, i])) for i in range(K)
              if 0 <= n_inst[g] <= K and i < n_inst[g] and np.isfinite(f_pref[g, i]) and np.isfinite(t_ms[g, i])]
        fg[g] = max([f for f, _ in ls], default=0.0)
        wg[g] = sum(t * (fg[g] ** 3 - f ** 3) for f, t in ls)
        opt += sum(t * f ** 3 for f, t in ls)
    return fg, wg, (wg.sum(), opt, wg.sum() / opt if opt else np.nan)


# ------------------------------------------------------------------ current-frequency dispatch
def dispatch_energy(p0, k, s, f, u, ttft, lout, tbt):
    """Power x latency on one operating point, in the fixed float64 order of the oracle."""
    P = p0 + k * s * (f * f * f) * u
    return P * (ttft + lout * tbt)


def dispatch_points(inp, r):
    """Per hosting GPU with memory for request r: (g, T_avail, SM_free, free memory, b)."""
    lut, av, rq = inp["lut"], inp["avail"], inp["requests"]
    m = int(rq["model"][r])
    need = int(av["kv_kib_per_token"][m]) * (int(rq["prompt_tokens"][r]) + padded_out(int(rq["pred_out_tokens"][r])))
    out = []
    for g in range(av["n_gpus"]):
        if not (int(av["resident"][g, m // 32]) >> (m % 32)) & 1 or int(av["batch"][g]) < 0:
            continue
        steps = [s for s in range(av["n_steps"]) if int(av["mem_free_mib"][g, s]) * 1024 >= need]
        if steps:
            s = steps[0]
            out.append((g, float(av["t_avail_ms"][g, s]), int(av["sm_free"][g, s]), int(av["mem_free_mib"][g, s]),
                        min(int(av["batch"][g]) + 1, 32)))
    return out


def point_energy(inp, r, j, k, t_avail, b, kg):
    """Energy of request r on (j, k) starting at t_avail with batch b, or None if an SLO misses."""
    lut, rq = inp["lut"], inp["requests"]
    NS, NF = lut["n_sm"], lut["n_freq"]
    if not (0 <= j < NS and 0 <= k < NF):
        return None
    m = int(rq["model"][r])
    prow = prompt_row(int(rq["prompt_tokens"][r]))
    ttft = lut["pf"][m, b - 1 if prow < 0 else prow, j, k]
    tbt = lut["dc"][m, b - 1, j, k]
    if not (t_avail + float(ttft) < float(rq["slo_ttft_ms"][r]) and tbt < rq["slo_tbt_ms"][r]):
        return None
    e = dispatch_energy(float(lut["p0_w"]), kg, float(lut["sm_level"][j]), float(lut["freq_level"][k]), b / 32,
                        float(ttft), float(padded_out(int(rq["pred_out_tokens"][r]))), float(tbt))
    return e if np.float32(e) < np.inf else None


def brute_dispatch(inp):
    lut, av, rq = inp["lut"], inp["avail"], inp["requests"]
    R, NS, NF = rq["n_requests"], lut["n_sm"], lut["n_freq"]
    res = []
    for r in range(R):
        pts = dispatch_points(inp, r)
        cands = []
        for g, ta, sm, mem, b in pts:
            e = point_energy(inp, r, sm, int(av["freq_cur"][g]), ta, b, float(av["k_dyn_w"][g]))
            if e is not None:
                cands.append((e, g, sm, mem))
        if cands:
            emin = min(c[0] for c in cands)
            tied = [c for c in cands if c[0] <= emin + 0.02 * abs(emin)]    # within 2%
            e, g, sm, mem = min(tied, key=lambda c: (-c[3], -c[2], c[1]))   # memory, SMs, id
            res.append((g, int(av["freq_cur"][g]), sm, 1, e))
            continue
        fb = []
        for g, ta, sm, mem, b in pts:
            e = point_energy(inp, r, sm, NF - 1, ta, b, float(av["k_dyn_w"][g]))
            if e is not None:
                fb.append((ta, g, sm, e))
        if fb:
            ta, g, sm, e = min(fb)                                          # earliest, then id
            res.append((g, NF - 1, sm, 2, e))
            continue
        knew = float(np.float32(av["k_new_w"]))                          # a float32 field of the ABI
        new = [(point_energy(inp, r, NS - 1, k, 0.0, 1, knew), k) for k in range(NF)]
        new = [(e, k) for e, k in new if e is not None]
        if new:
            e, k = min(new)
            res.append((-1, k, NS - 1, 3, e))
        else:
            res.append((-1, -1, -1, 0, np.inf))
    a = np.array([x[:4] for x in res], np.int32).reshape(-1, 4)
    return a[:, 0], a[:, 1], a[:, 2], a[:, 3], np.array([x[4] for x in res])


# ------------------------------------------------------------------ transfer plan
def transfer_mib(inp):
    """Bytes(u -> v) in MiB from Python sets: u's models that v lacks plus u's state; 0 on the diagonal."""
    t = inp["transfer"]
    G, M = t["n_gpus"], inp["n_models"]
    sets = [{m for m in range(M) if (int(t["resident"][g, m // 32]) >> (m % 32)) & 1} for g in range(G)]
    out = np.zeros((G, G), np.int64)
    for u in range(G):
        for v in range(G):
            if u != v:
                out[u, v] = int(t["state_mib"][u]) + sum(int(t["weights_mib"][m]) for m in sets[u] - sets[v])
    return out


def link_ms_per_byte(inp, u, v):
    t = inp["transfer"]
    gbs = float(np.float32(t["bw_intra_gbs"] if t["node"][u] == t["node"][v] else t["bw_inter_gbs"]))
    return 1e3 / (gbs * 1e9)


def brute_moves(inp):
    """Per request: -1 invalid, 0 finish in place, 1 move with the KV cache, 2 move and recompute."""
    lut, t, pl, mv = inp["lut"], inp["transfer"], inp["plan"], inp["moves"]
    NS, NF, M, G = lut["n_sm"], lut["n_freq"], lut["n_models"], t["n_gpus"]
    res = []
    for q in range(mv["n_requests"]):
        u, m = int(mv["src"][q]), int(mv["model"][q])
        ok = 0 <= u < G and 0 <= m < M
        v = int(pl["dest"][u]) if ok else -1
        ok = ok and 0 <= v < G
        if ok:
            ju, ku, jv, kv = (int(pl["sm_cur"][u]), int(pl["freq_cur"][u]), int(pl["sm_cur"][v]), int(pl["freq_cur"][v]))
            row = prompt_row(int(mv["context_tokens"][q]))
            ok = (0 <= ju < NS and 0 <= ku < NF and 0 <= jv < NS and 0 <= kv < NF and int(pl["batch"][u]) >= 0
                  and row is not None and row >= 0 and min(int(mv["remaining_tokens"][q]), int(mv["kv_kib"][q]),
                                                           int(mv["token_kib"][q])) >= 0)
        if not ok:
            res.append((-1, 0.0, 0.0))
            continue
        b = min(int(pl["batch"][u]) + 1, 32)
        remaining = int(mv["remaining_tokens"][q]) * float(lut["dc"][m, b - 1, ju, ku])
        if v == u:
            res.append((0, remaining, 0.0))
            continue
        mpb = link_ms_per_byte(inp, u, v)
        kv_ms = (int(mv["kv_kib"][q]) * 1024) * mpb
        rec_ms = float(lut["pf"][m, row, jv, kv])
        mig = (int(mv["token_kib"][q]) * 1024) * mpb + min(kv_ms, rec_ms)
        res.append(((1 if kv_ms < rec_ms else 2) if remaining > mig else 0, remaining, mig))
    return (np.array([r[0] for r in res], np.int32), np.array([r[1] for r in res]), np.array([r[2] for r in res]))
