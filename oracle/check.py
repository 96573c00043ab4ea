"""Acceptance rule for a result under test against the oracle (test infrastructure only).

Placement, per request:
  * the feasibility flag must equal the oracle's exactly;
  * when feasible, the tested energy must be within ``rtol`` (1e-5) of the oracle's
    float64 energy *of the tested choice*, and that choice must be feasible under
    the oracle;
  * a choice other than the oracle's is accepted only as a near-tie: its oracle energy
    is at most the oracle optimum times (1 + rtol).
Migration, per source: the same on (saving, destination), with the tolerance taken
relative to max(|saving|, P0), and the frequency level must be the oracle's k* for
the tested pair exactly.
Sweep, per batch: the flag exactly; the tested level must be usable under the oracle,
its energy within ``rtol`` of the oracle's float64 energy at that level, a level other
than the oracle's only as a near-tie, and every task's SM level equal to the oracle's
smallest sufficient level at the tested frequency level.
Preferred configuration, per instance slot: the flag exactly; each phase's tested cell
feasible under the oracle, at most the oracle's least energy times (1 + rtol), with its
duration and power within ``rtol``; the two averages within ``rtol`` of the oracle's at
the tested cells.  EWR: per-GPU frequencies exactly, waste and totals within 1e-9.
Dispatch, per request: GPU, levels and phase exactly, and the float32 energy equal to the
oracle's float64 energy rounded to float32 (both sides evaluate the same float64
expression, so the 2% decision is taken on identical values).
Transfer plan: every cost equal to the oracle's float64 cost rounded to float32; every
decision equal, and both times equal to the oracle's rounded to float32 (same float64
evaluation order on both sides).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import candidate_energy, min_sm, pair_saving, phase_cell, preferred_at, sweep_level

RTOL = 1e-5


@dataclass
class Report:
    n: int = 0
    mismatches: list = field(default_factory=list)
    near_ties: int = 0
    max_rel_err: float = 0.0

    @property
    def ok(self):
        return not self.mismatches

    def __str__(self):
        head = self.mismatches[:5]
        return (f"{self.n} checked, {len(self.mismatches)} mismatches, {self.near_ties} near-ties, "
                f"max rel err {self.max_rel_err:.3g}" + (f"; first: {head}" if head else ""))


def check_placements(inp, sel, oracle_out, gpu_out, rtol=RTOL) -> Report:
    """``sel``: request ids; ``oracle_out``/``gpu_out``: (choice, feasible, energy) for those ids."""
    oc, of, oe = oracle_out
    gc, gf, ge = gpu_out
    rep = Report(n=len(sel))
    for i, r in enumerate(sel):
        r = int(r)
        if int(gf[i]) != int(of[i]):
            rep.mismatches.append((r, "feasible", int(gf[i]), int(of[i])))
            continue
        if not of[i]:
            if int(gc[i]) != -1 or not np.isinf(ge[i]):
                rep.mismatches.append((r, "infeasible output", int(gc[i]), float(ge[i])))
            continue
        ok, e_at_gpu = candidate_energy(inp, r, int(gc[i]))
        if not ok:
            rep.mismatches.append((r, "choice infeasible under the oracle", int(gc[i]), int(oc[i])))
            continue
        rel = abs(float(ge[i]) - e_at_gpu) / max(abs(e_at_gpu), 1e-30)
        rep.max_rel_err = max(rep.max_rel_err, rel)
        if rel > rtol:
            rep.mismatches.append((r, "energy", float(ge[i]), e_at_gpu))
            continue
        if int(gc[i]) != int(oc[i]):
            if e_at_gpu <= float(oe[i]) * (1 + rtol) + 1e-30:
                rep.near_ties += 1
            else:
                rep.mismatches.append((r, "choice", int(gc[i]), int(oc[i]), e_at_gpu, float(oe[i])))
    return rep


def check_migrations(inp, sel, oracle_out, gpu_out, rtol=RTOL) -> Report:
    ob, osv, ok_ = oracle_out
    gb, gsv, gk = gpu_out
    p0 = float(inp["lut"]["p0_w"])
    rep = Report(n=len(sel))
    for i, s in enumerate(sel):
        s = int(s)
        if (int(gb[i]) >= 0) != (int(ob[i]) >= 0):
            rep.mismatches.append((s, "feasible", int(gb[i]), int(ob[i])))
            continue
        if int(ob[i]) < 0:
            if int(gk[i]) != -1 or not (np.isinf(gsv[i]) and gsv[i] < 0):
                rep.mismatches.append((s, "infeasible output", int(gk[i]), float(gsv[i])))
            continue
        ok, kstar, sv = pair_saving(inp, s, int(gb[i]))
        if not ok:
            rep.mismatches.append((s, "pair infeasible under the oracle", int(gb[i]), int(ob[i])))
            continue
        if int(gk[i]) != kstar:
            rep.mismatches.append((s, "freq level", int(gk[i]), kstar))
            continue
        scale = max(abs(sv), abs(p0), 1e-30)
        rel = abs(float(gsv[i]) - sv) / scale
        rep.max_rel_err = max(rep.max_rel_err, rel)
        if rel > rtol:
            rep.mismatches.append((s, "saving", float(gsv[i]), sv))
            continue
        if int(gb[i]) != int(ob[i]):
            if sv >= float(osv[i]) - rtol * max(abs(float(osv[i])), abs(p0)):
                rep.near_ties += 1
            else:
                rep.mismatches.append((s, "destination", int(gb[i]), int(ob[i]), sv, float(osv[i])))
    return rep


def check_sweep(inp, sel, oracle_out, gpu_out, rtol=RTOL) -> Report:
    """``sel``: batch ids; outputs: (freq_level, feasible, energy, task_sm) for those ids."""
    ol, of, oe, ot = oracle_out
    gl, gf, ge, gt = gpu_out
    bt = inp["batches"]
    T = int(bt["max_tasks"])
    rep = Report(n=len(sel))
    for i, b in enumerate(sel):
        b = int(b)
        if int(gf[i]) != int(of[i]):
            rep.mismatches.append((b, "feasible", int(gf[i]), int(of[i])))
            continue
        if not of[i]:
            if int(gl[i]) != -1 or not np.isinf(ge[i]) or np.any(gt[i] != -1):
                rep.mismatches.append((b, "infeasible output", int(gl[i]), float(ge[i])))
            continue
        k = int(gl[i])
        if k == int(ol[i]):                  # the oracle's own level: its outputs apply
            ok, e_at, exp_t = True, float(oe[i]), [int(x) for x in ot[i]]
        else:
            ok, e_at = sweep_level(inp, b, k)
            n = int(bt["n_tasks"][b])
            exp_t = [min_sm(inp, b, t, k) if t < n else -1 for t in range(T)] if ok else None
        if not ok:
            rep.mismatches.append((b, "level unusable under the oracle", k, int(ol[i])))
            continue
        rel = abs(float(ge[i]) - e_at) / max(abs(e_at), 1e-30)
        rep.max_rel_err = max(rep.max_rel_err, rel)
        if rel > rtol:
            rep.mismatches.append((b, "energy", float(ge[i]), e_at))
            continue
        if list(gt[i]) != exp_t:
            rep.mismatches.append((b, "task SM levels", list(gt[i]), exp_t))
            continue
        if k != int(ol[i]):
            if e_at <= float(oe[i]) * (1 + rtol) + 1e-30:
                rep.near_ties += 1
            else:
                rep.mismatches.append((b, "level", k, int(ol[i]), e_at, float(oe[i])))
    return rep


def _rel(a, b):
    return abs(float(a) - float(b)) / max(abs(float(b)), 1e-30)


def check_preferred(inp, oracle_out, gpu_out, rtol=RTOL) -> Report:
    """``oracle_out``: oracle.preferred(inp); ``gpu_out``: the same keys from the device
    (t_p_ms/t_d_ms/p_p_w/p_d_w/t_ms names for durations and powers)."""
    q = inp["llms"]
    G, K = int(q["n_gpus"]), int(q["max_inst"])
    o, d = oracle_out, gpu_out
    rep = Report(n=G * K)
    for g in range(G):
        for i in range(K):
            if int(d["feasible"][g, i]) != int(o["feasible"][g, i]):
                rep.mismatches.append(((g, i), "feasible", int(d["feasible"][g, i]), int(o["feasible"][g, i])))
                continue
            bad = False
            same = True
            for decode, js, ks, tk, pk, ot, op in ((False, "sm_p", "f_p", "t_p_ms", "p_p_w", "t_p", "p_p"),
                                                    (True, "sm_d", "f_d", "t_d_ms", "p_d_w", "t_d", "p_d")):
                gj, gk, oj = int(d[js][g, i]), int(d[ks][g, i]), int(o[js][g, i])
                if (gj < 0) != (oj < 0):
                    rep.mismatches.append(((g, i), f"{js} presence", gj, oj))
                    bad = True
                    break
                if gj < 0:
                    continue
                ok, t, p = phase_cell(inp, g, i, decode, gj, gk)
                if not ok:
                    rep.mismatches.append(((g, i), f"{js} cell infeasible under the oracle", (gj, gk)))
                    bad = True
                    break
                for got, want, what in ((d[tk][g, i], t, tk), (d[pk][g, i], p, pk)):
                    r = _rel(got, want)
                    rep.max_rel_err = max(rep.max_rel_err, r)
                    if r > rtol:
                        rep.mismatches.append(((g, i), what, float(got), want))
                        bad = True
                if (gj, gk) != (oj, int(o[ks][g, i])):
                    same = False
                    if p * t <= float(o[op][g, i] * o[ot][g, i]) * (1 + rtol) + 1e-30:
                        rep.near_ties += 1
                    else:
                        rep.mismatches.append(((g, i), f"{js} cell", (gj, gk), (oj, int(o[ks][g, i]))))
                        bad = True
            if bad or not o["feasible"][g, i]:
                if not bad and not (np.isnan(d["sm_pref"][g, i]) and np.isnan(d["f_pref"][g, i])):
                    rep.mismatches.append(((g, i), "averages of an infeasible slot", float(d["sm_pref"][g, i])))
                continue
            if same:
                want_sm, want_f, want_t = o["sm_pref"][g, i], o["f_pref"][g, i], o["t_p"][g, i] + o["t_d"][g, i]
            else:
                _, want_sm, want_f = preferred_at(inp, g, i, d["sm_p"][g, i], d["f_p"][g, i], d["sm_d"][g, i],
                                                  d["f_d"][g, i])
                want_t = phase_cell(inp, g, i, False, d["sm_p"][g, i], d["f_p"][g, i])[1] + \
                    phase_cell(inp, g, i, True, d["sm_d"][g, i], d["f_d"][g, i])[1]
            for got, want, what in ((d["sm_pref"][g, i], want_sm, "sm_pref"), (d["f_pref"][g, i], want_f, "f_pref"),
                                    (d["t_ms"][g, i], want_t, "t_ms")):
                r = _rel(got, want)
                rep.max_rel_err = max(rep.max_rel_err, r)
                if r > rtol:
                    rep.mismatches.append(((g, i), what, float(got), float(want)))
    return rep


def check_ewr(oracle_out, gpu_out, rtol=1e-9) -> Report:
    """``oracle_out``: oracle.fleet_ewr(...) on the same inputs; ``gpu_out``:
    (f_gpu, waste_gpu, totals[3]) from the device."""
    of, ow, ot = oracle_out
    gf, gw, gt = gpu_out
    rep = Report(n=len(of))
    if not np.array_equal(np.asarray(gf, np.float64), np.asarray(of, np.float64)):
        bad = np.flatnonzero(np.asarray(gf, np.float64) != np.asarray(of, np.float64))[:5]
        rep.mismatches.append(("f_gpu", [(int(b), float(gf[b]), float(of[b])) for b in bad]))
    scale = max(abs(ot[0]), abs(ot[1]) * 1e-6, 1e-30)
    dw = np.abs(np.asarray(gw) - np.asarray(ow))
    if np.any(dw > rtol * scale):
        rep.mismatches.append(("waste_gpu", float(dw.max())))
    for k, name in enumerate(("e_waste", "e_optimal", "ewr")):
        r = _rel(gt[k], ot[k]) if ot[k] != 0 else abs(float(gt[k]))
        rep.max_rel_err = max(rep.max_rel_err, r)
        if not (r <= rtol or (np.isnan(gt[k]) and np.isnan(ot[k]))):
            rep.mismatches.append((name, float(gt[k]), float(ot[k])))
    return rep


def check_dispatch(oracle_out, gpu_out) -> Report:
    og, ok, oj, oph, oe = oracle_out
    gg, gk, gj, gph, ge = gpu_out
    rep = Report(n=len(og))
    for i in range(len(og)):
        a = (int(gg[i]), int(gk[i]), int(gj[i]), int(gph[i]))
        b = (int(og[i]), int(ok[i]), int(oj[i]), int(oph[i]))
        if a != b:
            rep.mismatches.append((i, "choice", a, b))
            continue
        if not (np.float32(oe[i]) == ge[i]):
            rep.mismatches.append((i, "energy", float(ge[i]), float(oe[i])))
    return rep


def check_transfer(oracle_costs, oracle_moves, gpu_costs, gpu_moves) -> Report:
    rep = Report(n=oracle_costs.size + len(oracle_moves[0]))
    want = oracle_costs.astype(np.float32)
    bad = np.argwhere(want != gpu_costs)
    if len(bad):
        u, v = bad[0]
        rep.mismatches.append(("cost", len(bad), (int(u), int(v)), float(gpu_costs[u, v]), float(oracle_costs[u, v])))
    od, orem, omig = oracle_moves
    gd, grem, gmig = gpu_moves
    for name, a, b in (("decision", gd, od), ("remaining_ms", grem, orem.astype(np.float32)),
                       ("migrate_ms", gmig, omig.astype(np.float32))):
        bad = np.flatnonzero(a != b)
        if len(bad):
            rep.mismatches.append((name, len(bad), int(bad[0]), float(a[bad[0]]), float(b[bad[0]])))
    return rep
