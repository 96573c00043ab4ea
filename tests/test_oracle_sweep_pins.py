"""Pins of the local SM/frequency sweep oracle against things other than itself.

* a hand-worked golden example and its variants (exact arithmetic, tests/golden/),
* exhaustive enumeration of SM assignments on tiny random batches (tests/brute.py),
* a closed form: on analytic tables latency = a + c / (s f) the smallest SM level that
  meets a slack is floor(NS c / (f (slack - a))),
* metamorphic relations: energy adds over tasks, task order does not matter, zero power
  leaves the lowest usable level, the SM budget test is strict,
* invalid and empty batches, and invariants on the synthetic sweep workload.
"""
import numpy as np
import pytest

import oracle
from brute import brute_sweep
from conftest import golden_sweep
from paper_2606_30391_amd import workloads as W


# ------------------------------------------------------------------ golden values
def _expect(got, exp):
    lev, fe, en, tsm = got
    assert lev[0] == exp["freq_level"]
    assert fe[0] == exp["feasible"]
    if exp["energy_mj"] is None:
        assert en[0] == np.inf
    else:
        assert en[0] == exp["energy_mj"]
    assert list(tsm[0]) == exp["task_sm"]


def test_sweep_worked_example():
    inp, exp, d = golden_sweep()
    _expect(oracle.sweep(inp), exp)
    for k, e in exp["levels"].items():
        ok, v = oracle.sweep_level(inp, 0, int(k))
        assert ok == (e is not None)
        if ok:
            assert v == e
    assert oracle.min_sm(inp, 0, 0, 0) == 1 and oracle.min_sm(inp, 0, 1, 0) == 1
    assert oracle.min_sm(inp, 0, 0, 1) == 0 and oracle.min_sm(inp, 0, 1, 2) == 0


@pytest.mark.parametrize("variant", ["static power dominates", "budget reached exactly",
                                     "budget one unit above", "slack equal to a latency",
                                     "static power per batch", "static power per task, P0 = 640",
                                     "static power per batch, P0 = 640"])
def test_sweep_worked_example_variants(variant):
    inp, exp, d = golden_sweep(variant)
    _expect(oracle.sweep(inp), exp)
    _expect(brute_sweep(inp), exp)


# ------------------------------------------------------------------ brute force
@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("static_power", [0, 1])
def test_sweep_matches_enumeration(seed, static_power):
    rng = np.random.default_rng(7000 + seed)
    for case in range(40):
        inp = W.make_tiny_sweep(rng, nan_cells=(case % 3 == 0), zero_power=(case % 7 == 0))
        inp["batches"]["static_power"] = static_power
        lev, fe, en, tsm = oracle.sweep(inp)
        blev, bfe, ben, btsm = brute_sweep(inp)
        assert np.array_equal(fe, bfe), (seed, case)
        assert np.array_equal(lev, blev), (seed, case)
        assert np.array_equal(tsm, btsm), (seed, case)
        ok = fe == 1
        assert np.all(en[~ok] == np.inf)
        np.testing.assert_allclose(en[ok], ben[ok], rtol=1e-12, atol=0)


# ------------------------------------------------------------------ closed form
def test_sweep_min_sm_closed_form():
    """Analytic decode table a + c*b/(s f): the smallest s_j = (j+1)/NS above
    c*b/(f (slack - a)) is j = floor(NS c b / (f (slack - a)))."""
    rng = np.random.default_rng(71)
    NS, NF, M = 8, 16, 3
    s, f = W.sm_levels(NS), W.freq_levels(NF)
    a = rng.uniform(5, 20, M)
    c = rng.uniform(0.5, 3, M)
    rows = np.arange(1, 33, dtype=np.float64)
    sf = s.astype(np.float64)[:, None] * f.astype(np.float64)[None, :]
    dc = (a[:, None, None, None] + c[:, None, None, None] * rows[None, :, None, None] / sf[None, None]).astype(np.float32)
    lut = {"n_models": M, "n_rows": 32, "n_sm": NS, "n_freq": NF, "sm_level": s, "freq_level": f,
           "pf": dc.copy(), "dc": dc, "p0_w": 120.0}
    B, T = 300, 1
    bat = {"n_batches": B, "max_tasks": T, "n_tasks": np.ones(B, np.int32),
           "task_model": rng.integers(0, M, (B, T)).astype(np.int32), "task_phase": np.ones((B, T), np.int32),
           "task_tokens": rng.integers(1, 33, (B, T)).astype(np.int32),
           "task_slack_ms": rng.uniform(10, 120, (B, T)).astype(np.float32),
           "k_dyn_w": np.full(B, 400, np.float32), "util": np.full(B, 0.5, np.float32),
           "sm_units": W.sm_permille(s), "sm_budget": 100000}
    inp = {"lut": lut, "batches": bat}
    checked = 0
    for b in range(B):
        m, bb, sl = int(bat["task_model"][b, 0]), int(bat["task_tokens"][b, 0]), float(bat["task_slack_ms"][b, 0])
        for k in range(NF):
            if sl <= a[m]:
                exp = -1
            else:
                x = NS * c[m] * bb / (float(f[k]) * (sl - a[m]))
                if abs(x - round(x)) < 1e-3:
                    continue                      # too close to a level for float32 tables
                exp = int(np.floor(x)) if np.floor(x) < NS else -1
            assert oracle.min_sm(inp, b, 0, k) == exp, (b, k)
            checked += 1
    assert checked > 4000


# ------------------------------------------------------------------ metamorphic relations
def _one_batch(lut, tasks, kdyn, util, units, budget):
    T = len(tasks)
    return {"lut": lut, "batches": {
        "n_batches": 1, "max_tasks": max(T, 1), "n_tasks": np.array([T], np.int32),
        "task_model": np.array([[t[0] for t in tasks] or [0]], np.int32),
        "task_phase": np.array([[t[1] for t in tasks] or [0]], np.int32),
        "task_tokens": np.array([[t[2] for t in tasks] or [1]], np.int32),
        "task_slack_ms": np.array([[t[3] for t in tasks] or [0]], np.float32),
        "k_dyn_w": np.array([kdyn], np.float32), "util": np.array([util], np.float32),
        "sm_units": units, "sm_budget": budget}}


def _random_tasks(rng, n, M):
    return [(int(rng.integers(0, M)), int(rng.integers(0, 2)), int(rng.integers(1, 5000)),
             float(rng.uniform(20, 80))) for _ in range(n)]


def test_sweep_energy_adds_over_tasks():
    rng = np.random.default_rng(72)
    inp0 = W.make_tiny_sweep(rng, B=1, T=1, M=3, NS=4, NF=5)
    lut, units = inp0["lut"], inp0["batches"]["sm_units"]
    n_checked = 0
    for _ in range(200):
        A, Bt = _random_tasks(rng, 2, 3), _random_tasks(rng, 2, 3)
        kd, u = float(rng.uniform(0, 500)), float(rng.uniform(0, 1))
        whole = _one_batch(lut, A + Bt, kd, u, units, 10 ** 9)
        pa, pb = _one_batch(lut, A, kd, u, units, 10 ** 9), _one_batch(lut, Bt, kd, u, units, 10 ** 9)
        for k in range(lut["n_freq"]):
            ok, e = oracle.sweep_level(whole, 0, k)
            oka, ea = oracle.sweep_level(pa, 0, k)
            okb, eb = oracle.sweep_level(pb, 0, k)
            assert ok == (oka and okb)
            if ok:
                assert e == pytest.approx(ea + eb, rel=1e-13)
                n_checked += 1
    assert n_checked > 50


def test_sweep_task_order_does_not_matter():
    rng = np.random.default_rng(73)
    for _ in range(100):
        inp = W.make_tiny_sweep(rng, B=1, T=5, M=3, NS=4, NF=6)
        bt = inp["batches"]
        bt["n_tasks"][:] = 5
        lev, fe, en, tsm = oracle.sweep(inp)
        perm = rng.permutation(5)
        for key in ("task_model", "task_phase", "task_tokens", "task_slack_ms"):
            bt[key] = np.ascontiguousarray(bt[key][:, perm])
        lev2, fe2, en2, tsm2 = oracle.sweep(inp)
        assert lev2[0] == lev[0] and fe2[0] == fe[0]
        assert en2[0] == pytest.approx(en[0], rel=1e-13) or en[0] == en2[0] == np.inf
        if fe[0]:
            assert list(tsm2[0]) == list(tsm[0][perm])


def test_sweep_zero_power_takes_lowest_usable_level():
    """With P0 = 0 and k_dyn = 0 every usable level costs 0 mJ: exact ties, lowest k."""
    rng = np.random.default_rng(74)
    seen = 0
    for _ in range(200):
        inp = W.make_tiny_sweep(rng, B=1, T=3, M=2, NS=3, NF=6, zero_power=True)
        lev, fe, en, tsm = oracle.sweep(inp)
        usable = [k for k in range(6) if oracle.sweep_level(inp, 0, k)[0]]
        if usable:
            assert lev[0] == usable[0] and en[0] == 0.0
            seen += len(usable) > 1
        else:
            assert fe[0] == 0
    assert seen > 10


def test_sweep_budget_is_strict():
    rng = np.random.default_rng(75)
    hit = 0
    for _ in range(200):
        inp = W.make_tiny_sweep(rng, B=1, T=3, M=2, NS=4, NF=4)
        bt = inp["batches"]
        bt["sm_budget"] = 10 ** 9
        lev, fe, en, tsm = oracle.sweep(inp)
        if not fe[0] or bt["n_tasks"][0] == 0:
            continue
        used = int(sum(int(bt["sm_units"][j]) for j in tsm[0][:bt["n_tasks"][0]]))
        bt["sm_budget"] = used
        assert not oracle.sweep_level(inp, 0, int(lev[0]))[0]
        bt["sm_budget"] = used + 1
        assert oracle.sweep_level(inp, 0, int(lev[0]))[0]
        hit += 1
    assert hit > 50


# ------------------------------------------------------------------ invalid and empty
def test_sweep_invalid_tasks_and_empty_batches():
    rng = np.random.default_rng(76)
    inp = W.make_tiny_sweep(rng, B=6, T=3, M=2, NS=4, NF=4)
    bt = inp["batches"]
    bt["sm_budget"] = 10 ** 9
    bt["task_slack_ms"][:] = 1e9                     # every task meets its slack anywhere
    bt["n_tasks"][:] = [0, 3, 3, 3, 3, 4]
    bt["task_model"][1, 2] = 2                       # model out of range
    bt["task_phase"][2, 0] = 2                       # neither prefill nor decode
    bt["task_tokens"][3, 1] = 0                      # no tokens
    bt["task_tokens"][4, 0] = -5
    lev, fe, en, tsm = oracle.sweep(inp)
    assert lev[0] == 0 and fe[0] == 1 and en[0] == 0.0 and list(tsm[0]) == [-1, -1, -1]
    for b in range(1, 6):
        assert lev[b] == -1 and fe[b] == 0 and en[b] == np.inf and list(tsm[b]) == [-1, -1, -1]
    # NaN latencies are never below a slack
    inp = W.make_tiny_sweep(rng, B=1, T=1, M=1, NS=2, NF=2)
    inp["lut"]["pf"][:] = np.nan
    inp["lut"]["dc"][:] = np.nan
    inp["batches"]["n_tasks"][:] = 1
    assert oracle.sweep(inp)[1][0] == 0


# ------------------------------------------------------------------ workload invariants
def test_sweep_workload_invariants():
    inp = W.make_sweep(n_gpus=64, n_epochs=4)
    bt, lut = inp["batches"], inp["lut"]
    lev, fe, en, tsm = oracle.sweep(inp)
    assert 0.2 < fe.mean() < 0.9
    for b in range(bt["n_batches"]):
        usable = {k: oracle.sweep_level(inp, b, k) for k in range(lut["n_freq"])}
        usable = {k: e for k, (ok, e) in usable.items() if ok}
        if not fe[b]:
            assert not usable
            continue
        assert usable[int(lev[b])] == en[b]
        assert all(e >= en[b] for e in usable.values())
        assert all(e > en[b] for k, e in usable.items() if k < lev[b])
        n = int(bt["n_tasks"][b])
        assert int(sum(bt["sm_units"][tsm[b, :n]])) < bt["sm_budget"]
        assert np.all(tsm[b, n:] == -1)
