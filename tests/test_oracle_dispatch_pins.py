"""Pins of the current-frequency dispatch oracle (Sec. 3.3, Phases One to Three).

* a hand-worked example and five variants (2% margin in and out, equal memory, the F_max
  fallback by earliest availability, a new GPU, nothing feasible),
* enumeration on tiny random instances (tests/brute.py: list every operating point, the
  2% tie set, the stability order as a sort key, the fallback as the minimum of a list),
* the stability tie-break against numpy.lexsort on exact ties, scaling of power,
* invariants on the dispatch workload.
"""
import numpy as np
import pytest

import oracle
from brute import brute_dispatch, dispatch_points, point_energy
from conftest import golden_dispatch, load_golden
from paper_2606_30391_amd import workloads as W

VARIANTS = [v["name"] for v in load_golden("dispatch_worked_example.json")["variants"]]


def _expect(got, exp):
    g, k, j, ph, e = got
    assert (int(g[0]), int(k[0]), int(j[0]), int(ph[0])) == (exp["gpu"], exp["freq_level"], exp["sm_level"],
                                                              exp["phase"])
    assert (e[0] == np.inf) if exp["energy_mj"] is None else (e[0] == exp["energy_mj"])


@pytest.mark.parametrize("variant", [None] + VARIANTS)
def test_dispatch_worked_example(variant):
    inp, exp, d = golden_dispatch(variant)
    _expect(oracle.dispatch(inp), exp)
    _expect(brute_dispatch(inp), exp)


@pytest.mark.parametrize("seed", range(6))
def test_dispatch_matches_enumeration(seed):
    rng = np.random.default_rng(9000 + seed)
    for case in range(40):
        inp = W.make_tiny_dispatch(rng, ties=(case % 4 == 0))
        o, b = oracle.dispatch(inp), brute_dispatch(inp)
        for x, y, name in zip(o[:4], b[:4], ("gpu", "freq", "sm", "phase")):
            assert np.array_equal(x, y), (seed, case, name)
        assert np.array_equal(o[4], b[4]), (seed, case)


def test_stability_tie_break_is_a_lexicographic_order():
    """Exactly equal energies everywhere (one table value, no dynamic power): the choice is
    the lexsort maximum of (free memory, free SMs, -id) over the feasible GPUs."""
    rng = np.random.default_rng(91)
    checked = 0
    for it in range(100):
        inp = W.make_tiny_dispatch(rng, R=4, G=8, M=1, NS=3, NF=3, S=2, ties=True)
        inp["avail"]["k_dyn_w"][:] = 0.0
        if it % 2:                        # equal free memory everywhere: the free SMs decide
            inp["avail"]["mem_free_mib"][:] = inp["avail"]["mem_free_mib"][:1]
        g, k, j, ph, e = oracle.dispatch(inp)
        for r in range(4):
            pts = [(gg, ta, sm, mem, b) for gg, ta, sm, mem, b in dispatch_points(inp, r)
                   if point_energy(inp, r, sm, int(inp["avail"]["freq_cur"][gg]), ta, b, 0.0) is not None]
            if not pts:
                assert ph[r] != 1
                continue
            ids = np.array([p[0] for p in pts])
            order = np.lexsort((ids, -np.array([p[2] for p in pts]), -np.array([p[3] for p in pts])))
            assert ph[r] == 1 and g[r] == ids[order[0]]
            checked += 1
    assert checked > 100


def test_dispatch_power_scaling():
    rng = np.random.default_rng(92)
    inp = W.make_tiny_dispatch(rng, R=200, G=10, M=2, NS=4, NF=5, S=3)
    a = oracle.dispatch(inp)
    inp["lut"]["p0_w"] *= 2.0
    inp["avail"]["k_dyn_w"] = (inp["avail"]["k_dyn_w"] * 2).astype(np.float32)
    inp["avail"]["k_new_w"] *= 2.0
    b = oracle.dispatch(inp)
    for x, y in zip(a[:4], b[:4]):
        assert np.array_equal(x, y)
    assert np.array_equal(a[4] * 2, b[4])


def test_dispatch_workload_invariants():
    inp = W.make_dispatch(n_requests=600, n_gpus=96)
    g, k, j, ph, e = oracle.dispatch(inp)
    counts = np.bincount(ph, minlength=4)
    assert counts[1] > 300 and counts.min() >= 0
    b = brute_dispatch(inp)
    for x, y in zip((g, k, j, ph), b[:4]):
        assert np.array_equal(x, y)
    assert np.array_equal(e, b[4])


def test_dispatch_negative_energies():
    """Negative power terms: the 2% band is taken on |E_min|, so the least-energy GPU is
    always inside it and the stability order still decides among its neighbours."""
    rng = np.random.default_rng(93)
    for _ in range(30):
        inp = W.make_tiny_dispatch(rng, R=30, G=8, M=2, NS=3, NF=4, S=2)
        inp["lut"]["p0_w"] = float(np.float32(rng.uniform(0.0, 5.0)))
        inp["avail"]["k_dyn_w"] = (-rng.uniform(0.0, 500.0, 8)).astype(np.float32)
        o, b = oracle.dispatch(inp), brute_dispatch(inp)
        for x, y in zip(o, b):
            assert np.array_equal(x, y)
        assert np.any(o[4][o[3] == 1] < 0)
