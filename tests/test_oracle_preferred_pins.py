"""Pins of the preferred-configuration and energy-waste-ratio oracle.

* a hand-worked golden example of both (exact arithmetic, tests/golden/),
* exhaustive enumeration of each phase's cells on tiny random instances (tests/brute.py),
* special cases: zero output length leaves the prefill configuration, zero dynamic power
  reduces each phase to the lowest-latency feasible cell (numpy.argmin), a GPU with one
  LLM or with equal preferred frequencies wastes nothing,
* metamorphic relations and invariants: the averages are convex combinations of the two
  phases' values, F_g is the maximum over the GPU's LLMs, scaling execution times scales
  the energies and leaves the ratio, slot order within a GPU does not matter,
* invalid instances, and invariants on the fleet workload.
"""
from fractions import Fraction

import numpy as np
import pytest

import oracle
from brute import brute_ewr, brute_preferred
from conftest import golden_preferred, load_golden
from paper_2606_30391_amd import workloads as W


# ------------------------------------------------------------------ golden values
def test_preferred_worked_example():
    inp, exp, d = golden_preferred()
    o = oracle.preferred(inp)
    for f in ("sm_p", "f_p", "sm_d", "f_d", "feasible"):
        assert o[f][0, 0] == exp[f], f
    for f in ("t_p", "t_d", "p_p", "p_d"):
        assert o[f][0, 0] == exp[f], f
    for f in ("sm_pref", "f_pref"):
        num, den = exp[f]
        assert o[f][0, 0] == pytest.approx(float(Fraction(num) / Fraction(den)), rel=1e-15), f


@pytest.mark.parametrize("variant", ["TTFT SLO equal to the fastest prefill", "TBT SLO equal to the best decode latency"])
def test_preferred_worked_example_variants(variant):
    inp, exp, d = golden_preferred(variant)
    for o in (oracle.preferred(inp), brute_preferred(inp)):
        for f in ("sm_p", "f_p", "sm_d", "f_d", "feasible"):
            assert o[f][0, 0] == exp[f], (variant, f)
        for f in ("sm_pref", "f_pref"):
            if f in exp:
                num, den = exp[f]
                assert o[f][0, 0] == pytest.approx(num / den, rel=1e-15), (variant, f)
    o = oracle.preferred(inp)
    for f in ("t_d", "p_d"):
        if f in exp:
            assert o[f][0, 0] == exp[f]


def test_ewr_worked_example():
    d = load_golden("preferred_worked_example.json")["ewr"]
    fg, wg, (waste, opt, ewr) = oracle.fleet_ewr(np.array(d["n_inst"]), np.array(d["f_pref"]), np.array(d["t_ms"]))
    e = d["expected"]
    assert list(fg) == e["f_gpu"] and list(wg) == e["waste_gpu"]
    assert waste == e["e_waste"] and opt == e["e_optimal"]
    assert ewr == pytest.approx(e["ewr"][0] / e["ewr"][1], rel=1e-15)


# ------------------------------------------------------------------ brute force
@pytest.mark.parametrize("seed", range(5))
def test_preferred_matches_enumeration(seed):
    rng = np.random.default_rng(8000 + seed)
    for case in range(40):
        inp = W.make_tiny_llms(rng, nan_cells=(case % 3 == 0), zero_out=(case % 9 == 0))
        o, b = oracle.preferred(inp), brute_preferred(inp)
        for f in ("sm_p", "f_p", "sm_d", "f_d", "feasible"):
            assert np.array_equal(o[f], b[f]), (seed, case, f)
        ok = o["feasible"] == 1
        for f in ("sm_pref", "f_pref"):
            np.testing.assert_allclose(o[f][ok], b[f][ok], rtol=1e-12)
            assert np.all(np.isnan(o[f][~ok]))


@pytest.mark.parametrize("seed", range(3))
def test_ewr_matches_enumeration(seed):
    rng = np.random.default_rng(8100 + seed)
    for _ in range(50):
        G, K = int(rng.integers(1, 7)), int(rng.integers(1, 5))
        n = rng.integers(0, K + 1, G)
        f = rng.uniform(0.5, 1.0, (G, K)).astype(np.float32)
        t = rng.uniform(1.0, 500.0, (G, K)).astype(np.float32)
        f[rng.random((G, K)) < 0.1] = np.nan
        fg, wg, tot = oracle.fleet_ewr(n, f, t)
        bg, bw, btot = brute_ewr(n, f, t)
        np.testing.assert_allclose(fg, bg, rtol=0, atol=0)
        np.testing.assert_allclose(wg, bw, rtol=1e-12, atol=1e-9)
        np.testing.assert_allclose(tot, btot, rtol=1e-12, atol=1e-9)


# ------------------------------------------------------------------ special cases
def test_zero_output_keeps_the_prefill_configuration():
    rng = np.random.default_rng(81)
    inp = W.make_tiny_llms(rng, G=30, K=3, M=3, NS=4, NF=6, zero_out=True)
    o = oracle.preferred(inp)
    lut = inp["lut"]
    ok = o["feasible"] == 1
    assert ok.sum() > 10
    assert np.all(o["t_d"][ok] == 0.0)
    np.testing.assert_allclose(o["sm_pref"][ok], lut["sm_level"][o["sm_p"][ok]], rtol=1e-15)
    np.testing.assert_allclose(o["f_pref"][ok], lut["freq_level"][o["f_p"][ok]], rtol=1e-15)


def test_zero_dynamic_power_picks_the_fastest_cell():
    """k = 0: every cell costs P0 x duration, so each phase takes its lowest-latency
    feasible cell (first on ties), a textbook argmin."""
    rng = np.random.default_rng(82)
    inp = W.make_tiny_llms(rng, G=25, K=3, M=2, NS=4, NF=5)
    q, lut = inp["llms"], inp["lut"]
    q["k_dyn_w"][:] = 0.0
    q["avg_out_tokens"][:] = np.maximum(q["avg_out_tokens"], 1)
    o = oracle.preferred(inp)
    NF, checked = lut["n_freq"], 0
    for g in range(q["n_gpus"]):
        for i in range(int(q["n_inst"][g])):
            m, b = q["model"][g, i], min(q["batch"][g, i] + 1, 32)
            prow = min(-(-int(q["avg_in_tokens"][g, i]) // 256), 32) - 1
            for decode, tab, row, slo, key in ((False, lut["pf"], prow, q["slo_ttft_ms"][g, i], ("sm_p", "f_p")),
                                              (True, lut["dc"], b - 1, q["slo_tbt_ms"][g, i], ("sm_d", "f_d"))):
                lat = tab[m, row].reshape(-1).astype(np.float64)
                lat[~(lat < slo)] = np.inf
                if np.isinf(lat).all():
                    assert o[key[0]][g, i] == -1
                    continue
                c = int(np.argmin(lat))
                assert (o[key[0]][g, i], o[key[1]][g, i]) == divmod(c, NF)
                checked += 1
    assert checked > 40


def test_ewr_special_cases():
    rng = np.random.default_rng(83)
    G, K = 40, 4
    f = rng.uniform(0.5, 1.0, (G, K)).astype(np.float32)
    t = rng.uniform(1.0, 100.0, (G, K)).astype(np.float32)
    # one LLM per GPU: every GPU runs at its LLM's own frequency
    fg, wg, (waste, opt, ewr) = oracle.fleet_ewr(np.ones(G, np.int32), f, t)
    assert np.all(fg == f[:, 0].astype(np.float64)) and waste == 0.0 and ewr == 0.0
    # equal preferred frequencies on each GPU
    feq = np.repeat(f[:, :1], K, axis=1)
    fg, wg, (waste, opt, ewr) = oracle.fleet_ewr(np.full(G, K, np.int32), feq, t)
    assert waste == 0.0
    np.testing.assert_allclose(opt, float((t.astype(np.float64) * feq.astype(np.float64) ** 3).sum()), rtol=1e-12)
    # F_g is the maximum, waste is non-negative; time scaling keeps the ratio
    n = rng.integers(1, K + 1, G).astype(np.int32)
    fg, wg, (waste, opt, ewr) = oracle.fleet_ewr(n, f, t)
    live = np.arange(K)[None, :] < n[:, None]
    assert np.all(fg == np.where(live, f, -np.inf).max(axis=1))
    assert np.all(wg >= 0) and ewr > 0
    fg2, wg2, (w2, o2, e2) = oracle.fleet_ewr(n, f, (t * 4).astype(np.float32))
    assert w2 == pytest.approx(4 * waste, rel=1e-12) and e2 == pytest.approx(ewr, rel=1e-12)
    # slot order inside a GPU does not matter
    perm = rng.permutation(K)
    f3, t3 = f.copy(), t.copy()
    full = np.full(G, K, np.int32)
    a = oracle.fleet_ewr(full, f3, t3)
    b = oracle.fleet_ewr(full, f3[:, perm], t3[:, perm])
    assert np.array_equal(a[0], b[0])
    np.testing.assert_allclose(a[1], b[1], rtol=1e-12)


def test_preferred_invalid_and_unused_slots():
    rng = np.random.default_rng(84)
    inp = W.make_tiny_llms(rng, G=6, K=2, M=2, NS=3, NF=4)
    q = inp["llms"]
    q["slo_ttft_ms"][:] = 1e9
    q["slo_tbt_ms"][:] = 1e9
    q["n_inst"][:] = [2, 2, 2, 2, 1, 3]
    q["model"][0, 0] = 2
    q["batch"][1, 1] = -1
    q["avg_in_tokens"][2, 0] = 0
    q["avg_out_tokens"][3, 1] = -4
    o = oracle.preferred(inp)
    assert o["feasible"][0, 0] == 0 and o["feasible"][0, 1] == 1
    assert o["feasible"][1, 1] == 0 and o["feasible"][2, 0] == 0 and o["feasible"][3, 1] == 0
    assert o["feasible"][4, 0] == 1 and o["feasible"][4, 1] == 0      # past n_inst
    assert not o["feasible"][5].any()                                  # n_inst > max_inst
    assert np.isnan(o["f_pref"][o["feasible"] == 0]).all()


# ------------------------------------------------------------------ workload invariants
def test_preferred_workload_invariants():
    inp = W.make_llms(n_gpus=96)
    q, lut = inp["llms"], inp["lut"]
    o = oracle.preferred(inp)
    NS, NF = lut["n_sm"], lut["n_freq"]
    live = np.arange(q["max_inst"])[None, :] < q["n_inst"][:, None]
    assert 0.6 < o["feasible"][live].mean() < 1.0
    for g in range(q["n_gpus"]):
        for i in range(int(q["n_inst"][g])):
            if not o["feasible"][g, i]:
                continue
            for decode, js, ks in ((False, "sm_p", "f_p"), (True, "sm_d", "f_d")):
                ok, t, p = oracle.phase_cell(inp, g, i, decode, o[js][g, i], o[ks][g, i])
                assert ok
                best = p * t
                for j in range(NS):
                    for k in range(NF):
                        ok2, t2, p2 = oracle.phase_cell(inp, g, i, decode, j, k)
                        if ok2:
                            assert p2 * t2 >= best
            lo = float(min(lut["sm_level"][o["sm_p"][g, i]], lut["sm_level"][o["sm_d"][g, i]]))
            hi = float(max(lut["sm_level"][o["sm_p"][g, i]], lut["sm_level"][o["sm_d"][g, i]]))
            assert lo - 1e-12 <= o["sm_pref"][g, i] <= hi + 1e-12
            lo = float(min(lut["freq_level"][o["f_p"][g, i]], lut["freq_level"][o["f_d"][g, i]]))
            hi = float(max(lut["freq_level"][o["f_p"][g, i]], lut["freq_level"][o["f_d"][g, i]]))
            assert lo - 1e-12 <= o["f_pref"][g, i] <= hi + 1e-12


# ------------------------------------------------------------------ averages at given cells
def test_preferred_at_worked_example():
    """The two averages at hand-chosen cells of the worked example, as exact fractions."""
    inp, _, d = golden_preferred()
    for case in d["at_cells"]["cases"]:
        (jp, kp), (jd, kd) = case["prefill"], case["decode"]
        ok, sm, f = oracle.preferred_at(inp, 0, 0, jp, kp, jd, kd)
        assert ok == bool(case["feasible"]), case
        if ok:
            for got, (num, den) in ((sm, case["sm_pref"]), (f, case["f_pref"])):
                assert got == pytest.approx(float(Fraction(num) / Fraction(den)), rel=1e-15), case


def _averages_from_cells(inp, g, i, jp, kp, jd, kd):
    """Eq. preferred_sm / preferred_frequency at the given cells, from brute.phase_cells."""
    from brute import phase_cells
    NF = inp["lut"]["n_freq"]
    P = {c: (t, p) for _, c, t, p in phase_cells(inp, g, i, False)}
    D = {c: (t, p) for _, c, t, p in phase_cells(inp, g, i, True)}
    if jp * NF + kp not in P or jd * NF + kd not in D:
        return None
    (tp, pp), (td, pd) = P[jp * NF + kp], D[jd * NF + kd]
    sp, sd = float(inp["lut"]["sm_level"][jp]), float(inp["lut"]["sm_level"][jd])
    fp, fd = float(inp["lut"]["freq_level"][kp]), float(inp["lut"]["freq_level"][kd])
    return (sp * tp + sd * td) / (tp + td), (pp * tp * fp + pd * td * fd) / (pp * tp + pd * td)


def test_preferred_at_brute_force():
    """Every cell pair of tiny random fleets: feasible exactly when both cells meet their
    SLOs, and the averages equal the enumeration's."""
    rng = np.random.default_rng(30391700)
    n = 0
    for _ in range(60):
        inp = W.make_tiny_llms(rng)
        lut, q = inp["lut"], inp["llms"]
        NS, NF = lut["n_sm"], lut["n_freq"]
        for g in range(q["n_gpus"]):
            for i in range(int(q["n_inst"][g]) if 0 <= q["n_inst"][g] <= q["max_inst"] else 0):
                for _ in range(6):
                    jp, jd = rng.integers(0, NS, 2)
                    kp, kd = rng.integers(0, NF, 2)
                    ok, sm, f = oracle.preferred_at(inp, g, i, jp, kp, jd, kd)
                    want = _averages_from_cells(inp, g, i, jp, kp, jd, kd)
                    assert ok == (want is not None)
                    if ok:
                        assert sm == pytest.approx(want[0], rel=1e-12) and f == pytest.approx(want[1], rel=1e-12)
                        n += 1
    assert n > 100


def test_preferred_at_reproduces_preferred_on_the_fleet_workload():
    """At the oracle's own preferred cells the averages are the preferred configuration's."""
    inp = W.make_llms(n_gpus=256)
    o = oracle.preferred(inp)
    q = inp["llms"]
    checked = 0
    for g in range(q["n_gpus"]):
        for i in range(int(q["n_inst"][g])):
            ok, sm, f = oracle.preferred_at(inp, g, i, o["sm_p"][g, i], o["f_p"][g, i], o["sm_d"][g, i],
                                            o["f_d"][g, i])
            assert ok == bool(o["feasible"][g, i])
            if ok:
                assert sm == o["sm_pref"][g, i] and f == o["f_pref"][g, i]
                checked += 1
    assert checked > 300
