"""Pins of the placement oracle against things other than itself.

* hand-worked golden examples (exact arithmetic, tests/golden/),
* exhaustive enumeration on tiny random instances (tests/brute.py),
* closed forms: analytic tables, the k=0 special case (a textbook argmin), the
  convex energy-frequency curve of Eq. energy (the continuous optimum is a root of
  a quartic, found with numpy.roots; the grid optimum must bracket it),
* metamorphic relations (scaling, permutation, monotonicity, duplication),
* invariants on the five configurations (feasibility, optimality, planted flags).
"""
import numpy as np
import pytest
from hypothesis import given, settings
from hypothesis import strategies as st

import oracle
from brute import brute_placements, padded_out as bpad, prompt_row as brow
from conftest import golden_placement, load_golden
from paper_2606_30391_amd import workloads as W


# ------------------------------------------------------------------ golden values
def test_preprocess_golden():
    g = load_golden("preprocess.json")
    for e in g["padded_out"]:
        assert oracle.padded_out(e["pred"]) == e["out"], e
        assert bpad(e["pred"]) == e["out"], e
    for e in g["prompt_row"]:
        assert oracle.prompt_row(e["tokens"]) == e["row"], e
        exp = None if e["row"] == -2 else e["row"]
        assert brow(e["tokens"]) == exp, e


def test_worked_example():
    inp, exp, d = golden_placement()
    ch, fe, en = oracle.score_placements(inp)
    assert ch[0] == exp["choice"] and fe[0] == exp["feasible"] and en[0] == exp["energy_mj"]
    allE = {int(k): v for k, v in exp["all_energies"].items()}
    for idx in range(2 * 2 * 2):
        ok, e = oracle.candidate_energy(inp, 0, idx)
        assert ok == (idx in allE), idx
        if ok:
            assert e == allE[idx], idx


def test_worked_example_capped():
    inp, exp, _ = golden_placement("capped")
    ch, fe, en = oracle.score_placements(inp)
    assert (ch[0], fe[0], en[0]) == (exp["choice"], exp["feasible"], exp["energy_mj"])


def test_strict_slo_boundary():
    inp, _, _ = golden_placement()
    # TBT of g0 (j1,k1) is 5: an SLO of exactly 5 must reject it, 5+ulp must accept it
    inp["requests"]["slo_tbt_ms"][:] = 5.0
    ok, _ = oracle.candidate_energy(inp, 0, 3)
    assert not ok
    inp["requests"]["slo_tbt_ms"][:] = np.nextafter(np.float32(5.0), np.float32(10))
    ok, e = oracle.candidate_energy(inp, 0, 3)
    assert ok and e == 15000.0


# ------------------------------------------------------------------ brute force
def _agree(inp):
    c1, f1, e1 = oracle.score_placements(inp)
    c2, f2, e2 = brute_placements(inp)
    assert np.array_equal(f1, f2)
    for r in range(len(c1)):
        if c1[r] == c2[r]:
            assert (e1[r] == e2[r]) or abs(e1[r] - e2[r]) <= 1e-12 * abs(e2[r]), r
        else:
            # different summation order in float64 may only separate candidates
            # whose energies agree to 1e-12
            assert abs(e1[r] - e2[r]) <= 1e-12 * abs(e2[r]), (r, c1[r], c2[r])
            ok, e = oracle.candidate_energy(inp, r, int(c2[r]))
            assert ok and abs(e - e1[r]) <= 1e-12 * abs(e1[r])


@pytest.mark.parametrize("seed", range(10))
def test_brute_force_random(seed):
    """2,000 random tiny instances (R <= 8, G <= 5, NS <= 4, NF <= 6, M <= 3)."""
    rng = np.random.default_rng(1000 + seed)
    for _ in range(200):
        _agree(W.make_tiny_placement(rng))


@settings(max_examples=300, deadline=None)
@given(seed=st.integers(0, 2**32 - 1), caps=st.booleans(), ties=st.booleans(), nan_cells=st.booleans(),
       waves=st.integers(1, 2))
def test_brute_force_search(seed, caps, ties, nan_cells, waves):
    """Hypothesis explores generator seeds and flags (and shrinks a failure to a small one)."""
    inp = W.make_tiny_placement(np.random.default_rng(seed), caps=caps, ties=ties, nan_cells=nan_cells, W=waves)
    _agree(inp)


def test_brute_force_ties():
    rng = np.random.default_rng(77)
    for _ in range(60):
        inp = W.make_tiny_placement(rng, ties=True)
        c1, f1, e1 = oracle.score_placements(inp)
        c2, f2, e2 = brute_placements(inp)
        assert np.array_equal(c1, c2) and np.array_equal(f1, f2)


def test_brute_force_nan_inf_tables():
    rng = np.random.default_rng(78)
    for _ in range(60):
        _agree(W.make_tiny_placement(rng, nan_cells=True))


def test_brute_force_bad_elements():
    rng = np.random.default_rng(79)
    for _ in range(40):
        inp = W.make_tiny_placement(rng, caps=True)
        R, G = inp["requests"]["n_requests"], inp["gpus"]["n_gpus"]
        q, g = inp["requests"], inp["gpus"]
        q["model"][rng.random(R) < 0.2] = inp["lut"]["n_models"] + 3
        q["model"][rng.random(R) < 0.1] = -1
        q["wave"][rng.random(R) < 0.1] = g["n_waves"]
        q["prompt_tokens"][rng.random(R) < 0.1] = -7
        q["pred_out_tokens"][rng.random(R) < 0.1] = -1
        g["batch"][rng.random(g["batch"].shape) < 0.2] = -3
        g["batch"][rng.random(g["batch"].shape) < 0.2] = 99
        g["cap_pf"][rng.random(G) < 0.2] = 100
        g["cap_dc"][rng.random(G) < 0.2] = -1
        _agree(inp)


# ------------------------------------------------------------------ closed forms
def _analytic_energy(d, r, idx):
    """Energy of a candidate from the generator's latency parameters (not the tables)."""
    lut, gp, rq, meta = d["lut"], d["gpus"], d["requests"], d["meta"]
    NS, NF = lut["n_sm"], lut["n_freq"]
    g, j, k = idx // (NS * NF), (idx // NF) % NS, idx % NF
    m, w = int(rq["model"][r]), int(rq["wave"][r])
    b = min(int(gp["batch"][w, g]) + 1, 32)
    s = float(lut["sm_level"][j]); f = float(lut["freq_level"][k])
    a, c = meta["a"][m], meta["c"][m]
    tbt = a + c * b / (s * f)
    if meta["cp"] is None:
        ttft = tbt
    else:
        tok = 256 * (min(-(-int(rq["prompt_tokens"][r]) // 256), 32))
        ttft = a + meta["cp"][m] * tok / (s * f)
    P = lut["p0_w"] + float(gp["k_dyn_w"][g]) * s * f ** 3 * (b / 32)
    return P * ttft + bpad(int(rq["pred_out_tokens"][r])) * P * tbt


@pytest.mark.parametrize("cfg", [1, 2])
def test_energy_matches_analytic_tables(cfg):
    d = W.make_placement(cfg)
    rng = np.random.default_rng(5)
    R = d["requests"]["n_requests"]
    sel = rng.choice(R, min(R, 300), replace=False)
    ch, fe, en = oracle.score_placements(d, sel)
    n_checked = 0
    for i, r in enumerate(sel):
        if fe[i]:
            ref = _analytic_energy(d, r, int(ch[i]))
            assert abs(en[i] - ref) <= 1e-6 * ref
            n_checked += 1
        # also random candidates of this request
        NS, NF, G = d["lut"]["n_sm"], d["lut"]["n_freq"], d["gpus"]["n_gpus"]
        for idx in rng.integers(0, G * NS * NF, 20):
            ok, e = oracle.candidate_energy(d, r, int(idx))
            if ok:
                ref = _analytic_energy(d, r, int(idx))
                assert abs(e - ref) <= 1e-6 * ref
    assert n_checked > 0


def test_zero_dynamic_power_is_lowest_latency():
    """k_g = 0: E = P0 * TTFT (no decode in the tiny configuration), so the choice is
    the lowest-latency feasible cell: the least-loaded GPU (lowest index on equal
    load) at the top SM and frequency levels."""
    d = W.make_placement(1)
    d["gpus"]["k_dyn_w"][:] = 0.0
    ch, fe, en = oracle.score_placements(d)
    NS, NF = d["lut"]["n_sm"], d["lut"]["n_freq"]
    gbest = int(np.argmin(d["gpus"]["batch"][0]))
    exp = (gbest * NS + NS - 1) * NF + NF - 1
    b = d["gpus"]["batch"][0, gbest] + 1
    for r in range(d["requests"]["n_requests"]):
        lat = d["lut"]["dc"][d["requests"]["model"][r], b - 1, NS - 1, NF - 1]
        if lat < 50.0:
            assert fe[r] == 1 and ch[r] == exp
            assert en[r] == pytest.approx(120.0 * float(lat), rel=1e-12)
        else:
            assert fe[r] == 0


@pytest.mark.parametrize("lout_pred", [0, 40])
def test_convex_frequency_optimum_brackets_quartic_root(lout_pred):
    """Eq. energy with P = P0 + K f^3 and time A + C/f is strictly convex in f>0;
    dE/df = 0  <=>  3 K A f^4 + 2 K C f^3 - P0 C = 0 (one positive root).  The grid
    argmin must be one of the two levels around that root."""
    rng = np.random.default_rng(11)
    NF = 41
    f = np.linspace(0.2, 1.0, NF).astype(np.float32)
    for trial in range(40):
        a1, c1 = rng.uniform(5, 20), rng.uniform(20, 200)
        a2, c2 = rng.uniform(2, 10), rng.uniform(1, 10)
        kg = rng.uniform(300, 500)
        p0 = rng.uniform(20, 150)
        B = int(rng.integers(0, 32))
        b = B + 1
        pf = np.zeros((1, 32, 1, NF), np.float32)
        dc = np.zeros((1, 32, 1, NF), np.float32)
        pf[0, 3, 0, :] = a1 + c1 / f.astype(np.float64)
        dc[0, b - 1, 0, :] = a2 + c2 / f.astype(np.float64)
        lut = {"n_models": 1, "n_rows": 32, "n_sm": 1, "n_freq": NF,
               "sm_level": np.ones(1, np.float32), "freq_level": f, "pf": pf, "dc": dc, "p0_w": p0}
        gpus = {"n_gpus": 1, "n_waves": 1, "batch": np.array([[B]], np.int32),
                "k_dyn_w": np.array([kg], np.float32), "resident": np.ones((1, 1), np.uint32),
                "cap_pf": None, "cap_dc": None}
        req = {"n_requests": 1, "model": np.zeros(1, np.int32), "wave": None,
               "prompt_tokens": np.array([1000], np.int32),        # row 3
               "pred_out_tokens": np.array([lout_pred], np.int32),
               "slo_ttft_ms": np.array([1e30], np.float32), "slo_tbt_ms": np.array([1e30], np.float32)}
        ch, fe, en = oracle.score_placements({"lut": lut, "gpus": gpus, "requests": req})
        lout = bpad(lout_pred)
        A = a1 + lout * a2
        Cc = c1 + lout * c2
        K = float(np.float32(kg)) * b / 32
        roots = np.roots([3 * K * A, 2 * K * Cc, 0.0, 0.0, -p0 * Cc])
        fstar = [x.real for x in roots if abs(x.imag) < 1e-9 and x.real > 0]
        assert len(fstar) == 1
        fstar = fstar[0]
        fl = f.astype(np.float64)
        if fstar <= fl[0]:
            allowed = {0}
        elif fstar >= fl[-1]:
            allowed = {NF - 1}
        else:
            hi = int(np.searchsorted(fl, fstar))
            allowed = {hi - 1, hi}
        assert fe[0] == 1 and int(ch[0]) in allowed, (trial, fstar, int(ch[0]))


# ------------------------------------------------------------------ metamorphic
def test_scaling_power_by_two_scales_energy_exactly():
    d = W.make_placement(2)
    sel = np.arange(0, 4096, 7)
    c1, f1, e1 = oracle.score_placements(d, sel)
    d["lut"]["p0_w"] *= 2.0
    d["gpus"]["k_dyn_w"] = d["gpus"]["k_dyn_w"] * np.float32(2.0)
    c2, f2, e2 = oracle.score_placements(d, sel)
    assert np.array_equal(c1, c2) and np.array_equal(f1, f2)
    m = f1 == 1
    assert np.array_equal(e2[m], 2.0 * e1[m])


def test_gpu_permutation():
    d = W.make_placement(3, n_requests=600)
    G, NS, NF = d["gpus"]["n_gpus"], d["lut"]["n_sm"], d["lut"]["n_freq"]
    c1, f1, e1 = oracle.score_placements(d)
    perm = np.random.default_rng(3).permutation(G)      # new position p holds old GPU perm[p]
    inv = np.argsort(perm)
    g = d["gpus"]
    d2 = {"lut": d["lut"], "requests": d["requests"],
          "gpus": {"n_gpus": G, "n_waves": 1, "batch": g["batch"][:, perm].copy(),
                   "k_dyn_w": g["k_dyn_w"][perm].copy(), "resident": g["resident"][perm].copy(),
                   "cap_pf": None, "cap_dc": None}}
    c2, f2, e2 = oracle.score_placements(d2)
    assert np.array_equal(f1, f2)
    m = f1 == 1
    old_g = c1[m] // (NS * NF)
    cell = c1[m] % (NS * NF)
    assert np.array_equal(c2[m], inv[old_g] * NS * NF + cell)
    assert np.array_equal(e1[m], e2[m])


def test_tighter_slo_never_lowers_energy_and_more_gpus_never_raise_it():
    d = W.make_placement(2, n_requests=800)
    _, f0, e0 = oracle.score_placements(d)
    d["requests"]["slo_tbt_ms"] = d["requests"]["slo_tbt_ms"] * np.float32(0.7)
    _, f1, e1 = oracle.score_placements(d)
    assert np.all(f1 <= f0) and np.all(e1[f1 == 1] >= e0[f1 == 1])
    d = W.make_placement(2, n_requests=800)
    small = W.make_placement(2, n_requests=800)
    keep = 40
    small["gpus"] = {k: (v[..., :keep] if k == "batch" else v[:keep]) if isinstance(v, np.ndarray) else v
                     for k, v in d["gpus"].items()}
    small["gpus"]["n_gpus"] = keep
    _, fs, es = oracle.score_placements(small)
    _, fb, eb = oracle.score_placements(d)
    assert np.all(fs <= fb) and np.all(eb[fs == 1] <= es[fs == 1])


def test_duplicated_gpu_and_request_tie_to_lower_index():
    d = W.make_placement(2, n_requests=500)
    c1, f1, e1 = oracle.score_placements(d)
    g = d["gpus"]
    G = g["n_gpus"]
    d2 = {"lut": d["lut"], "requests": d["requests"],
          "gpus": {"n_gpus": 2 * G, "n_waves": 1, "batch": np.concatenate([g["batch"], g["batch"]], 1),
                   "k_dyn_w": np.concatenate([g["k_dyn_w"]] * 2),
                   "resident": np.concatenate([g["resident"]] * 2), "cap_pf": None, "cap_dc": None}}
    c2, f2, e2 = oracle.score_placements(d2)
    assert np.array_equal(c1, c2) and np.array_equal(e1, e2)
    # duplicated requests give identical outputs
    sel = np.array([5, 5, 17, 17])
    c3, _, e3 = oracle.score_placements(d, sel)
    assert c3[0] == c3[1] and c3[2] == c3[3] and e3[0] == e3[1]


# ------------------------------------------------------------------ invariants on the configs
def _all_candidates(d, r):
    """Vectorised feasibility and energy of every (g, j, k) of request r (numpy, float64)."""
    lut, gp, rq = d["lut"], d["gpus"], d["requests"]
    NS, NF, G = lut["n_sm"], lut["n_freq"], gp["n_gpus"]
    m, w = int(rq["model"][r]), int(rq["wave"][r])
    host = ((gp["resident"][:, m // 32] >> np.uint32(m % 32)) & 1).astype(bool)
    b = np.minimum(gp["batch"][w] + 1, 32)
    j = np.arange(NS)
    capp = np.full(G, NS - 1) if gp["cap_pf"] is None else gp["cap_pf"].astype(int)
    capd = np.full(G, NS - 1) if gp["cap_dc"] is None else gp["cap_dc"].astype(int)
    jp = np.minimum(j[None, :], capp[:, None])            # [G][NS]
    jd = np.minimum(j[None, :], capd[:, None])
    pt = int(rq["prompt_tokens"][r])
    prow = (np.full(G, min(-(-pt // 256), 32) - 1) if pt > 0 else b - 1)
    ttft = lut["pf"][m][prow[:, None], jp]                # [G][NS][NF]
    tbt = lut["dc"][m][(b - 1)[:, None], jd]
    feas = (ttft < rq["slo_ttft_ms"][r]) & (tbt < rq["slo_tbt_ms"][r]) & host[:, None, None]
    f3 = lut["freq_level"].astype(np.float64) ** 3
    s = lut["sm_level"].astype(np.float64)
    ku = gp["k_dyn_w"].astype(np.float64) * b / 32
    Pp = lut["p0_w"] + ku[:, None, None] * s[jp][:, :, None] * f3[None, None, :]
    Pd = lut["p0_w"] + ku[:, None, None] * s[jd][:, :, None] * f3[None, None, :]
    lout = bpad(int(rq["pred_out_tokens"][r]))
    E = Pp * ttft + lout * Pd * tbt
    return feas.reshape(-1), E.reshape(-1)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_invariants_on_configs(cfg):
    d = W.make_placement(cfg)
    R = d["requests"]["n_requests"]
    sel = np.random.default_rng(cfg).choice(R, min(R, 250), replace=False)
    ch, fe, en = oracle.score_placements(d, sel)
    for i, r in enumerate(sel):
        feas, E = _all_candidates(d, r)
        assert fe[i] == (1 if feas.any() else 0)
        if fe[i]:
            assert feas[ch[i]]
            assert abs(E[ch[i]] - en[i]) <= 1e-12 * en[i]
            lower = feas & (E < en[i] * (1 - 1e-12))
            assert not lower.any()
            # among (numerically) equal energies the lowest index was taken
            eq = np.flatnonzero(feas & (np.abs(E - en[i]) <= 1e-12 * en[i]))
            assert ch[i] == eq.min()
        else:
            assert ch[i] == -1 and en[i] == np.inf


def test_config3_planted_requests_are_flagged():
    d = W.make_placement(3)
    pl = np.flatnonzero(d["meta"]["planted"])[:400]
    ch, fe, en = oracle.score_placements(d, pl)
    assert np.all(fe == 0) and np.all(ch == -1) and np.all(np.isinf(en))


def test_config4_capped_levels_prefer_lower_sm_level():
    """Levels above both caps duplicate the capped cell exactly; the lower level wins."""
    d = W.make_placement(4)
    sel = np.arange(0, 262144, 509)
    ch, fe, _ = oracle.score_placements(d, sel)
    NS, NF = d["lut"]["n_sm"], d["lut"]["n_freq"]
    g = ch[fe == 1] // (NS * NF)
    j = (ch[fe == 1] // NF) % NS
    top = np.maximum(d["gpus"]["cap_pf"][g], d["gpus"]["cap_dc"][g])
    assert np.all(j <= top)
