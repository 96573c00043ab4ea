"""Pins of the migration (consolidation pair) oracle against things other than itself:
a hand-worked golden example, set-based enumeration on tiny fleets, the loose-SLO /
unbounded-budget closed form (a textbook argmin), and invariants on configuration 5."""
import numpy as np
import pytest

import oracle
from brute import brute_migrations, feasible_levels, migration_pairs
from conftest import golden_migration
from paper_2606_30391_amd import workloads as W


def test_worked_example():
    inp, exp, _ = golden_migration()
    b, s, k = oracle.score_migrations(inp)
    assert b.tolist() == exp["best_dst"]
    assert s.tolist() == exp["saving_w"]
    assert k.tolist() == exp["freq_level"]


def test_worked_example_budget_boundary_is_inclusive():
    inp, _, _ = golden_migration()
    # s2 -> d0 needs 300000 MiB: with a budget of exactly 300000 it fits
    inp["fleet"]["hbm_cap_mib"] = 300000
    ok, kstar, sv = oracle.pair_saving(inp, 2, 0)
    # k*=1 (s2 needs level 1), d0's own lowest level is 0:
    # 100 - 300*((0.5+0.25)*1 - 0.125*0.25) = 100 - 215.625
    assert ok and kstar == 1 and sv == 100.0 - 300.0 * (0.75 - 0.03125)
    inp["fleet"]["hbm_cap_mib"] = 299999
    assert not oracle.pair_saving(inp, 2, 0)[0]


@pytest.mark.parametrize("seed", range(5))
def test_brute_force_random(seed):
    rng = np.random.default_rng(2000 + seed)
    for _ in range(40):
        inp = W.make_tiny_fleet(rng)
        b1, s1, k1 = oracle.score_migrations(inp)
        b2, s2, k2 = brute_migrations(inp)
        assert np.array_equal(k1 >= 0, k2 >= 0)
        for s in range(inp["fleet"]["n_gpus"]):
            if b1[s] == b2[s]:
                assert k1[s] == k2[s]
                assert s1[s] == s2[s] or abs(s1[s] - s2[s]) <= 1e-12 * max(abs(s2[s]), 1.0)
            else:
                assert abs(s1[s] - s2[s]) <= 1e-12 * max(abs(s2[s]), 1.0)


@pytest.mark.parametrize("K", [1, 2, 6])
def test_brute_force_instance_slots(K):
    rng = np.random.default_rng(2200 + K)
    for _ in range(30):
        inp = W.make_tiny_fleet(rng, K=K)
        b1, s1, k1 = oracle.score_migrations(inp)
        b2, s2, k2 = brute_migrations(inp)
        assert np.array_equal(k1 >= 0, k2 >= 0)
        assert np.array_equal(b1, b2) and np.array_equal(k1, k2)
        assert np.allclose(s1, s2, rtol=1e-12, atol=1e-12) or np.array_equal(s1, s2)


def test_brute_force_bad_elements():
    rng = np.random.default_rng(2100)
    for _ in range(30):
        inp = W.make_tiny_fleet(rng)
        fl = inp["fleet"]
        G = fl["n_gpus"]
        fl["n_inst"][rng.random(G) < 0.15] = 0
        fl["n_inst"][rng.random(G) < 0.1] = 9
        fl["inst_model"][rng.random(fl["inst_model"].shape) < 0.1] = 50
        fl["inst_sm"][rng.random(fl["inst_sm"].shape) < 0.1] = -2
        fl["inst_batch"][rng.random(fl["inst_batch"].shape) < 0.1] = -1
        fl["inst_prompt_tokens"][rng.random(fl["inst_prompt_tokens"].shape) < 0.1] = -9
        b1, s1, k1 = oracle.score_migrations(inp)
        b2, s2, k2 = brute_migrations(inp)
        assert np.array_equal(b1, b2) and np.array_equal(k1, k2)


@pytest.mark.parametrize("seed", range(3))
def test_loose_slo_unbounded_budget_is_argmin_of_k(seed):
    """Every level is feasible for every GPU: k* = kd0 = 0, so
    saving(s, d) = P0 - k_d * f0^3 * u_s, maximal at the d != s with the least k_d."""
    rng = np.random.default_rng(3000 + seed)
    inp = W.make_tiny_fleet(rng, G=12, loose=True, huge_budget=True)
    fl = inp["fleet"]
    fl["n_inst"][:] = np.clip(fl["n_inst"], 1, 4)
    fl["inst_model"][:] = 0
    fl["inst_sm"][:] = 0
    fl["inst_batch"][:] = 0
    fl["inst_prompt_tokens"][:] = 10
    b, s, k = oracle.score_migrations(inp)
    kd = fl["k_dyn_w"].astype(np.float64)
    f0 = float(inp["lut"]["freq_level"][0])
    p0 = inp["lut"]["p0_w"]
    for src in range(fl["n_gpus"]):
        others = np.where(np.arange(fl["n_gpus"]) == src, np.inf, kd)
        us = float(fl["util"][src])
        if us > 0:
            exp_d = int(np.argmin(others))
        else:
            exp_d = 0 if src != 0 else 1                    # all savings equal P0
        assert b[src] == exp_d and k[src] == 0
        assert s[src] == pytest.approx(p0 - kd[exp_d] * f0 ** 3 * us, rel=1e-12)


def _levels_table(inp):
    return [feasible_levels(inp, g) for g in range(inp["fleet"]["n_gpus"])]


def test_invariants_on_config5_sample():
    inp = W.make_fleet()
    fl = inp["fleet"]
    G = fl["n_gpus"]
    sel = np.random.default_rng(5).choice(G, 40, replace=False)
    b, s, k = oracle.score_migrations(inp, sel)
    lv = _levels_table(inp)
    assert 0.3 < (b >= 0).mean() < 1.0
    for i, src in enumerate(sel):
        if b[i] < 0:
            assert k[i] == -1 and s[i] == -np.inf
            # no destination may be feasible
            for d in range(G):
                if d == src:
                    continue
                fits = (fl["hbm_mib"][src] + fl["hbm_mib"][d] <= fl["hbm_cap_mib"]
                        and fl["sm_permille"][src] + fl["sm_permille"][d] <= fl["sm_cap_permille"])
                assert not (fits and (lv[src] & lv[d]))
            continue
        d = int(b[i])
        assert d != src
        assert fl["hbm_mib"][src] + fl["hbm_mib"][d] <= fl["hbm_cap_mib"]
        assert fl["sm_permille"][src] + fl["sm_permille"][d] <= fl["sm_cap_permille"]
        both = lv[src] & lv[d]
        assert k[i] in both and k[i] == min(both)        # all SLOs hold; no lower level does
        # the saving is maximal over all destinations (set-based enumeration)
        best = max(t[0] for t in migration_pairs(inp, int(src)))
        assert s[i] == pytest.approx(best, rel=1e-12)
