"""Generator tests: determinism, shapes, ranges, and the closed-form tables."""
import numpy as np
import pytest

from paper_2606_30391_amd import workloads as W


def _eq(a, b):
    if isinstance(a, dict):
        return all(_eq(a[k], b[k]) for k in a if k != "models_per_gpu")
    if a is None:
        return b is None
    return np.array_equal(np.asarray(a), np.asarray(b))


@pytest.mark.parametrize("cfg", [1, 2, 3, 4])
def test_placement_deterministic_and_shaped(cfg):
    a = W.make_placement(cfg)
    b = W.make_placement(cfg)
    for part in ("lut", "gpus", "requests"):
        assert _eq(a[part], b[part])
    lut, gp, rq = a["lut"], a["gpus"], a["requests"]
    M, NS, NF = lut["n_models"], lut["n_sm"], lut["n_freq"]
    assert lut["pf"].shape == (M, 32, NS, NF) and lut["pf"].dtype == np.float32
    assert gp["batch"].shape == (gp["n_waves"], gp["n_gpus"])
    assert gp["batch"].min() >= 0 and gp["batch"].max() <= 31
    assert rq["model"].min() >= 0 and rq["model"].max() < M
    assert np.all(np.diff(lut["sm_level"]) > 0) and np.all(np.diff(lut["freq_level"]) > 0)
    assert np.all(np.isfinite(lut["pf"])) and lut["pf"].min() > 0
    if cfg > 1:
        assert rq["prompt_tokens"].min() >= 16 and rq["prompt_tokens"].max() <= 8192
        assert rq["pred_out_tokens"].min() >= 1
    # every GPU hosts at least one model
    assert np.all(gp["resident"].any(axis=1))


def test_seeds_differ():
    a, b = W.make_placement(2), W.make_placement(2, seed=W.config_seed(2, 100))
    assert not np.array_equal(a["requests"]["model"], b["requests"]["model"])


def test_levels_exact():
    assert list(W.sm_levels(4)) == [0.25, 0.5, 0.75, 1.0]
    assert list(W.sm_levels(8)) == [(j + 1) / 8 for j in range(8)]
    f = W.freq_levels(16)
    assert f[0] == 0.5 and f[-1] == 1.0
    assert np.allclose(np.diff(f.astype(np.float64)), 0.5 / 15, rtol=1e-6)


def test_tiny_tables_closed_form():
    d = W.make_placement(1)
    lut, a, c = d["lut"], d["meta"]["a"], d["meta"]["c"]
    s, f = lut["sm_level"].astype(np.float64), lut["freq_level"].astype(np.float64)
    b = np.arange(1, 33, dtype=np.float64)
    ref = a[:, None, None, None] + c[:, None, None, None] * b[None, :, None, None] / (s[:, None] * f[None, :])[None, None]
    assert np.array_equal(lut["dc"], ref.astype(np.float32))
    assert np.array_equal(lut["pf"], lut["dc"])


def test_config3_planted_and_config4_caps():
    d3 = W.make_placement(3)
    pl = d3["meta"]["planted"]
    assert 0.08 < pl.mean() < 0.12
    assert np.all(d3["requests"]["slo_ttft_ms"][pl] == 1.0)
    d4 = W.make_placement(4)
    assert set(np.unique(d4["gpus"]["cap_pf"])) <= {1, 3, 5}
    assert d4["gpus"]["n_waves"] == 64
    assert np.array_equal(np.bincount(d4["requests"]["wave"]), np.full(64, 4096))


def test_fleet_budgets():
    f = W.make_fleet()["fleet"]
    assert f["n_inst"].min() >= 1 and f["n_inst"].max() <= 4
    assert f["hbm_mib"].max() <= W.HBM_CAP_MIB
    assert np.all(f["util"] == (f["sm_permille"] / 1000.0).astype(np.float32))
    assert f["sm_permille"].max() <= 600
    for g in range(0, 2048, 97):
        ms = f["inst_model"][g, : f["n_inst"][g]]
        assert len(set(ms.tolist())) == len(ms)
