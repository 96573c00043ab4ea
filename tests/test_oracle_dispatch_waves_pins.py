"""Pins of the wave-by-wave dispatch oracle (Sec. 3.3's dispatcher over arrival waves, each
wave committed to the GPUs' state before the next).

* a hand-worked example of four waves whose every decision depends on one commit rule
  (two requests of one wave share a snapshot; memory is taken from the admitting step on;
  the decode batch grows; an F_max placement leaves its GPU boosted),
* a closed form: identical requests, one GPU, one profile step -- as many fit as the
  free memory holds at ceil(need / 1024) MiB each, the rest scale out, and the i-th
  placed one pays for batch B + i,
* reduction: one wave is the one-snapshot dispatcher (itself pinned by enumeration in
  tests/test_oracle_dispatch_pins.py),
* conservation on random instances: the batches grow by the placements, the free memory
  shrinks by at most their demand, frequencies change only to the top level,
* argument checks.
"""
import numpy as np
import pytest

import oracle
from brute import brute_dispatch
from paper_2606_30391_amd import workloads as W


def worked_example():
    """Two GPUs, one model, two profile steps, constant tables; p0 = 100 W and no dynamic
    power, so E = 100 * (TTFT + Lout * TBT).  TTFT is 10 ms at level 0 and 5 ms at the top
    level 1; TBT on batch row b is 1 + (b-1)/4 ms at both levels.  KV cache 1024 KiB per
    token, so a request needs (prompt + Lout) MiB.

    GPU 0: level 0, batch 0, steps (t 0: 100 MiB, SM 0), (t 30: 300 MiB, SM 1).
    GPU 1: level 0, batch 0, steps (t 0:  80 MiB, SM 0), (t 30: 500 MiB, SM 1).

    wave 0: r0, r1 (39 + 21 tokens = 60 MiB, TTFT SLO 25): both GPUs admit at t 0 with
            E = 100 * (10 + 21 * 1) = 3100, an exact tie, and the most free memory wins:
            GPU 0 for both (the second does not see the first: one snapshot).
            Commit: GPU 0 batch 2; its steps lose 120 MiB from step 0 on: -20 -> -1, 180.
    wave 1: r2 (same): GPU 0 now admits only at t 30 (30 + 10 >= 25), GPU 1 at t 0: GPU 1,
            E 3100.  Commit: GPU 1 batch 1, memory 20, 440.
    wave 2: r3 (15 + 0 tokens, TTFT SLO 8): no GPU meets 8 ms at level 0 (10 ms); at the
            top level GPU 1 (t 0, 5 ms) does: the F_max fallback, E = 100 * 5 = 500.
            Commit: GPU 1 batch 2, boosted to level 1, memory 5, 425.
    wave 3: r4 (1 + 2 tokens = 3 MiB, TTFT SLO 8): GPU 1 runs at level 1 now, so Phase Two
            finds it: E = 100 * (5 + 2 * TBT(row 3) = 1.5) = 800.
            r5 (60 MiB, TTFT SLO 100), same snapshot: GPU 0 admits at t 30 on level 0 with
            b = 3: E = 100 * (10 + 21 * 1.5) = 4150; GPU 1 admits at t 30 (5 MiB at t 0)
            on level 1 with b = 3: E = 100 * (5 + 21 * 1.5) = 3650, more than 2% below:
            GPU 1, SM level 1.  Commit: GPU 1 batch 4; memory 5 - 3 = 2 at step 0 (r5 was
            admitted at step 1) and 425 - 3 - 60 = 362.
    """
    M, NS, NF = 1, 2, 2
    pf = np.zeros((M, 32, NS, NF), np.float32)
    pf[..., 0], pf[..., 1] = 10.0, 5.0
    dc = np.zeros((M, 32, NS, NF), np.float32)
    dc[:] = (1.0 + np.arange(32, dtype=np.float32) / 4.0)[None, :, None, None]
    lut = {"n_models": M, "n_rows": 32, "n_sm": NS, "n_freq": NF, "sm_level": W.sm_levels(NS),
           "freq_level": W.freq_levels(NF), "pf": pf, "dc": dc, "p0_w": 100.0}
    avail = {"n_gpus": 2, "n_steps": 2, "freq_cur": np.array([0, 0], np.int32), "batch": np.array([0, 0], np.int32),
             "k_dyn_w": np.zeros(2, np.float32), "resident": np.ones((2, 1), np.uint32),
             "t_avail_ms": np.array([[0, 30], [0, 30]], np.float32),
             "mem_free_mib": np.array([[100, 300], [80, 500]], np.int32),
             "sm_free": np.array([[0, 1], [0, 1]], np.int32),
             "kv_kib_per_token": np.array([1024], np.int32), "k_new_w": 0.0}
    requests = {"n_requests": 6, "model": np.zeros(6, np.int32), "wave": None,
                "prompt_tokens": np.array([39, 39, 39, 15, 1, 39], np.int32),
                "pred_out_tokens": np.array([20, 20, 20, 0, 1, 20], np.int32),
                "slo_ttft_ms": np.array([25, 25, 25, 8, 8, 100], np.float32),
                "slo_tbt_ms": np.full(6, 100.0, np.float32)}
    inp = {"lut": lut, "avail": avail, "requests": requests}
    wave_start = [0, 2, 3, 4, 6]
    expect = {"gpu": [0, 0, 1, 1, 1, 1], "freq_level": [0, 0, 0, 1, 1, 1], "sm_level": [0, 0, 0, 0, 0, 1],
              "phase": [1, 1, 1, 2, 1, 1], "energy": [3100.0, 3100.0, 3100.0, 500.0, 800.0, 3650.0],
              "state": {"freq_cur": [0, 1], "batch": [2, 4], "mem_free_mib": [[-1, 180], [2, 362]]}}
    return inp, wave_start, expect


def test_wave_dispatch_worked_example():
    inp, ws, exp = worked_example()
    (g, k, j, ph, e), st = oracle.dispatch_waves(inp, ws)
    assert g.tolist() == exp["gpu"]
    assert k.tolist() == exp["freq_level"]
    assert j.tolist() == exp["sm_level"]
    assert ph.tolist() == exp["phase"]
    assert e.tolist() == exp["energy"]
    for key, v in exp["state"].items():
        assert st[key].tolist() == v, key


def test_one_request_per_wave_differs_from_one_snapshot_in_the_example():
    """The first wave's two requests split over both GPUs when each is its own wave."""
    inp, _, _ = worked_example()
    (g, *_), _ = oracle.dispatch_waves(inp, [0, 1, 2, 3, 4, 5, 6])
    assert g[:2].tolist() == [0, 1]


@pytest.mark.parametrize("free,need_kib,n,batch", [(100, 30 * 1024, 6, 0), (1000, 7 * 1024, 200, 3),
                                                   (59, 60 * 1024, 3, 5), (0, 0, 4, 0), (640, 64 * 1024, 10, 28),
                                                   (100, 31232, 5, 2), (10, 8, 20, 0)])
def test_capacity_closed_form(free, need_kib, n, batch):
    """One GPU, one step with `free` MiB, n identical requests of `need_kib` KiB, each its own
    wave, SLOs that every point meets.  Each placement takes q = ceil(need / 1024) MiB, so
    the i-th request (from 0) fits while (free - i q) MiB still hold `need` KiB: that is
    floor((1024 free - need) / (1024 q)) + 1 of them (all n when nothing is needed); the
    rest go to a new GPU.  The i-th placed request is served on batch row
    min(batch + i + 1, 32), and P = p0 + k s f^3 b / 32 makes its energy the closed form
    below."""
    p0, kd, tt, tb = 50.0, 200.0, 4.0, 0.5
    NS, NF = 1, 1
    lut = {"n_models": 1, "n_rows": 32, "n_sm": NS, "n_freq": NF, "sm_level": W.sm_levels(NS),
           "freq_level": W.freq_levels(NF), "pf": np.full((1, 32, NS, NF), tt, np.float32),
           "dc": np.full((1, 32, NS, NF), tb, np.float32), "p0_w": p0}
    avail = {"n_gpus": 1, "n_steps": 1, "freq_cur": np.zeros(1, np.int32), "batch": np.array([batch], np.int32),
             "k_dyn_w": np.array([kd], np.float32), "resident": np.ones((1, 1), np.uint32),
             "t_avail_ms": np.zeros((1, 1), np.float32), "mem_free_mib": np.array([[free]], np.int32),
             "sm_free": np.zeros((1, 1), np.int32), "kv_kib_per_token": np.array([need_kib // 8], np.int32),
             "k_new_w": 0.0}
    # prompt 8 tokens, no output: need = kv * 8 KiB
    req = {"n_requests": n, "model": np.zeros(n, np.int32), "wave": None, "prompt_tokens": np.full(n, 8, np.int32),
           "pred_out_tokens": np.zeros(n, np.int32), "slo_ttft_ms": np.full(n, 1e6, np.float32),
           "slo_tbt_ms": np.full(n, 1e6, np.float32)}
    inp = {"lut": lut, "avail": avail, "requests": req}
    (g, k, j, ph, e), st = oracle.dispatch_waves(inp, list(range(n + 1)))
    q = -(-need_kib // 1024)
    fit = n if q == 0 else (0 if 1024 * free < need_kib else (1024 * free - need_kib) // (1024 * q) + 1)
    placed = min(n, fit)
    assert ph.tolist() == [1] * placed + [3] * (n - placed)
    assert g.tolist() == [0] * placed + [-1] * (n - placed)
    for i in range(placed):
        b = min(batch + i + 1, 32)
        assert e[i] == (p0 + kd * 1.0 * 1.0 * (b / 32.0)) * tt, i      # s = f = 1, Lout = 0
    assert st["batch"].tolist() == [batch + placed]
    assert st["mem_free_mib"].tolist() == [[free - placed * q]]


@pytest.mark.parametrize("seed", range(4))
def test_one_wave_is_the_snapshot_dispatcher(seed):
    rng = np.random.default_rng(7300 + seed)
    for case in range(30):
        inp = W.make_tiny_dispatch(rng, ties=(case % 3 == 0))
        R = inp["requests"]["n_requests"]
        got, _ = oracle.dispatch_waves(inp, [0, R])
        for x, y in zip(got, brute_dispatch(inp)):
            assert np.array_equal(x, y), (seed, case)


@pytest.mark.parametrize("seed", range(4))
def test_commits_conserve_placements_and_memory(seed):
    """Any wave split: each GPU's batch grows by the requests placed on it; its free memory
    at every step falls by at most their total demand in MiB (rounded up) and never below
    -1; only GPUs that took an F_max placement change level, to the top one; requests of
    the first wave see the caller's state, so they decide as the one-snapshot dispatcher."""
    rng = np.random.default_rng(7400 + seed)
    for case in range(30):
        inp = W.make_tiny_dispatch(rng, R=int(rng.integers(1, 24)), ties=(case % 3 == 0))
        av, rq = inp["avail"], inp["requests"]
        R, G = rq["n_requests"], av["n_gpus"]
        cuts = np.sort(rng.integers(0, R + 1, int(rng.integers(0, 4))))
        ws = [0, *cuts.tolist(), R]
        (g, k, j, ph, e), st = oracle.dispatch_waves(inp, ws)
        first = brute_dispatch({**inp, "requests": {**rq, "n_requests": ws[1]}})
        assert np.array_equal(g[:ws[1]], first[0]) and np.array_equal(ph[:ws[1]], first[3])
        placed = (ph == 1) | (ph == 2)
        assert np.array_equal(st["batch"] - av["batch"], np.bincount(g[placed], minlength=G))
        lout = (rq["pred_out_tokens"].astype(np.int64) * 105 + 99) // 100
        need = av["kv_kib_per_token"][rq["model"]].astype(np.int64) * (rq["prompt_tokens"] + lout)
        demand = np.bincount(g[placed], weights=(need[placed] + 1023) // 1024, minlength=G)
        drop = av["mem_free_mib"].astype(np.int64) - st["mem_free_mib"]
        assert (drop >= 0).all() and (drop <= demand[:, None]).all() and (st["mem_free_mib"] >= -1).all()
        boosted = np.zeros(G, bool)
        boosted[g[ph == 2]] = True
        top = inp["lut"]["n_freq"] - 1
        assert np.array_equal(st["freq_cur"], np.where(boosted, top, av["freq_cur"]))


def test_rejects_bad_wave_bounds():
    inp, _, _ = worked_example()
    for ws in ([0, 2, 3], [1, 6], [0, 4, 3, 6], [0, 7]):
        with pytest.raises(ValueError):
            oracle.dispatch_waves(inp, ws)
