"""GPU parity of the paper's own dispatcher (Sec. 3.3: current frequency, 2% stability
tie-break, F_max fallback, scale-out): the HIP path through the C ABI against the CPU
oracle.  Both evaluate the same float64 energies in the same order, so every output must
match exactly: GPU, levels, phase, and the energy rounded to float32."""
import sys

import numpy as np
import pytest

import oracle
from conftest import golden_dispatch, load_golden
from oracle.check import check_dispatch
from paper_2606_30391_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

VARIANTS = [v["name"] for v in load_golden("dispatch_worked_example.json")["variants"]]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run(inp):
    from paper_2606_30391_amd import festina as F
    F.lib()
    dd = F.DeviceDispatch(inp, "cuda")
    dd.run()
    torch.cuda.synchronize()
    return dd.results()


def parity(inp, label=""):
    say(f"[gpu] dispatch {label}: R={inp['requests']['n_requests']} G={inp['avail']['n_gpus']} "
        f"S={inp['avail']['n_steps']} NS={inp['lut']['n_sm']} NF={inp['lut']['n_freq']}")
    got = run(inp)
    ref = oracle.dispatch(inp)
    rep = check_dispatch(ref, got)
    say(f"      {rep}; phases {np.bincount(got[3], minlength=4).tolist()}")
    assert rep.ok, str(rep)
    return got


def test_dispatch_workload_full_size():
    got = parity(W.make_dispatch(), label="65536 requests, 512 GPUs")
    ph = np.bincount(got[3], minlength=4)
    assert ph[1] > 0.5 * ph.sum() and ph[2] > 0 and ph[3] > 0 and ph[0] > 0


@pytest.mark.parametrize("extra", [100, 200])
def test_dispatch_workload_seeds(extra):
    parity(W.make_dispatch(seed=W.DISPATCH_SEED + extra, n_requests=8000, n_gpus=1024), label=f"seed +{extra}")


@pytest.mark.parametrize("variant", [None] + VARIANTS)
def test_dispatch_worked_example(variant):
    inp, exp, d = golden_dispatch(variant)
    g, k, j, ph, e = run(inp)
    assert (int(g[0]), int(k[0]), int(j[0]), int(ph[0])) == (exp["gpu"], exp["freq_level"], exp["sm_level"],
                                                              exp["phase"])
    assert e[0] == (np.inf if exp["energy_mj"] is None else np.float32(exp["energy_mj"]))


@pytest.mark.parametrize("NS,NF,S", [(1, 1, 1), (3, 5, 2), (4, 8, 3), (8, 16, 9), (16, 16, 4), (2, 70, 1)])
def test_dispatch_shapes(NS, NF, S):
    rng = np.random.default_rng(1500 + NS * 100 + NF)
    parity(W.make_tiny_dispatch(rng, R=3000, G=150, M=3, NS=NS, NF=NF, S=S), label="shapes")


def test_dispatch_exact_and_near_ties():
    rng = np.random.default_rng(1600)
    inp = W.make_tiny_dispatch(rng, R=4000, G=90, M=2, NS=3, NF=4, S=2, ties=True)
    parity(inp, label="ties")
    inp["avail"]["k_dyn_w"][:] = 0.0
    inp["avail"]["mem_free_mib"][:] = inp["avail"]["mem_free_mib"][:1]
    parity(inp, label="exact ties, equal memory")


def test_dispatch_invalid_elements():
    rng = np.random.default_rng(1700)
    inp = W.make_tiny_dispatch(rng, R=500, G=40, M=3, NS=4, NF=6, S=3)
    rq, av = inp["requests"], inp["avail"]
    rq["model"][:20] = 3
    rq["model"][20:30] = -1
    rq["prompt_tokens"][30:40] = -5
    rq["pred_out_tokens"][40:50] = -1
    av["batch"][:5] = -1
    av["freq_cur"][5:10] = 9
    av["sm_free"][10:15] = 7
    av["sm_free"][15:20] = -1
    got = parity(inp, label="invalid elements")
    assert np.all(got[3][:50] == 0)


def test_dispatch_many_hosts():
    """More hosting GPUs than lanes in a wavefront: several hosts per lane."""
    rng = np.random.default_rng(1800)
    parity(W.make_tiny_dispatch(rng, R=700, G=700, M=2, NS=4, NF=6, S=2), label="700 GPUs")


def test_dispatch_negative_energies():
    rng = np.random.default_rng(1900)
    inp = W.make_tiny_dispatch(rng, R=2000, G=60, M=2, NS=3, NF=4, S=2)
    inp["lut"]["p0_w"] = float(np.float32(2.0))
    inp["avail"]["k_dyn_w"] = (-rng.uniform(0.0, 500.0, 60)).astype(np.float32)
    got = parity(inp, label="negative energies")
    assert np.any(got[4][got[3] == 1] < 0)


# ------------------------------------------------------------------ wave by wave
def run_waves(inp, ws, dd=None):
    from paper_2606_30391_amd import festina as F
    F.lib()
    dd = dd or F.DeviceDispatch(inp, "cuda")
    dd.run_waves(ws)
    torch.cuda.synchronize()
    return dd.results(), dd.state_results(), dd


def wave_parity(inp, ws, label="", dd=None):
    ws = np.asarray(ws, np.int32)
    say(f"[gpu] wave dispatch {label}: R={inp['requests']['n_requests']} G={inp['avail']['n_gpus']} "
        f"S={inp['avail']['n_steps']} waves={len(ws) - 1}")
    got, st, dd = run_waves(inp, ws, dd)
    ref, ref_st = oracle.dispatch_waves(inp, ws)
    rep = check_dispatch(ref, got)
    say(f"      {rep}; phases {np.bincount(got[3], minlength=4).tolist()}")
    assert rep.ok, str(rep)
    for k, v in ref_st.items():
        assert np.array_equal(st[k], v), k
    return got, st, dd


def test_wave_dispatch_worked_example():
    from test_oracle_dispatch_waves_pins import worked_example
    inp, ws, exp = worked_example()
    (g, k, j, ph, e), st, _ = run_waves(inp, ws)
    assert (g.tolist(), k.tolist(), j.tolist(), ph.tolist()) == (exp["gpu"], exp["freq_level"], exp["sm_level"],
                                                                  exp["phase"])
    assert e.tolist() == [float(np.float32(x)) for x in exp["energy"]]
    for key, v in exp["state"].items():
        assert st[key].tolist() == v, key


def test_wave_dispatch_workload_full_size():
    inp = W.make_dispatch_waves()
    got, st, _ = wave_parity(inp, inp["wave_start"], label="65536 requests, 512 GPUs, 64 waves")
    ph = np.bincount(got[3], minlength=4)
    assert ph[1] > 0 and ph[2] > 0 and ph[3] > 0
    assert (st["batch"] >= inp["avail"]["batch"]).all() and (st["batch"] > inp["avail"]["batch"]).any()


def test_wave_dispatch_configuration_4_shape():
    """Configuration 4's arrival structure: 262,144 requests in 64 waves of 4,096, 1,024 GPUs."""
    inp = W.make_dispatch_waves(n_requests=262144, n_gpus=1024, n_waves=64)
    got, st, _ = wave_parity(inp, inp["wave_start"], label="262144 requests, 1024 GPUs, 64 waves")
    ph = np.bincount(got[3], minlength=4)
    assert ph[1] > 0 and ph[2] > 0 and ph[3] > 0 and ph[0] > 0


@pytest.mark.parametrize("n_waves", [1, 7, 300])
def test_wave_dispatch_workload_seeds(n_waves):
    inp = W.make_dispatch_waves(seed=W.DISPATCH_SEED + 300, n_requests=6000, n_gpus=256, n_waves=n_waves)
    wave_parity(inp, inp["wave_start"], label=f"{n_waves} waves")


@pytest.mark.parametrize("NS,NF,S", [(1, 1, 1), (3, 5, 2), (4, 8, 3), (8, 16, 9), (2, 70, 1)])
def test_wave_dispatch_shapes_and_empty_waves(NS, NF, S):
    rng = np.random.default_rng(1700 + NS * 100 + NF)
    inp = W.make_tiny_dispatch(rng, R=2000, G=60, M=3, NS=NS, NF=NF, S=S)
    cuts = np.sort(rng.integers(0, 2001, 40))
    cuts[:3] = cuts[3]                                   # empty waves
    wave_parity(inp, [0, *cuts.tolist(), 2000], label="shapes")


def test_wave_dispatch_ties_and_one_request_per_wave():
    rng = np.random.default_rng(1800)
    inp = W.make_tiny_dispatch(rng, R=300, G=12, M=2, NS=3, NF=4, S=2, ties=True)
    wave_parity(inp, np.arange(301), label="ties, one request per wave")
    inp["avail"]["k_dyn_w"][:] = 0.0
    wave_parity(inp, [0, 150, 300], label="exact ties, two waves")


def test_wave_dispatch_repeated_calls_and_no_requests():
    """Pending commits never leak from one call into the next; no requests: the state is the
    caller's, copied."""
    rng = np.random.default_rng(1900)
    inp = W.make_tiny_dispatch(rng, R=1500, G=40, M=3, NS=4, NF=6, S=3)
    _, _, dd = wave_parity(inp, [0, 500, 1000, 1500], label="first call")
    wave_parity(inp, [0, 1500], label="second call, one wave", dd=dd)
    wave_parity(inp, W.wave_bounds(1500, 11), label="third call, 11 waves", dd=dd)
    empty = W.make_tiny_dispatch(rng, R=0, G=9, M=2, NS=2, NF=3, S=2)
    for ws in ([0], [0, 0, 0]):
        _, st, _ = run_waves(empty, ws)
        for k in ("freq_cur", "batch", "mem_free_mib"):
            assert np.array_equal(st[k], empty["avail"][k]), k


def test_wave_dispatch_state_in_place():
    """The carried state may be the caller's own arrays: they then end as the final state."""
    from paper_2606_30391_amd import festina as F
    rng = np.random.default_rng(2000)
    inp = W.make_tiny_dispatch(rng, R=1200, G=30, M=2, NS=4, NF=5, S=2)
    ws = W.wave_bounds(1200, 9)
    ref, ref_st = oracle.dispatch_waves(inp, ws)
    dd = F.DeviceDispatch(inp, "cuda")
    state = F.festina_gpu_state(*(F._ptr(dd.t[k]) for k in ("freq_cur", "batch", "mem_free_mib")))
    nbytes = F.festina_dispatch_waves_workspace_bytes(dd.lut, dd.avail)
    wsp = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    F.festina_dispatch_waves(dd.lut, dd.avail, dd.req, ws, state, dd.out, wsp, nbytes)
    torch.cuda.synchronize()
    rep = check_dispatch(ref, dd.results())
    assert rep.ok, str(rep)
    G, S = inp["avail"]["n_gpus"], inp["avail"]["n_steps"]
    assert np.array_equal(dd.t["freq_cur"].cpu().numpy(), ref_st["freq_cur"])
    assert np.array_equal(dd.t["batch"].cpu().numpy(), ref_st["batch"])
    assert np.array_equal(dd.t["mem_free_mib"].cpu().numpy().reshape(G, S), ref_st["mem_free_mib"])


def test_wave_dispatch_invalid_elements_and_many_hosts():
    rng = np.random.default_rng(2100)
    inp = W.make_tiny_dispatch(rng, R=600, G=40, M=3, NS=4, NF=6, S=3)
    rq, av = inp["requests"], inp["avail"]
    rq["model"][:20] = 3
    rq["model"][20:30] = -1
    rq["prompt_tokens"][30:40] = -5
    rq["pred_out_tokens"][40:50] = -1
    av["batch"][:5] = -1
    av["freq_cur"][5:10] = 9
    av["sm_free"][10:15] = 7
    av["sm_free"][15:20] = -1
    got, st, _ = wave_parity(inp, W.wave_bounds(600, 6), label="invalid elements")
    assert np.all(got[3][:50] == 0) and np.array_equal(st["batch"][:5], av["batch"][:5])
    # more hosts per model than 64 lanes x 4 cached hosts: the second pass over the rest
    wave_parity(W.make_tiny_dispatch(rng, R=700, G=700, M=2, NS=4, NF=6, S=2), W.wave_bounds(700, 5),
                label="700 GPUs")


def test_wave_dispatch_waves_of_16_lanes_per_request():
    """Waves above 8,192 requests take the 16-lanes-per-request kernel."""
    inp = W.make_dispatch_waves(seed=W.DISPATCH_SEED + 400, n_requests=20000, n_gpus=256, n_waves=2)
    wave_parity(inp, inp["wave_start"], label="two waves of 10000")
