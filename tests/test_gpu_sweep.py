"""GPU parity of the local SM/frequency sweep: the HIP path through the C ABI against
the CPU oracle.

Flags, levels and per-task SM levels must match exactly (a different level only as a
near-tie judged by the oracle's float64 energies) and energies within 1e-5 relative
(oracle/check.py).  Covers the sweep workload at full size and extra seeds, the worked
example, many table shapes (1..64 frequency levels, up to 16 SM levels), wide batches
(up to 40 task slots), NaN/inf tables, exact ties, invalid tasks and empty batches.
"""
import sys

import numpy as np
import pytest

import oracle
from conftest import golden_sweep
from oracle.check import check_sweep
from paper_2606_30391_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_sweep(inp, stream=None):
    from paper_2606_30391_amd import festina as F
    F.lib()
    ds = F.DeviceSweep(inp, "cuda")
    ds.run(stream)
    torch.cuda.synchronize()
    return ds.results()


def parity_sweep(inp, sel=None, label=""):
    bt = inp["batches"]
    B = bt["n_batches"]
    say(f"[gpu] sweep {label}: B={B} T={bt['max_tasks']} NS={inp['lut']['n_sm']} NF={inp['lut']['n_freq']}")
    got = run_sweep(inp)
    sel = np.arange(B) if sel is None else np.asarray(sel)
    ref = oracle.sweep(inp, sel)
    rep = check_sweep(inp, sel, ref, tuple(x[sel] for x in got))
    say(f"      {rep}")
    assert rep.ok, str(rep)
    return got, rep


def test_sweep_workload_full_size():
    inp = W.make_sweep()
    got, rep = parity_sweep(inp, label="1024 GPUs x 64 epochs")
    fe = got[1]
    assert 0.3 < fe.mean() < 0.8


def test_sweep_workload_static_power_per_batch():
    inp = W.make_sweep(n_gpus=512, n_epochs=32)
    inp["batches"]["static_power"] = 1
    got, rep = parity_sweep(inp, label="static power per batch, 512 GPUs x 32 epochs")


@pytest.mark.parametrize("NS,NF,T", [(4, 8, 7), (8, 16, 16), (3, 5, 40)])
def test_sweep_static_power_per_batch_shapes(NS, NF, T):
    rng = np.random.default_rng(900 + NS * 100 + NF)
    inp = W.make_tiny_sweep(rng, B=517, T=T, M=3, NS=NS, NF=NF, nan_cells=True)
    inp["batches"]["static_power"] = 1
    parity_sweep(inp, label=f"static power per batch NS={NS} NF={NF} T={T}")


@pytest.mark.parametrize("extra", [100, 200, 300])
def test_sweep_workload_seeds(extra):
    parity_sweep(W.make_sweep(seed=W.SWEEP_SEED + extra, n_gpus=256, n_epochs=16), label=f"seed +{extra}")


@pytest.mark.parametrize("variant", [None, "static power dominates", "budget reached exactly",
                                     "budget one unit above", "slack equal to a latency",
                                     "static power per batch", "static power per task, P0 = 640",
                                     "static power per batch, P0 = 640"])
def test_sweep_worked_example(variant):
    inp, exp, d = golden_sweep(variant)
    lev, fe, en, tsm = run_sweep(inp)
    assert lev[0] == exp["freq_level"] and fe[0] == exp["feasible"]
    assert list(tsm[0]) == exp["task_sm"]
    if exp["energy_mj"] is None:
        assert en[0] == np.inf
    else:
        assert en[0] == np.float32(exp["energy_mj"])


@pytest.mark.parametrize("NS,NF", [(1, 1), (3, 5), (4, 8), (8, 16), (16, 16), (2, 33), (4, 64), (8, 17)])
def test_sweep_table_shapes(NS, NF):
    rng = np.random.default_rng(800 + NS * 100 + NF)
    inp = W.make_tiny_sweep(rng, B=517, T=7, M=3, NS=NS, NF=NF, nan_cells=True)
    parity_sweep(inp, label="tiny shapes")


@pytest.mark.parametrize("T", [1, 8, 16, 17, 40])
def test_sweep_task_slots(T):
    rng = np.random.default_rng(900 + T)
    inp = W.make_tiny_sweep(rng, B=300, T=T, M=4, NS=8, NF=16)
    inp["batches"]["sm_budget"] = 10 ** 6
    parity_sweep(inp, label=f"{T} task slots")


@pytest.mark.parametrize("NS,NF", [(4, 12), (8, 16)])
def test_sweep_exact_ties_take_lowest_level(NS, NF):
    rng = np.random.default_rng(950 + NF)
    inp = W.make_tiny_sweep(rng, B=400, T=4, M=2, NS=NS, NF=NF, zero_power=True)
    got, rep = parity_sweep(inp, label="zero power")
    lev, fe, en, tsm = got
    assert np.all(en[fe == 1] == 0.0)
    ref = oracle.sweep(inp)
    assert np.array_equal(lev, ref[0])


@pytest.mark.parametrize("NS,NF", [(4, 8), (8, 16)])
def test_sweep_invalid_tasks_and_empty_batches(NS, NF):
    rng = np.random.default_rng(951 + NF)
    inp = W.make_tiny_sweep(rng, B=64, T=5, M=3, NS=NS, NF=NF)
    bt = inp["batches"]
    bt["n_tasks"][0] = 0
    bt["n_tasks"][1] = 6              # more than max_tasks
    bt["n_tasks"][2] = -1
    bt["n_tasks"][3:10] = 5
    bt["task_model"][3, 4] = 3        # model out of range
    bt["task_model"][4, 0] = -1
    bt["task_phase"][5, 2] = 7        # unknown phase
    bt["task_tokens"][6, 1] = 0       # no tokens
    bt["task_tokens"][7, 3] = -100
    bt["task_slack_ms"][8, :] = np.nan
    bt["task_slack_ms"][9, :] = np.inf
    got, rep = parity_sweep(inp, label="invalid tasks")
    lev, fe, en, tsm = got
    assert fe[0] == 1 or bt["sm_budget"] <= 0
    assert not fe[1:8].any() and not fe[8]
    assert np.all(tsm[1:9] == -1)


def test_sweep_side_stream_and_repeat():
    inp = W.make_sweep(n_gpus=128, n_epochs=8)
    s = torch.cuda.Stream()
    a = run_sweep(inp, stream=s)
    b = run_sweep(inp)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_sweep_more_batches_than_one_grid_pass():
    """Above 131072 batches the 8x16 kernel's blocks loop over several groups of 16."""
    rng = np.random.default_rng(952)
    inp = W.make_tiny_sweep(rng, B=140_011, T=3, M=3, NS=8, NF=16)
    sel = np.concatenate([np.arange(200), np.random.default_rng(3).choice(140_011, 3000, replace=False),
                          np.arange(140_011 - 200, 140_011)])
    parity_sweep(inp, sel, label="140011 batches")
