"""Every C-ABI call captured in a HIP graph (torch.cuda.CUDAGraph on the call's stream) and
replayed: the calls allocate nothing, synchronise nothing and clear their counters with a
kernel rather than a memset node, so a serving loop can capture them.  Each replay follows
eager work that overwrites the outputs, and must reproduce the eager call's outputs bit for
bit, three times in a row.  (The eager outputs themselves are checked against the oracle
by the parity tests.)"""
import sys

import numpy as np
import pytest

from paper_2606_30391_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

REPLAYS = 3


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _flat(res):
    if isinstance(res, dict):
        return [res[k] for k in sorted(res)]
    return list(res)


def _poison(tensors):
    for t in tensors:
        if t.dtype.is_floating_point:
            t.fill_(float("nan"))
        else:
            t.fill_(-7 if t.dtype != torch.uint8 else 77)


def _replay_matches_eager(run, results, outputs, label):
    """run(): the calls; results(): host copies of the outputs; outputs: device tensors."""
    say(f"[gpu] graph replay: {label}")
    run()
    torch.cuda.synchronize()
    ref = [np.copy(x) for x in _flat(results())]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):               # a warm-up call on the capture stream
        run()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    torch.cuda.synchronize()
    for i in range(REPLAYS):
        _poison(outputs)                        # eager work between the replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = _flat(results())
        assert len(got) == len(ref)
        for a, b in zip(got, ref):
            assert a.dtype == b.dtype and a.shape == b.shape
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"{label}: replay {i} differs"


def test_placement_call_in_a_graph():
    from paper_2606_30391_amd import festina as F
    for cfg in (3, 4):
        d = F.DevicePlacement(W.make_placement(cfg), "cuda")
        _replay_matches_eager(d.run, d.results, [d.choice, d.feasible, d.energy], f"placement config {cfg}")


def test_migration_call_in_a_graph():
    from paper_2606_30391_amd import festina as F
    d = F.DeviceMigration(W.make_fleet(), "cuda")
    _replay_matches_eager(d.run, d.results, [d.best_dst, d.saving, d.level], "migration config 5")


def test_sweep_call_in_a_graph():
    from paper_2606_30391_amd import festina as F
    d = F.DeviceSweep(W.make_sweep(), "cuda")
    _replay_matches_eager(d.run, d.results, [d.level, d.feasible, d.energy, d.task_sm], "sweep")


def test_preferred_and_ewr_calls_in_a_graph():
    from paper_2606_30391_amd import festina as F
    d = F.DevicePreferred(W.make_llms(), "cuda")

    def results():
        r = d.results()
        f, w, t = d.ewr_results()
        return _flat(r) + [f, w, t]

    outs = list(d.o.values()) + [d.f_gpu, d.waste_gpu, d.totals]
    _replay_matches_eager(d.run, results, outs, "preferred configurations + EWR")


def test_dispatch_call_in_a_graph():
    from paper_2606_30391_amd import festina as F
    d = F.DeviceDispatch(W.make_dispatch(), "cuda")
    _replay_matches_eager(d.run, d.results, list(d.o.values()), "dispatcher")


def test_wave_dispatch_call_in_a_graph():
    from paper_2606_30391_amd import festina as F
    inp = W.make_dispatch_waves()
    d = F.DeviceDispatch(inp, "cuda")

    def results():
        return list(d.results()) + _flat(d.state_results())

    d.run_waves(inp["wave_start"])                # sizes the state and workspace before capture
    _replay_matches_eager(lambda: d.run_waves(inp["wave_start"]), results,
                          list(d.o.values()) + list(d.state_t.values()), "dispatcher over 64 waves")


def test_transfer_calls_in_a_graph():
    from paper_2606_30391_amd import festina as F
    d = F.DeviceTransfer(W.make_transfer(), "cuda")

    def run():
        d.run_costs()
        d.run_moves()

    _replay_matches_eager(run, d.results, [d.cost, d.decision, d.remaining, d.migrate], "transfer plan")
