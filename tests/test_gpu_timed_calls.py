"""The timed entry points festina_score_placements_timed / festina_score_migrations_timed:
they record the caller's events around the scoring kernel, their outputs are bit-identical
to the plain calls, the bracketed time is positive and no longer than the whole call, and
a later plain call records nothing (the library keeps no timing state)."""
import os
import sys

import numpy as np
import pytest

from paper_2606_30391_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))


def _check(hip, run, results, label):
    print(f"[gpu] timed call: {label}", flush=True)
    run()
    torch.cuda.synchronize()
    ref = [np.copy(x) for x in results()]
    st = torch.cuda.current_stream().cuda_stream
    ev = [hip.event(), hip.event()]
    whole = [hip.event(), hip.event()]
    try:
        hip.record(whole[0], st)
        run(events=(ev[0], ev[1]))
        hip.record(whole[1], st)
        torch.cuda.synchronize()
        kernel_ms = hip.elapsed_ms(ev[0], ev[1])
        call_ms = hip.elapsed_ms(whole[0], whole[1])
        assert 0.0 < kernel_ms <= call_ms, (kernel_ms, call_ms)
        for a, b in zip(results(), ref):
            assert np.array_equal(np.asarray(a).view(np.uint8), b.view(np.uint8))
        run()                                   # plain call: the events keep their timestamps
        torch.cuda.synchronize()
        assert hip.elapsed_ms(ev[0], ev[1]) == kernel_ms
    finally:
        for e in ev + whole:
            hip.destroy(e)


def test_timed_calls_around_the_scoring_kernels():
    import bench
    from paper_2606_30391_amd import festina as F
    hip = bench.Hip()
    dp = F.DevicePlacement(W.make_placement(3), "cuda")
    _check(hip, dp.run, dp.results, "placement config 3")
    dm = F.DeviceMigration(W.make_fleet(), "cuda")
    _check(hip, dm.run, dm.results, "consolidation config 5")
