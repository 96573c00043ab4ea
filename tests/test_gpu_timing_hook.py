"""The measurement hook festina_set_timing_events: while set, the placement call records
its events around the scoring kernel and the consolidation call around its pair-scoring
kernel, the outputs stay bit-identical to calls without it, the bracketed time is positive
and no longer than the whole call, and once cleared no call records the events again."""
import os
import sys

import numpy as np
import pytest

from paper_2606_30391_amd import workloads as W

torch = pytest.importorskip("torch")
pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))


def _check(hip, F, run, results, which, label):
    print(f"[gpu] timing hook: {label}", flush=True)
    run()
    torch.cuda.synchronize()
    ref = [np.copy(x) for x in results()]
    st = torch.cuda.current_stream().cuda_stream
    ev = [hip.event() for _ in range(4)]
    whole = [hip.event(), hip.event()]
    try:
        args = [None] * 4
        args[2 * which], args[2 * which + 1] = ev[0], ev[1]
        F.festina_set_timing_events(*args)
        hip.record(whole[0], st)
        run()
        hip.record(whole[1], st)
        torch.cuda.synchronize()
        kernel_ms = hip.elapsed_ms(ev[0], ev[1])
        call_ms = hip.elapsed_ms(whole[0], whole[1])
        assert 0.0 < kernel_ms <= call_ms, (kernel_ms, call_ms)
        for a, b in zip(results(), ref):
            assert np.array_equal(np.asarray(a).view(np.uint8), b.view(np.uint8))
        F.festina_set_timing_events()
        run()                                   # cleared: the events keep their timestamps
        torch.cuda.synchronize()
        assert hip.elapsed_ms(ev[0], ev[1]) == kernel_ms
    finally:
        F.festina_set_timing_events()
        for e in ev + whole:
            hip.destroy(e)


def test_timing_hook_around_the_scoring_kernels():
    import bench
    from paper_2606_30391_amd import festina as F
    hip = bench.Hip()
    dp = F.DevicePlacement(W.make_placement(3), "cuda")
    _check(hip, F, dp.run, dp.results, 0, "placement config 3")
    dm = F.DeviceMigration(W.make_fleet(), "cuda")
    _check(hip, F, dm.run, dm.results, 1, "consolidation config 5")
