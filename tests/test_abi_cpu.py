"""C-ABI checks that need no GPU: the library loads, exports every function that
include/festina.h declares, sizes workspaces, and rejects bad arguments before
launching anything."""
import ctypes as C
import os
import re

import numpy as np
import pytest

from paper_2606_30391_amd import festina as F

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "festina.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(festina_[a-z_]+)\s*\(", text)
    return sorted(set(names))


def _no_gpu_visible():
    import torch
    return torch.cuda.device_count() == 0


# The error-path calls below pass fake device pointers that must never be launched on;
# they run only where no GPU is visible, so a validation regression cannot fault a device.
no_gpu = pytest.mark.skipif(not _no_gpu_visible(), reason="fake-pointer error paths run only without a GPU")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(F.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return F.lib()


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert set(names) >= set(F.EXPORTED)
    for n in names:
        assert hasattr(lib, n), n


def test_version_and_status_strings(lib):
    assert F.festina_abi_version() == 4
    for s in range(5):
        assert F.festina_status_string(s)
    assert "scratch" in F.festina_status_string(F.FESTINA_ERR_TOO_LARGE)
    assert "unknown" in F.festina_status_string(99)


def _structs(M=2, NS=4, NF=8, G=8, W=1, R=64):
    fake = C.c_void_p(0x1000)       # never dereferenced: the calls below fail validation first
    lut = F.festina_lut(M, 32, NS, NF, fake, fake, fake, fake, 120.0)
    gpus = F.festina_gpus(G, W, fake, fake, fake, None, None)
    req = F.festina_requests(R, fake, None, fake, fake, fake, fake)
    out = F.festina_placements(fake, fake, fake)
    return lut, gpus, req, out


def test_placement_workspace_grows_with_shapes(lib):
    lut, gpus, req, _ = _structs()
    small = F.festina_placements_workspace_bytes(lut, gpus, req)
    lut2, gpus2, req2, _ = _structs(M=32, NS=8, NF=16, G=1024, W=64, R=262144)
    big = F.festina_placements_workspace_bytes(lut2, gpus2, req2)
    assert 0 < small < big
    assert big % 256 == 0
    lut.n_rows = 31
    assert F.festina_placements_workspace_bytes(lut, gpus, req) == 0


def _call(lut, gpus, req, out, ws, nbytes):
    return lib_().festina_score_placements(C.byref(lut), C.byref(gpus), C.byref(req), C.byref(out),
                                           ws, nbytes, None)


def lib_():
    return F.lib()


@no_gpu
def test_placement_rejects_bad_arguments_before_launch(lib):
    lut, gpus, req, out = _structs()
    need = F.festina_placements_workspace_bytes(lut, gpus, req)
    ws = C.c_void_p(0x100000)                                 # 256-aligned, never touched
    assert _call(lut, gpus, req, out, None, need) == F.FESTINA_ERR_INVALID
    assert _call(lut, gpus, req, out, ws, need - 1) == F.FESTINA_ERR_INVALID
    assert _call(lut, gpus, req, out, C.c_void_p(0x100004), need) == F.FESTINA_ERR_INVALID
    bad = [("n_rows", 16), ("n_models", 0), ("n_sm", 0), ("n_freq", -1)]
    for field, v in bad:
        l2, g2, r2, o2 = _structs()
        setattr(l2, field, v)
        assert _call(l2, g2, r2, o2, ws, 1 << 30) == F.FESTINA_ERR_INVALID, field
    l2, g2, r2, o2 = _structs(NS=16, NF=17)                   # 272 cells
    assert _call(l2, g2, r2, o2, ws, 1 << 30) == F.FESTINA_ERR_UNSUPPORTED
    l2, g2, r2, o2 = _structs()
    g2.n_gpus = 0
    assert _call(l2, g2, r2, o2, ws, 1 << 30) == F.FESTINA_ERR_INVALID
    l2, g2, r2, o2 = _structs()
    r2.model = None
    assert _call(l2, g2, r2, o2, ws, 1 << 30) == F.FESTINA_ERR_INVALID
    l2, g2, r2, o2 = _structs()
    o2.energy_mj = None
    assert _call(l2, g2, r2, o2, ws, 1 << 30) == F.FESTINA_ERR_INVALID
    l2, g2, r2, o2 = _structs()
    l2.pf = None
    assert _call(l2, g2, r2, o2, ws, 1 << 30) == F.FESTINA_ERR_INVALID
    assert lib.festina_score_placements(None, C.byref(gpus), C.byref(req), C.byref(out), ws, need,
                                        None) == F.FESTINA_ERR_INVALID


@no_gpu
def test_placement_zero_requests_is_a_no_op(lib):
    lut, gpus, req, out = _structs(R=0)
    need = F.festina_placements_workspace_bytes(lut, gpus, req)
    assert need > 0
    assert _call(lut, gpus, req, out, None, 0) == F.FESTINA_OK


@no_gpu
def test_migration_rejects_bad_arguments_before_launch(lib):
    fake = C.c_void_p(0x1000)
    lut = F.festina_lut(32, 32, 8, 16, fake, fake, fake, fake, 120.0)
    fl = F.festina_fleet(2048, 4, *([fake] * 11), 294912, 1000)
    out = F.festina_migrations(fake, fake, fake)
    need = F.festina_migrations_workspace_bytes(lut, fl)
    assert need >= 2048 * 8
    ws = C.c_void_p(0x100000)
    call = lambda l, f, o, w, n: lib.festina_score_migrations(C.byref(l), C.byref(f), C.byref(o), w, n, None)
    assert call(lut, fl, out, ws, need - 1) == F.FESTINA_ERR_INVALID
    lut.n_freq = 33
    assert call(lut, fl, out, ws, 1 << 30) == F.FESTINA_ERR_UNSUPPORTED
    lut.n_freq = 16
    fl.n_gpus = 1
    assert call(lut, fl, out, ws, 1 << 30) == F.FESTINA_ERR_INVALID
    fl.n_gpus = 2048
    fl.util = None
    assert call(lut, fl, out, ws, 1 << 30) == F.FESTINA_ERR_INVALID


def test_product_binding_does_not_touch_the_oracle():
    import paper_2606_30391_amd.festina as mod
    src = open(mod.__file__).read()
    assert "oracle" not in src.replace("no CPU fallback", "")
    hip = open(os.path.join(ROOT, "paper_2606_30391_amd", "csrc", "festina.hip")).read()
    assert "oracle" not in hip


def _sweep_structs(M=2, NS=4, NF=8, B=16, T=4):
    fake = C.c_void_p(0x1000)       # never dereferenced: the calls below fail validation first
    lut = F.festina_lut(M, 32, NS, NF, fake, fake, fake, fake, 120.0)
    bat = F.festina_batches(B, T, fake, fake, fake, fake, fake, fake, fake, fake, 1000)
    out = F.festina_sweep_result(fake, fake, fake, fake)
    return lut, bat, out


def _sweep_status(lut, bat, out):
    return F.lib().festina_sweep_batches(C.byref(lut), C.byref(bat), C.byref(out), None)


@no_gpu
def test_sweep_rejects_bad_arguments(lib):
    lut, bat, out = _sweep_structs()
    L = F.lib()
    assert L.festina_sweep_batches(None, C.byref(bat), C.byref(out), None) == F.FESTINA_ERR_INVALID
    assert L.festina_sweep_batches(C.byref(lut), None, C.byref(out), None) == F.FESTINA_ERR_INVALID
    assert L.festina_sweep_batches(C.byref(lut), C.byref(bat), None, None) == F.FESTINA_ERR_INVALID
    for field, value, status in [("n_rows", 31, F.FESTINA_ERR_INVALID), ("n_sm", 0, F.FESTINA_ERR_INVALID),
                                 ("n_freq", 0, F.FESTINA_ERR_INVALID), ("n_models", 0, F.FESTINA_ERR_INVALID),
                                 ("n_freq", 65, F.FESTINA_ERR_UNSUPPORTED),
                                 ("n_sm", 257, F.FESTINA_ERR_UNSUPPORTED), ("pf", None, F.FESTINA_ERR_INVALID)]:
        lut, bat, out = _sweep_structs()
        setattr(lut, field, value)
        assert _sweep_status(lut, bat, out) == status, field
    for field, value in [("n_batches", -1), ("max_tasks", 0), ("sm_units", None), ("task_slack_ms", None),
                         ("n_tasks", None), ("util", None), ("static_power", 2), ("static_power", -1)]:
        lut, bat, out = _sweep_structs()
        setattr(bat, field, value)
        assert _sweep_status(lut, bat, out) == F.FESTINA_ERR_INVALID, field
    for field in ("freq_level", "feasible", "energy_mj", "task_sm"):
        lut, bat, out = _sweep_structs()
        setattr(out, field, None)
        assert _sweep_status(lut, bat, out) == F.FESTINA_ERR_INVALID, field
    # no batches: nothing to do, nothing launched, outputs untouched
    lut, bat, out = _sweep_structs(B=0)
    bat.n_tasks = None
    out.task_sm = None
    assert _sweep_status(lut, bat, out) == F.FESTINA_OK


@no_gpu
def test_preferred_and_ewr_reject_bad_arguments(lib):
    fake = C.c_void_p(0x1000)
    L = F.lib()

    def structs(NS=4, NF=8, G=4, K=2):
        lut = F.festina_lut(2, 32, NS, NF, fake, fake, fake, fake, 120.0)
        q = F.festina_llms(G, K, *([fake] * 8))
        out = F.festina_preferred(*([fake] * 12))
        return lut, q, out

    call = lambda lut, q, out: L.festina_preferred_configs(C.byref(lut), C.byref(q), C.byref(out), None)
    lut, q, out = structs()
    assert L.festina_preferred_configs(None, C.byref(q), C.byref(out), None) == F.FESTINA_ERR_INVALID
    assert L.festina_preferred_configs(C.byref(lut), None, C.byref(out), None) == F.FESTINA_ERR_INVALID
    assert call(*structs(NS=16, NF=17)) == F.FESTINA_ERR_UNSUPPORTED
    for field in ("n_inst", "avg_out_tokens", "k_dyn_w"):
        lut, q, out = structs()
        setattr(q, field, None)
        assert call(lut, q, out) == F.FESTINA_ERR_INVALID, field
    for field in ("sm_p", "t_ms", "f_pref", "feasible"):
        lut, q, out = structs()
        setattr(out, field, None)
        assert call(lut, q, out) == F.FESTINA_ERR_INVALID, field
    lut, q, out = structs()
    q.max_inst = 0
    assert call(lut, q, out) == F.FESTINA_ERR_INVALID
    lut, q, out = structs(G=0)
    q.n_inst = None
    assert call(lut, q, out) == F.FESTINA_OK

    assert F.festina_ewr_workspace_bytes(0) == 0
    assert F.festina_ewr_workspace_bytes(1) == 256 and F.festina_ewr_workspace_bytes(257) == 256
    assert F.festina_ewr_workspace_bytes(256 * 17) == 512
    ewr = F.festina_ewr(fake, fake, fake)
    ws = C.c_void_p(0x100000)
    ecall = lambda G, K, n, out, w, nb: L.festina_fleet_ewr(G, K, n, fake, fake, C.byref(out) if out else None,
                                                            w, nb, None)
    assert ecall(0, 4, fake, ewr, ws, 256) == F.FESTINA_ERR_INVALID
    assert ecall(8, 0, fake, ewr, ws, 256) == F.FESTINA_ERR_INVALID
    assert ecall(8, 4, None, ewr, ws, 256) == F.FESTINA_ERR_INVALID
    assert ecall(8, 4, fake, None, ws, 256) == F.FESTINA_ERR_INVALID
    assert ecall(8, 4, fake, ewr, ws, 255) == F.FESTINA_ERR_INVALID
    assert ecall(8, 4, fake, ewr, C.c_void_p(0x100010), 256) == F.FESTINA_ERR_INVALID
    assert ecall(8, 4, fake, ewr, None, 256) == F.FESTINA_ERR_INVALID


@no_gpu
def test_dispatch_rejects_bad_arguments(lib):
    fake = C.c_void_p(0x1000)
    L = F.lib()

    def structs(NS=8, NF=16, G=64, S=4, R=512):
        lut = F.festina_lut(32, 32, NS, NF, fake, fake, fake, fake, 120.0)
        av = F.festina_gpu_avail(G, S, *([fake] * 8), 400.0)
        req = F.festina_requests(R, fake, None, fake, fake, fake, fake)
        out = F.festina_dispatches(*([fake] * 5))
        return lut, av, req, out

    def call(lut, av, req, out, ws, nbytes):
        return L.festina_dispatch_requests(C.byref(lut), C.byref(av), C.byref(req), C.byref(out), ws, nbytes, None)

    lut, av, req, out = structs()
    need = F.festina_dispatch_workspace_bytes(lut, av)
    assert need > 0 and need % 256 == 0
    ws = C.c_void_p(0x100000)
    assert L.festina_dispatch_requests(None, C.byref(av), C.byref(req), C.byref(out), ws, need, None) == \
        F.FESTINA_ERR_INVALID
    assert L.festina_dispatch_requests(C.byref(lut), None, C.byref(req), C.byref(out), ws, need, None) == \
        F.FESTINA_ERR_INVALID
    assert L.festina_dispatch_requests(C.byref(lut), C.byref(av), None, C.byref(out), ws, need, None) == \
        F.FESTINA_ERR_INVALID
    assert call(lut, av, req, out, None, need) == F.FESTINA_ERR_INVALID
    assert call(lut, av, req, out, ws, need - 1) == F.FESTINA_ERR_INVALID
    assert call(lut, av, req, out, C.c_void_p(0x100008), need) == F.FESTINA_ERR_INVALID
    assert call(*structs(NS=16, NF=17), ws, 1 << 30) == F.FESTINA_ERR_UNSUPPORTED
    for obj, field, value in [("lut", "n_rows", 31), ("lut", "n_models", 0), ("lut", "pf", None),
                              ("av", "n_gpus", 0), ("av", "n_gpus", 1 << 24), ("av", "n_steps", 0),
                              ("av", "sm_free", None), ("av", "kv_kib_per_token", None),
                              ("req", "n_requests", -1), ("req", "slo_tbt_ms", None),
                              ("out", "phase", None), ("out", "energy_mj", None)]:
        s = dict(zip(("lut", "av", "req", "out"), structs()))
        setattr(s[obj], field, value)
        assert call(s["lut"], s["av"], s["req"], s["out"], ws, 1 << 30) == F.FESTINA_ERR_INVALID, (obj, field)
    assert F.festina_dispatch_workspace_bytes(*structs()[:1], F.festina_gpu_avail(0, 4, *([fake] * 8), 1.0)) == 0
    # no requests: nothing launched, outputs untouched
    lut, av, req, out = structs(R=0)
    req.model = None
    out.gpu = None
    assert call(lut, av, req, out, ws, need) == F.FESTINA_OK


@no_gpu
def test_dispatch_waves_rejects_bad_arguments(lib):
    fake = C.c_void_p(0x1000)
    L = F.lib()
    R = 512

    def structs(NS=8, NF=16, G=64, S=4):
        lut = F.festina_lut(32, 32, NS, NF, fake, fake, fake, fake, 120.0)
        av = F.festina_gpu_avail(G, S, *([fake] * 8), 400.0)
        req = F.festina_requests(R, fake, None, fake, fake, fake, fake)
        out = F.festina_dispatches(*([fake] * 5))
        state = F.festina_gpu_state(fake, fake, fake)
        return lut, av, req, out, state

    def call(lut, av, req, out, state, bounds, ws, nbytes):
        b = np.ascontiguousarray(bounds, np.int32)
        return L.festina_dispatch_waves(C.byref(lut), C.byref(av), C.byref(req), b.size - 1,
                                        b.ctypes.data if b.size else None, None if state is None else C.byref(state),
                                        C.byref(out), ws, nbytes, None)

    lut, av, req, out, state = structs()
    need = F.festina_dispatch_waves_workspace_bytes(lut, av)
    assert need > 0 and need % 256 == 0
    ws = C.c_void_p(0x100000)
    good = [0, 100, 100, 512]
    assert call(lut, av, req, out, None, good, ws, need) == F.FESTINA_ERR_INVALID
    for bad in ([0, 511], [1, 512], [0, 300, 200, 512], [0, 513], [], [0]):
        assert call(lut, av, req, out, state, bad, ws, need) == F.FESTINA_ERR_INVALID, bad
    assert L.festina_dispatch_waves(C.byref(lut), C.byref(av), C.byref(req), 2, None, C.byref(state), C.byref(out),
                                    ws, need, None) == F.FESTINA_ERR_INVALID
    assert call(lut, av, req, out, state, good, None, need) == F.FESTINA_ERR_INVALID
    assert call(lut, av, req, out, state, good, ws, need - 1) == F.FESTINA_ERR_INVALID
    assert call(lut, av, req, out, state, good, C.c_void_p(0x100008), need) == F.FESTINA_ERR_INVALID
    assert call(*structs(NS=16, NF=17), good, ws, 1 << 30) == F.FESTINA_ERR_UNSUPPORTED
    for obj, field, value in [("state", "freq_cur", None), ("state", "batch", None), ("state", "mem_free_mib", None),
                              ("av", "n_gpus", 0), ("av", "n_steps", 0), ("av", "mem_free_mib", None),
                              ("req", "model", None), ("out", "gpu", None), ("lut", "dc", None)]:
        s = dict(zip(("lut", "av", "req", "out", "state"), structs()))
        setattr(s[obj], field, value)
        assert call(s["lut"], s["av"], s["req"], s["out"], s["state"], good, ws, 1 << 30) == F.FESTINA_ERR_INVALID, \
            (obj, field)
    assert F.festina_dispatch_waves_workspace_bytes(*structs()[:1], F.festina_gpu_avail(0, 4, *([fake] * 8), 1.0)) == 0


@no_gpu
def test_transfer_costs_and_moves_reject_bad_arguments(lib):
    fake = C.c_void_p(0x1000)
    L = F.lib()

    def structs(G=64, M=32, Q=128):
        tr = F.festina_transfer(G, M, fake, fake, fake, fake, 153.6, 50.0)
        lut = F.festina_lut(M, 32, 8, 16, fake, fake, fake, fake, 120.0)
        plan = F.festina_plan(fake, fake, fake, fake)
        req = F.festina_inflight(Q, *([fake] * 6))
        out = F.festina_moves(fake, fake, fake)
        return tr, lut, plan, req, out

    cost = lambda tr, c: L.festina_transfer_costs(C.byref(tr) if tr is not None else None, c, None)
    tr, *_ = structs()
    assert cost(None, fake) == F.FESTINA_ERR_INVALID
    assert cost(tr, None) == F.FESTINA_ERR_INVALID
    for field, value in [("n_gpus", 0), ("n_models", 0), ("resident", None), ("weights_mib", None),
                         ("state_mib", None), ("node", None), ("bw_intra_gbs", 0.0), ("bw_inter_gbs", -1.0),
                         ("bw_intra_gbs", float("nan"))]:
        tr, *_ = structs()
        setattr(tr, field, value)
        assert cost(tr, fake) == F.FESTINA_ERR_INVALID, field
    tr, *_ = structs(G=(1 << 20) + 1)
    assert cost(tr, fake) == F.FESTINA_ERR_UNSUPPORTED          # more than 2^40 matrix entries

    def moves(tr, lut, plan, req, out):
        return L.festina_request_moves(C.byref(lut), C.byref(tr), C.byref(plan), C.byref(req), C.byref(out), None)

    assert L.festina_request_moves(None, *(C.byref(x) for x in structs()[:1]), *(
        C.byref(x) for x in structs()[2:]), None) == F.FESTINA_ERR_INVALID
    for obj, field, value in [("tr", "bw_inter_gbs", 0.0), ("lut", "n_rows", 16), ("lut", "n_sm", 0),
                              ("lut", "dc", None), ("plan", "dest", None), ("plan", "batch", None),
                              ("req", "n_requests", -1), ("req", "kv_kib", None), ("req", "src", None),
                              ("out", "decision", None), ("out", "migrate_ms", None)]:
        s = dict(zip(("tr", "lut", "plan", "req", "out"), structs()))
        setattr(s[obj], field, value)
        assert moves(s["tr"], s["lut"], s["plan"], s["req"], s["out"]) == F.FESTINA_ERR_INVALID, (obj, field)
    s = dict(zip(("tr", "lut", "plan", "req", "out"), structs()))
    s["lut"].n_sm, s["lut"].n_freq = 16, 17
    assert moves(s["tr"], s["lut"], s["plan"], s["req"], s["out"]) == F.FESTINA_ERR_UNSUPPORTED
    # no in-flight requests: nothing launched
    s = dict(zip(("tr", "lut", "plan", "req", "out"), structs(Q=0)))
    s["req"].src = None
    s["out"].decision = None
    assert moves(s["tr"], s["lut"], s["plan"], s["req"], s["out"]) == F.FESTINA_OK


def test_binding_refuses_a_library_built_from_other_sources(tmp_path, monkeypatch):
    """festina.lib() loads the library only while its recorded source hash matches the tree."""
    import paper_2606_30391_amd.build as B
    if not os.path.exists(F.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    F._check_fresh()                                         # the built library matches
    stale = tmp_path / "libfestina.so.sources"
    stale.write_text("0" * 64 + "\n")
    monkeypatch.setattr(B, "HASH_FILE", str(stale))
    with pytest.raises(RuntimeError, match="not built from the sources"):
        F._check_fresh()
    monkeypatch.setattr(B, "HASH_FILE", str(tmp_path / "missing"))
    with pytest.raises(RuntimeError, match="not built from the sources"):
        F._check_fresh()


@no_gpu
def test_noalloc_placement_rejects_bad_arguments_and_oversized_inputs(lib):
    """The allocation-free entry point checks its arguments like festina_score_placements and
    refuses, before any launch, shapes whose workspace exceeds its fixed scratch."""
    L = F.lib()
    call = lambda l, g, r, o: L.festina_score_placements_noalloc(C.byref(l), C.byref(g), C.byref(r),
                                                                 C.byref(o), None)
    lut, gpus, req, out = _structs(M=32, NS=8, NF=16, G=1024, W=64, R=1 << 22)
    assert F.festina_placements_workspace_bytes(lut, gpus, req) > F.FESTINA_NOALLOC_WORKSPACE_BYTES
    assert call(lut, gpus, req, out) == F.FESTINA_ERR_TOO_LARGE
    lut, gpus, req, out = _structs(M=32, NS=8, NF=16, G=1024, W=64, R=262144)
    assert F.festina_placements_workspace_bytes(lut, gpus, req) <= F.FESTINA_NOALLOC_WORKSPACE_BYTES
    assert call(lut, gpus, req, out) == F.FESTINA_ERR_DEVICE          # fits, but there is no device here
    for obj, field, value in [("lut", "n_rows", 16), ("lut", "pf", None), ("gpus", "n_gpus", 0),
                              ("req", "model", None), ("out", "choice", None)]:
        s = dict(zip(("lut", "gpus", "req", "out"), _structs()))
        setattr(s[obj], field, value)
        assert call(s["lut"], s["gpus"], s["req"], s["out"]) == F.FESTINA_ERR_INVALID, (obj, field)
    assert call(*_structs(NS=16, NF=17)) == F.FESTINA_ERR_UNSUPPORTED
    assert L.festina_score_placements_noalloc(None, C.byref(gpus), C.byref(req), C.byref(out), None) == \
        F.FESTINA_ERR_INVALID
    assert call(*_structs(R=0)) == F.FESTINA_OK                           # nothing to do
