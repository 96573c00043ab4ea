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
    assert F.festina_abi_version() == 1
    for s in range(4):
        assert F.festina_status_string(s)
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
                         ("n_tasks", None), ("util", None)]:
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
