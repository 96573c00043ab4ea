"""Thin ctypes binding of the C ABI in include/festina.h.

Argument marshalling only: every step of the search runs in the HIP library
(``libfestina.so`` built from ``csrc/festina.hip``, ``csrc/sweep.hip``,
``csrc/preferred.hip``, ``csrc/dispatch.hip`` and ``csrc/transfer.hip``).  PyTorch provides device
memory and streams.  There is no CPU fallback: if the library is missing this
module raises.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfestina.so")

FESTINA_OK = 0
FESTINA_ERR_INVALID = 1
FESTINA_ERR_DEVICE = 2
FESTINA_ERR_UNSUPPORTED = 3
FESTINA_ERR_TOO_LARGE = 4
FESTINA_NOALLOC_WORKSPACE_BYTES = 32 << 20
FESTINA_STATIC_PER_TASK = 0      # sweep energy readings (festina_batches.static_power)
FESTINA_STATIC_PER_BATCH = 1


class FestinaError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {festina_status_string(status)} (status {status})")
        self.status = status


class festina_lut(C.Structure):
    _fields_ = [("n_models", C.c_int32), ("n_rows", C.c_int32), ("n_sm", C.c_int32),
                ("n_freq", C.c_int32), ("sm_level", C.c_void_p), ("freq_level", C.c_void_p),
                ("pf", C.c_void_p), ("dc", C.c_void_p), ("p0_w", C.c_float)]


class festina_gpus(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("n_waves", C.c_int32), ("batch", C.c_void_p),
                ("k_dyn_w", C.c_void_p), ("resident", C.c_void_p), ("cap_pf", C.c_void_p),
                ("cap_dc", C.c_void_p)]


class festina_requests(C.Structure):
    _fields_ = [("n_requests", C.c_int32), ("model", C.c_void_p), ("wave", C.c_void_p),
                ("prompt_tokens", C.c_void_p), ("pred_out_tokens", C.c_void_p),
                ("slo_ttft_ms", C.c_void_p), ("slo_tbt_ms", C.c_void_p)]


class festina_placements(C.Structure):
    _fields_ = [("choice", C.c_void_p), ("feasible", C.c_void_p), ("energy_mj", C.c_void_p)]


class festina_fleet(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("max_inst", C.c_int32), ("n_inst", C.c_void_p),
                ("inst_model", C.c_void_p), ("inst_prompt_tokens", C.c_void_p),
                ("inst_batch", C.c_void_p), ("inst_sm", C.c_void_p),
                ("inst_slo_ttft_ms", C.c_void_p), ("inst_slo_tbt_ms", C.c_void_p),
                ("hbm_mib", C.c_void_p), ("sm_permille", C.c_void_p), ("util", C.c_void_p),
                ("k_dyn_w", C.c_void_p), ("hbm_cap_mib", C.c_int32), ("sm_cap_permille", C.c_int32)]


class festina_migrations(C.Structure):
    _fields_ = [("best_dst", C.c_void_p), ("saving_w", C.c_void_p), ("freq_level", C.c_void_p)]


class festina_batches(C.Structure):
    _fields_ = [("n_batches", C.c_int32), ("max_tasks", C.c_int32), ("n_tasks", C.c_void_p),
                ("task_model", C.c_void_p), ("task_phase", C.c_void_p), ("task_tokens", C.c_void_p),
                ("task_slack_ms", C.c_void_p), ("k_dyn_w", C.c_void_p), ("util", C.c_void_p),
                ("sm_units", C.c_void_p), ("sm_budget", C.c_int32), ("static_power", C.c_int32)]


class festina_sweep_result(C.Structure):
    _fields_ = [("freq_level", C.c_void_p), ("feasible", C.c_void_p), ("energy_mj", C.c_void_p),
                ("task_sm", C.c_void_p)]


class festina_llms(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("max_inst", C.c_int32), ("n_inst", C.c_void_p),
                ("model", C.c_void_p), ("avg_in_tokens", C.c_void_p), ("avg_out_tokens", C.c_void_p),
                ("batch", C.c_void_p), ("slo_ttft_ms", C.c_void_p), ("slo_tbt_ms", C.c_void_p),
                ("k_dyn_w", C.c_void_p)]


class festina_preferred(C.Structure):
    _fields_ = [("sm_p", C.c_void_p), ("f_p", C.c_void_p), ("sm_d", C.c_void_p), ("f_d", C.c_void_p),
                ("t_p_ms", C.c_void_p), ("t_d_ms", C.c_void_p), ("p_p_w", C.c_void_p), ("p_d_w", C.c_void_p),
                ("t_ms", C.c_void_p), ("sm_pref", C.c_void_p), ("f_pref", C.c_void_p), ("feasible", C.c_void_p)]


class festina_ewr(C.Structure):
    _fields_ = [("f_gpu", C.c_void_p), ("waste_gpu", C.c_void_p), ("totals", C.c_void_p)]


class festina_gpu_avail(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("n_steps", C.c_int32), ("freq_cur", C.c_void_p), ("batch", C.c_void_p),
                ("k_dyn_w", C.c_void_p), ("resident", C.c_void_p), ("t_avail_ms", C.c_void_p),
                ("mem_free_mib", C.c_void_p), ("sm_free", C.c_void_p), ("kv_kib_per_token", C.c_void_p),
                ("k_new_w", C.c_float)]


class festina_dispatches(C.Structure):
    _fields_ = [("gpu", C.c_void_p), ("freq_level", C.c_void_p), ("sm_level", C.c_void_p),
                ("phase", C.c_void_p), ("energy_mj", C.c_void_p)]


class festina_gpu_state(C.Structure):
    _fields_ = [("freq_cur", C.c_void_p), ("batch", C.c_void_p), ("mem_free_mib", C.c_void_p)]


class festina_transfer(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("n_models", C.c_int32), ("resident", C.c_void_p),
                ("weights_mib", C.c_void_p), ("state_mib", C.c_void_p), ("node", C.c_void_p),
                ("bw_intra_gbs", C.c_float), ("bw_inter_gbs", C.c_float)]


class festina_plan(C.Structure):
    _fields_ = [("dest", C.c_void_p), ("freq_cur", C.c_void_p), ("sm_cur", C.c_void_p), ("batch", C.c_void_p)]


class festina_inflight(C.Structure):
    _fields_ = [("n_requests", C.c_int32), ("src", C.c_void_p), ("model", C.c_void_p),
                ("context_tokens", C.c_void_p), ("remaining_tokens", C.c_void_p), ("kv_kib", C.c_void_p),
                ("token_kib", C.c_void_p)]


class festina_moves(C.Structure):
    _fields_ = [("decision", C.c_void_p), ("remaining_ms", C.c_void_p), ("migrate_ms", C.c_void_p)]


EXPORTED = ("festina_abi_version", "festina_status_string", "festina_placements_workspace_bytes",
            "festina_score_placements", "festina_score_placements_noalloc", "festina_migrations_workspace_bytes",
            "festina_score_migrations",
            "festina_sweep_batches", "festina_preferred_configs", "festina_ewr_workspace_bytes",
            "festina_fleet_ewr", "festina_dispatch_workspace_bytes", "festina_dispatch_requests",
            "festina_transfer_costs", "festina_request_moves", "festina_score_placements_timed",
            "festina_score_migrations_timed", "festina_dispatch_waves_workspace_bytes", "festina_dispatch_waves")

_lib = None


def _check_fresh():
    """Raise unless the library was built from the sources now in the tree."""
    from .build import HASH_FILE, source_hash
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"HIP library {LIB_PATH} is not built; run __graft_entry__.build()")
    try:
        with open(HASH_FILE) as f:
            built = f.read().strip()
    except OSError:
        built = ""
    if built != source_hash():
        raise RuntimeError(f"HIP library {LIB_PATH} was not built from the sources in this tree "
                           "(csrc/, include/festina.h or the flags changed); run __graft_entry__.build()")


def lib():
    """Load the built HIP library (raises if it has not been built, or was built from other
    sources than the ones in the tree)."""
    global _lib
    if _lib is None:
        _check_fresh()
        L = C.CDLL(LIB_PATH)
        P = C.POINTER
        L.festina_abi_version.restype = C.c_int32
        L.festina_status_string.argtypes = [C.c_int]
        L.festina_status_string.restype = C.c_char_p
        L.festina_placements_workspace_bytes.argtypes = [P(festina_lut), P(festina_gpus), P(festina_requests)]
        L.festina_placements_workspace_bytes.restype = C.c_size_t
        L.festina_score_placements.argtypes = [P(festina_lut), P(festina_gpus), P(festina_requests),
                                               P(festina_placements), C.c_void_p, C.c_size_t, C.c_void_p]
        L.festina_score_placements.restype = C.c_int
        L.festina_score_placements_noalloc.argtypes = [P(festina_lut), P(festina_gpus), P(festina_requests),
                                                       P(festina_placements), C.c_void_p]
        L.festina_score_placements_noalloc.restype = C.c_int
        L.festina_migrations_workspace_bytes.argtypes = [P(festina_lut), P(festina_fleet)]
        L.festina_migrations_workspace_bytes.restype = C.c_size_t
        L.festina_score_migrations.argtypes = [P(festina_lut), P(festina_fleet), P(festina_migrations),
                                               C.c_void_p, C.c_size_t, C.c_void_p]
        L.festina_score_migrations.restype = C.c_int
        L.festina_sweep_batches.argtypes = [P(festina_lut), P(festina_batches), P(festina_sweep_result),
                                            C.c_void_p]
        L.festina_sweep_batches.restype = C.c_int
        L.festina_preferred_configs.argtypes = [P(festina_lut), P(festina_llms), P(festina_preferred),
                                                C.c_void_p]
        L.festina_preferred_configs.restype = C.c_int
        L.festina_ewr_workspace_bytes.argtypes = [C.c_int32]
        L.festina_ewr_workspace_bytes.restype = C.c_size_t
        L.festina_fleet_ewr.argtypes = [C.c_int32, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p,
                                        P(festina_ewr), C.c_void_p, C.c_size_t, C.c_void_p]
        L.festina_fleet_ewr.restype = C.c_int
        L.festina_dispatch_workspace_bytes.argtypes = [P(festina_lut), P(festina_gpu_avail)]
        L.festina_dispatch_workspace_bytes.restype = C.c_size_t
        L.festina_dispatch_requests.argtypes = [P(festina_lut), P(festina_gpu_avail), P(festina_requests),
                                                P(festina_dispatches), C.c_void_p, C.c_size_t, C.c_void_p]
        L.festina_dispatch_requests.restype = C.c_int
        L.festina_dispatch_waves_workspace_bytes.argtypes = [P(festina_lut), P(festina_gpu_avail)]
        L.festina_dispatch_waves_workspace_bytes.restype = C.c_size_t
        L.festina_dispatch_waves.argtypes = [P(festina_lut), P(festina_gpu_avail), P(festina_requests), C.c_int32,
                                             C.c_void_p, P(festina_gpu_state), P(festina_dispatches), C.c_void_p,
                                             C.c_size_t, C.c_void_p]
        L.festina_dispatch_waves.restype = C.c_int
        L.festina_transfer_costs.argtypes = [P(festina_transfer), C.c_void_p, C.c_void_p]
        L.festina_transfer_costs.restype = C.c_int
        L.festina_request_moves.argtypes = [P(festina_lut), P(festina_transfer), P(festina_plan),
                                            P(festina_inflight), P(festina_moves), C.c_void_p]
        L.festina_request_moves.restype = C.c_int
        L.festina_score_placements_timed.argtypes = L.festina_score_placements.argtypes + [C.c_void_p, C.c_void_p]
        L.festina_score_placements_timed.restype = C.c_int
        L.festina_score_migrations_timed.argtypes = L.festina_score_migrations.argtypes + [C.c_void_p, C.c_void_p]
        L.festina_score_migrations_timed.restype = C.c_int
        _lib = L
    return _lib



def festina_abi_version() -> int:
    return int(lib().festina_abi_version())


def festina_status_string(status: int) -> str:
    return lib().festina_status_string(int(status)).decode()


# ------------------------------------------------------------------ device marshalling
def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream_handle(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(stream.cuda_stream)


def _dev(a, dtype, device):
    import torch
    if a is None:
        return None
    return torch.from_numpy(np.ascontiguousarray(a, dtype=dtype)).to(device)


class DevicePlacement:
    """Placement inputs copied to device memory once, with the ABI structs pointing at them."""

    def __init__(self, inp: dict, device="cuda"):
        import torch
        lut, gp, rq = inp["lut"], inp["gpus"], inp["requests"]
        d = lambda a, t: _dev(a, t, device)
        self.t = {
            "sm_level": d(lut["sm_level"], np.float32), "freq_level": d(lut["freq_level"], np.float32),
            "pf": d(lut["pf"], np.float32), "dc": d(lut["dc"], np.float32),
            "batch": d(gp["batch"], np.int32), "k_dyn_w": d(gp["k_dyn_w"], np.float32),
            "resident": d(np.asarray(gp["resident"], np.uint32).view(np.int32), np.int32),
            "cap_pf": d(gp.get("cap_pf"), np.int8), "cap_dc": d(gp.get("cap_dc"), np.int8),
            "model": d(rq["model"], np.int32), "wave": d(rq.get("wave"), np.int32),
            "prompt_tokens": d(rq["prompt_tokens"], np.int32),
            "pred_out_tokens": d(rq["pred_out_tokens"], np.int32),
            "slo_ttft_ms": d(rq["slo_ttft_ms"], np.float32), "slo_tbt_ms": d(rq["slo_tbt_ms"], np.float32),
        }
        t = self.t
        self.lut = festina_lut(int(lut["n_models"]), int(lut["n_rows"]), int(lut["n_sm"]), int(lut["n_freq"]),
                               _ptr(t["sm_level"]), _ptr(t["freq_level"]), _ptr(t["pf"]), _ptr(t["dc"]),
                               float(lut["p0_w"]))
        self.gpus = festina_gpus(int(gp["n_gpus"]), int(gp["n_waves"]), _ptr(t["batch"]), _ptr(t["k_dyn_w"]),
                                 _ptr(t["resident"]), _ptr(t["cap_pf"]), _ptr(t["cap_dc"]))
        self.R = int(rq["n_requests"])
        self.req = festina_requests(self.R, _ptr(t["model"]), _ptr(t["wave"]), _ptr(t["prompt_tokens"]),
                                    _ptr(t["pred_out_tokens"]), _ptr(t["slo_ttft_ms"]), _ptr(t["slo_tbt_ms"]))
        n = max(self.R, 1)
        self.choice = torch.empty(n, dtype=torch.int32, device=device)
        self.feasible = torch.empty(n, dtype=torch.uint8, device=device)
        self.energy = torch.empty(n, dtype=torch.float32, device=device)
        self.out = festina_placements(_ptr(self.choice), _ptr(self.feasible), _ptr(self.energy))
        self.ws_bytes = festina_placements_workspace_bytes(self.lut, self.gpus, self.req)
        self.workspace = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=device)

    def run(self, stream=None, events=None):
        """One search; `events` = (begin, end) raw hipEvent_t handles recorded around the
        scoring kernel (the timed entry point), else None."""
        festina_score_placements(self.lut, self.gpus, self.req, self.out, self.workspace, self.ws_bytes, stream,
                                 events)

    def run_noalloc(self, stream=None):
        """The same search through the allocation-free entry point (the library's scratch)."""
        festina_score_placements_noalloc(self.lut, self.gpus, self.req, self.out, stream)

    def results(self):
        R = self.R
        return (self.choice[:R].cpu().numpy(), self.feasible[:R].cpu().numpy(), self.energy[:R].cpu().numpy())


class DeviceMigration:
    """Consolidation fleet copied to device memory once, with the ABI structs pointing at it."""

    def __init__(self, inp: dict, device="cuda"):
        import torch
        lut, fl = inp["lut"], inp["fleet"]
        d = lambda a, t: _dev(a, t, device)
        self.t = {
            "freq_level": d(lut["freq_level"], np.float32), "sm_level": d(lut["sm_level"], np.float32),
            "pf": d(lut["pf"], np.float32), "dc": d(lut["dc"], np.float32),
        }
        for k in ("n_inst", "inst_model", "inst_prompt_tokens", "inst_batch", "inst_sm", "hbm_mib", "sm_permille"):
            self.t[k] = d(fl[k], np.int32)
        for k in ("inst_slo_ttft_ms", "inst_slo_tbt_ms", "util", "k_dyn_w"):
            self.t[k] = d(fl[k], np.float32)
        t = self.t
        self.lut = festina_lut(int(lut["n_models"]), int(lut["n_rows"]), int(lut["n_sm"]), int(lut["n_freq"]),
                               _ptr(t["sm_level"]), _ptr(t["freq_level"]), _ptr(t["pf"]), _ptr(t["dc"]),
                               float(lut["p0_w"]))
        self.G = int(fl["n_gpus"])
        self.fleet = festina_fleet(self.G, int(fl["max_inst"]), _ptr(t["n_inst"]), _ptr(t["inst_model"]),
                                   _ptr(t["inst_prompt_tokens"]), _ptr(t["inst_batch"]), _ptr(t["inst_sm"]),
                                   _ptr(t["inst_slo_ttft_ms"]), _ptr(t["inst_slo_tbt_ms"]), _ptr(t["hbm_mib"]),
                                   _ptr(t["sm_permille"]), _ptr(t["util"]), _ptr(t["k_dyn_w"]),
                                   int(fl["hbm_cap_mib"]), int(fl["sm_cap_permille"]))
        self.best_dst = torch.empty(self.G, dtype=torch.int32, device=device)
        self.saving = torch.empty(self.G, dtype=torch.float32, device=device)
        self.level = torch.empty(self.G, dtype=torch.int32, device=device)
        self.out = festina_migrations(_ptr(self.best_dst), _ptr(self.saving), _ptr(self.level))
        self.ws_bytes = festina_migrations_workspace_bytes(self.lut, self.fleet)
        self.workspace = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=device)

    def run(self, stream=None, events=None):
        """One search; `events` = (begin, end) raw hipEvent_t handles recorded around the
        pair-scoring kernel (the timed entry point), else None."""
        festina_score_migrations(self.lut, self.fleet, self.out, self.workspace, self.ws_bytes, stream, events)

    def results(self):
        return self.best_dst.cpu().numpy(), self.saving.cpu().numpy(), self.level.cpu().numpy()


class DeviceSweep:
    """Local-scheduler task batches copied to device memory once, with the ABI structs."""

    def __init__(self, inp: dict, device="cuda"):
        import torch
        lut, bt = inp["lut"], inp["batches"]
        d = lambda a, t: _dev(a, t, device)
        self.t = {
            "freq_level": d(lut["freq_level"], np.float32), "sm_level": d(lut["sm_level"], np.float32),
            "pf": d(lut["pf"], np.float32), "dc": d(lut["dc"], np.float32),
        }
        for k in ("n_tasks", "task_model", "task_phase", "task_tokens", "sm_units"):
            self.t[k] = d(bt[k], np.int32)
        for k in ("task_slack_ms", "k_dyn_w", "util"):
            self.t[k] = d(bt[k], np.float32)
        t = self.t
        self.lut = festina_lut(int(lut["n_models"]), int(lut["n_rows"]), int(lut["n_sm"]), int(lut["n_freq"]),
                               _ptr(t["sm_level"]), _ptr(t["freq_level"]), _ptr(t["pf"]), _ptr(t["dc"]),
                               float(lut["p0_w"]))
        self.B, self.T = int(bt["n_batches"]), int(bt["max_tasks"])
        self.batches = festina_batches(self.B, self.T, _ptr(t["n_tasks"]), _ptr(t["task_model"]),
                                       _ptr(t["task_phase"]), _ptr(t["task_tokens"]), _ptr(t["task_slack_ms"]),
                                       _ptr(t["k_dyn_w"]), _ptr(t["util"]), _ptr(t["sm_units"]),
                                       int(bt["sm_budget"]), int(bt.get("static_power", 0)))
        n = max(self.B, 1)
        self.level = torch.empty(n, dtype=torch.int32, device=device)
        self.feasible = torch.empty(n, dtype=torch.uint8, device=device)
        self.energy = torch.empty(n, dtype=torch.float32, device=device)
        self.task_sm = torch.empty((n, self.T), dtype=torch.int32, device=device)
        self.out = festina_sweep_result(_ptr(self.level), _ptr(self.feasible), _ptr(self.energy),
                                        _ptr(self.task_sm))

    def run(self, stream=None):
        festina_sweep_batches(self.lut, self.batches, self.out, stream)

    def results(self):
        B = self.B
        return (self.level[:B].cpu().numpy(), self.feasible[:B].cpu().numpy(), self.energy[:B].cpu().numpy(),
                self.task_sm[:B].cpu().numpy())


PREF_INT = ("sm_p", "f_p", "sm_d", "f_d")
PREF_FLOAT = ("t_p_ms", "t_d_ms", "p_p_w", "p_d_w", "t_ms", "sm_pref", "f_pref")


class DevicePreferred:
    """Active LLM instances copied to device memory once; run() computes every preferred
    configuration and then the fleet's EWR from them (execution time t_ms = t_p + t_d)."""

    def __init__(self, inp: dict, device="cuda"):
        import torch
        lut, q = inp["lut"], inp["llms"]
        d = lambda a, t: _dev(a, t, device)
        self.t = {
            "freq_level": d(lut["freq_level"], np.float32), "sm_level": d(lut["sm_level"], np.float32),
            "pf": d(lut["pf"], np.float32), "dc": d(lut["dc"], np.float32),
        }
        for k in ("n_inst", "model", "avg_in_tokens", "avg_out_tokens", "batch"):
            self.t[k] = d(q[k], np.int32)
        for k in ("slo_ttft_ms", "slo_tbt_ms", "k_dyn_w"):
            self.t[k] = d(q[k], np.float32)
        t = self.t
        self.lut = festina_lut(int(lut["n_models"]), int(lut["n_rows"]), int(lut["n_sm"]), int(lut["n_freq"]),
                               _ptr(t["sm_level"]), _ptr(t["freq_level"]), _ptr(t["pf"]), _ptr(t["dc"]),
                               float(lut["p0_w"]))
        self.G, self.K = int(q["n_gpus"]), int(q["max_inst"])
        self.llms = festina_llms(self.G, self.K, _ptr(t["n_inst"]), _ptr(t["model"]), _ptr(t["avg_in_tokens"]),
                                 _ptr(t["avg_out_tokens"]), _ptr(t["batch"]), _ptr(t["slo_ttft_ms"]),
                                 _ptr(t["slo_tbt_ms"]), _ptr(t["k_dyn_w"]))
        n = max(self.G * self.K, 1)
        self.o = {k: torch.empty(n, dtype=torch.int32, device=device) for k in PREF_INT}
        self.o.update({k: torch.empty(n, dtype=torch.float32, device=device) for k in PREF_FLOAT})
        self.o["feasible"] = torch.empty(n, dtype=torch.uint8, device=device)
        self.out = festina_preferred(*(_ptr(self.o[k]) for k in PREF_INT + PREF_FLOAT + ("feasible",)))
        g = max(self.G, 1)
        self.f_gpu = torch.empty(g, dtype=torch.float32, device=device)
        self.waste_gpu = torch.empty(g, dtype=torch.float64, device=device)
        self.totals = torch.empty(3, dtype=torch.float64, device=device)
        self.ewr = festina_ewr(_ptr(self.f_gpu), _ptr(self.waste_gpu), _ptr(self.totals))
        self.ws_bytes = festina_ewr_workspace_bytes(self.G)
        self.workspace = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=device)

    def run_preferred(self, stream=None):
        festina_preferred_configs(self.lut, self.llms, self.out, stream)

    def run_ewr(self, f_pref=None, t_ms=None, stream=None):
        """EWR from device tensors f_pref/t_ms [G*K] (default: this object's own results)."""
        if f_pref is None:
            f_pref = self.o["f_pref"]
            t_ms = self.o["t_ms"]
        festina_fleet_ewr(self.G, self.K, self.t["n_inst"], f_pref, t_ms, self.ewr, self.workspace,
                          self.ws_bytes, stream)

    def run(self, stream=None):
        """Preferred configurations, then the EWR of the fleet from them."""
        self.run_preferred(stream)
        self.run_ewr(stream=stream)

    def results(self):
        G, K = self.G, self.K
        r = {k: self.o[k][:G * K].cpu().numpy().reshape(G, K) for k in PREF_INT + PREF_FLOAT + ("feasible",)}
        return r

    def ewr_results(self):
        return self.f_gpu[:self.G].cpu().numpy(), self.waste_gpu[:self.G].cpu().numpy(), self.totals.cpu().numpy()


class DeviceDispatch:
    """Requests and the GPUs' answers for the paper's own dispatcher, on the device."""

    def __init__(self, inp: dict, device="cuda"):
        import torch
        lut, av, rq = inp["lut"], inp["avail"], inp["requests"]
        d = lambda a, t: _dev(a, t, device)
        self.t = {
            "sm_level": d(lut["sm_level"], np.float32), "freq_level": d(lut["freq_level"], np.float32),
            "pf": d(lut["pf"], np.float32), "dc": d(lut["dc"], np.float32),
            "resident": d(np.asarray(av["resident"], np.uint32).view(np.int32), np.int32),
        }
        for k in ("freq_cur", "batch", "mem_free_mib", "sm_free", "kv_kib_per_token"):
            self.t[k] = d(av[k], np.int32)
        for k in ("k_dyn_w", "t_avail_ms"):
            self.t[k] = d(av[k], np.float32)
        for k in ("model", "prompt_tokens", "pred_out_tokens"):
            self.t[k] = d(rq[k], np.int32)
        for k in ("slo_ttft_ms", "slo_tbt_ms"):
            self.t[k] = d(rq[k], np.float32)
        t = self.t
        self.lut = festina_lut(int(lut["n_models"]), int(lut["n_rows"]), int(lut["n_sm"]), int(lut["n_freq"]),
                               _ptr(t["sm_level"]), _ptr(t["freq_level"]), _ptr(t["pf"]), _ptr(t["dc"]),
                               float(lut["p0_w"]))
        self.avail = festina_gpu_avail(int(av["n_gpus"]), int(av["n_steps"]), _ptr(t["freq_cur"]), _ptr(t["batch"]),
                                       _ptr(t["k_dyn_w"]), _ptr(t["resident"]), _ptr(t["t_avail_ms"]),
                                       _ptr(t["mem_free_mib"]), _ptr(t["sm_free"]), _ptr(t["kv_kib_per_token"]),
                                       float(av["k_new_w"]))
        self.R = int(rq["n_requests"])
        self.req = festina_requests(self.R, _ptr(t["model"]), None, _ptr(t["prompt_tokens"]),
                                    _ptr(t["pred_out_tokens"]), _ptr(t["slo_ttft_ms"]), _ptr(t["slo_tbt_ms"]))
        n = max(self.R, 1)
        self.o = {k: torch.empty(n, dtype=torch.int32, device=device) for k in ("gpu", "freq_level", "sm_level")}
        self.o["phase"] = torch.empty(n, dtype=torch.uint8, device=device)
        self.o["energy_mj"] = torch.empty(n, dtype=torch.float32, device=device)
        self.out = festina_dispatches(*(_ptr(self.o[k]) for k in ("gpu", "freq_level", "sm_level", "phase",
                                                                  "energy_mj")))
        self.ws_bytes = festina_dispatch_workspace_bytes(self.lut, self.avail)
        self.workspace = torch.empty(max(self.ws_bytes, 256), dtype=torch.uint8, device=device)

    def run(self, stream=None):
        festina_dispatch_requests(self.lut, self.avail, self.req, self.out, self.workspace, self.ws_bytes, stream)

    def run_waves(self, wave_start, stream=None):
        """Dispatch wave by wave (requests ordered by wave), committing each wave; the
        carried state lands in self.state_t."""
        import torch
        if not hasattr(self, "state_t"):
            dev = self.t["batch"].device
            G, S = int(self.avail.n_gpus), int(self.avail.n_steps)
            self.state_t = {"freq_cur": torch.empty(G, dtype=torch.int32, device=dev),
                            "batch": torch.empty(G, dtype=torch.int32, device=dev),
                            "mem_free_mib": torch.empty(G * S, dtype=torch.int32, device=dev)}
            self.state = festina_gpu_state(*(_ptr(self.state_t[k]) for k in ("freq_cur", "batch", "mem_free_mib")))
            self.wws_bytes = festina_dispatch_waves_workspace_bytes(self.lut, self.avail)
            self.wworkspace = torch.empty(max(self.wws_bytes, 256), dtype=torch.uint8, device=dev)
        festina_dispatch_waves(self.lut, self.avail, self.req, wave_start, self.state, self.out, self.wworkspace,
                               self.wws_bytes, stream)

    def results(self):
        R = self.R
        return tuple(self.o[k][:R].cpu().numpy() for k in ("gpu", "freq_level", "sm_level", "phase", "energy_mj"))

    def state_results(self):
        G, S = int(self.avail.n_gpus), int(self.avail.n_steps)
        return {"freq_cur": self.state_t["freq_cur"].cpu().numpy(), "batch": self.state_t["batch"].cpu().numpy(),
                "mem_free_mib": self.state_t["mem_free_mib"].cpu().numpy().reshape(G, S)}


class DeviceTransfer:
    """A reconfiguring fleet on the device: the device-mapping cost matrix and the
    in-flight requests' finish-or-move decisions."""

    def __init__(self, inp: dict, device="cuda"):
        import torch
        lut, tr, pl, mv = inp["lut"], inp["transfer"], inp["plan"], inp["moves"]
        d = lambda a, t: _dev(a, t, device)
        self.t = {"sm_level": d(lut["sm_level"], np.float32), "freq_level": d(lut["freq_level"], np.float32),
                  "pf": d(lut["pf"], np.float32), "dc": d(lut["dc"], np.float32),
                  "resident": d(np.asarray(tr["resident"], np.uint32).view(np.int32), np.int32)}
        for k in ("weights_mib", "state_mib", "node"):
            self.t[k] = d(tr[k], np.int32)
        for k in ("dest", "freq_cur", "sm_cur", "batch"):
            self.t["plan_" + k] = d(pl[k], np.int32)
        for k in ("src", "model", "context_tokens", "remaining_tokens", "kv_kib", "token_kib"):
            self.t["req_" + k] = d(mv[k], np.int32)
        t = self.t
        self.lut = festina_lut(int(lut["n_models"]), int(lut["n_rows"]), int(lut["n_sm"]), int(lut["n_freq"]),
                               _ptr(t["sm_level"]), _ptr(t["freq_level"]), _ptr(t["pf"]), _ptr(t["dc"]),
                               float(lut["p0_w"]))
        self.G = int(tr["n_gpus"])
        self.transfer = festina_transfer(self.G, int(inp["n_models"]), _ptr(t["resident"]), _ptr(t["weights_mib"]),
                                         _ptr(t["state_mib"]), _ptr(t["node"]), float(tr["bw_intra_gbs"]),
                                         float(tr["bw_inter_gbs"]))
        self.plan = festina_plan(_ptr(t["plan_dest"]), _ptr(t["plan_freq_cur"]), _ptr(t["plan_sm_cur"]),
                                 _ptr(t["plan_batch"]))
        self.Q = int(mv["n_requests"])
        self.req = festina_inflight(self.Q, *(_ptr(t["req_" + k]) for k in ("src", "model", "context_tokens",
                                                                           "remaining_tokens", "kv_kib",
                                                                           "token_kib")))
        self.cost = torch.empty((self.G, self.G), dtype=torch.float32, device=device)
        n = max(self.Q, 1)
        self.decision = torch.empty(n, dtype=torch.int32, device=device)
        self.remaining = torch.empty(n, dtype=torch.float32, device=device)
        self.migrate = torch.empty(n, dtype=torch.float32, device=device)
        self.moves = festina_moves(_ptr(self.decision), _ptr(self.remaining), _ptr(self.migrate))

    def run_costs(self, stream=None):
        festina_transfer_costs(self.transfer, self.cost, stream)

    def run_moves(self, stream=None):
        festina_request_moves(self.lut, self.transfer, self.plan, self.req, self.moves, stream)

    def results(self):
        Q = self.Q
        return (self.cost.cpu().numpy(), self.decision[:Q].cpu().numpy(), self.remaining[:Q].cpu().numpy(),
                self.migrate[:Q].cpu().numpy())


# ------------------------------------------------------------------ the ABI calls
def festina_placements_workspace_bytes(lut, gpus, req) -> int:
    return int(lib().festina_placements_workspace_bytes(C.byref(lut), C.byref(gpus), C.byref(req)))


def _events(events):
    b, e = events
    return (C.c_void_p(b) if b else None), (C.c_void_p(e) if e else None)


def festina_score_placements(lut, gpus, req, out, workspace, workspace_bytes, stream=None, events=None) -> None:
    """festina_score_placements, or festina_score_placements_timed when `events` = (begin, end)
    raw hipEvent_t handles."""
    ws = None if workspace is None else C.c_void_p(workspace.data_ptr())
    args = (C.byref(lut), C.byref(gpus), C.byref(req), C.byref(out), ws, int(workspace_bytes),
            _stream_handle(stream))
    if events is None:
        st = lib().festina_score_placements(*args)
    else:
        st = lib().festina_score_placements_timed(*args, *_events(events))
    if st != FESTINA_OK:
        raise FestinaError(st, "festina_score_placements")


def festina_score_placements_noalloc(lut, gpus, req, out, stream=None) -> None:
    st = lib().festina_score_placements_noalloc(C.byref(lut), C.byref(gpus), C.byref(req), C.byref(out),
                                                _stream_handle(stream))
    if st != FESTINA_OK:
        raise FestinaError(st, "festina_score_placements_noalloc")


def festina_migrations_workspace_bytes(lut, fleet) -> int:
    return int(lib().festina_migrations_workspace_bytes(C.byref(lut), C.byref(fleet)))


def festina_score_migrations(lut, fleet, out, workspace, workspace_bytes, stream=None, events=None) -> None:
    """festina_score_migrations, or festina_score_migrations_timed when `events` = (begin, end)
    raw hipEvent_t handles."""
    ws = None if workspace is None else C.c_void_p(workspace.data_ptr())
    args = (C.byref(lut), C.byref(fleet), C.byref(out), ws, int(workspace_bytes), _stream_handle(stream))
    if events is None:
        st = lib().festina_score_migrations(*args)
    else:
        st = lib().festina_score_migrations_timed(*args, *_events(events))
    if st != FESTINA_OK:
        raise FestinaError(st, "festina_score_migrations")


def festina_sweep_batches(lut, batches, out, stream=None) -> None:
    st = lib().festina_sweep_batches(C.byref(lut), C.byref(batches), C.byref(out), _stream_handle(stream))
    if st != FESTINA_OK:
        raise FestinaError(st, "festina_sweep_batches")


def festina_preferred_configs(lut, llms, out, stream=None) -> None:
    st = lib().festina_preferred_configs(C.byref(lut), C.byref(llms), C.byref(out), _stream_handle(stream))
    if st != FESTINA_OK:
        raise FestinaError(st, "festina_preferred_configs")


def festina_ewr_workspace_bytes(n_gpus: int) -> int:
    return int(lib().festina_ewr_workspace_bytes(int(n_gpus)))


def festina_fleet_ewr(n_gpus, max_inst, n_inst, f_pref, t_ms, out, workspace, workspace_bytes, stream=None) -> None:
    ws = None if workspace is None else C.c_void_p(workspace.data_ptr())
    st = lib().festina_fleet_ewr(int(n_gpus), int(max_inst), _ptr(n_inst), _ptr(f_pref), _ptr(t_ms), C.byref(out),
                                 ws, int(workspace_bytes), _stream_handle(stream))
    if st != FESTINA_OK:
        raise FestinaError(st, "festina_fleet_ewr")


def festina_dispatch_workspace_bytes(lut, avail) -> int:
    return int(lib().festina_dispatch_workspace_bytes(C.byref(lut), C.byref(avail)))


def festina_dispatch_requests(lut, avail, req, out, workspace, workspace_bytes, stream=None) -> None:
    ws = None if workspace is None else C.c_void_p(workspace.data_ptr())
    st = lib().festina_dispatch_requests(C.byref(lut), C.byref(avail), C.byref(req), C.byref(out), ws,
                                         int(workspace_bytes), _stream_handle(stream))
    if st != FESTINA_OK:
        raise FestinaError(st, "festina_dispatch_requests")


def festina_dispatch_waves_workspace_bytes(lut, avail) -> int:
    return int(lib().festina_dispatch_waves_workspace_bytes(C.byref(lut), C.byref(avail)))


def festina_dispatch_waves(lut, avail, req, wave_start, state, out, workspace, workspace_bytes, stream=None) -> None:
    """wave_start: host sequence of n_waves + 1 request offsets."""
    ws = None if workspace is None else C.c_void_p(workspace.data_ptr())
    bounds = np.ascontiguousarray(wave_start, dtype=np.int32)
    st = lib().festina_dispatch_waves(C.byref(lut), C.byref(avail), C.byref(req), int(bounds.size) - 1,
                                      bounds.ctypes.data if bounds.size else None, C.byref(state), C.byref(out), ws,
                                      int(workspace_bytes), _stream_handle(stream))
    if st != FESTINA_OK:
        raise FestinaError(st, "festina_dispatch_waves")


def festina_transfer_costs(transfer, cost, stream=None) -> None:
    st = lib().festina_transfer_costs(C.byref(transfer), _ptr(cost), _stream_handle(stream))
    if st != FESTINA_OK:
        raise FestinaError(st, "festina_transfer_costs")


def festina_request_moves(lut, transfer, plan, req, out, stream=None) -> None:
    st = lib().festina_request_moves(C.byref(lut), C.byref(transfer), C.byref(plan), C.byref(req), C.byref(out),
                                     _stream_handle(stream))
    if st != FESTINA_OK:
        raise FestinaError(st, "festina_request_moves")
