"""CPU oracle of the batched energy-aware placement and migration search and of the
local SM/frequency sweep.

TEST INFRASTRUCTURE ONLY: the test suite, the package smoke check and the
benchmark's CPU-baseline leg are the only callers.  The product path never
imports this package.  It wraps ``festina_oracle.c`` (plain C, float64) with
ctypes; nothing here is shared with the HIP library.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "festina_oracle.c")
LIB_PATH = os.environ.get("FESTINA_ORACLE_LIB") or os.path.join(_HERE, "libfestina_oracle.so")
BUILD_CMD = ["gcc", "-O2", "-ffp-contract=off", "-fPIC", "-shared", "-Wall", "-Wextra",
             "-o", LIB_PATH, _SRC, "-lm"]

_lib = None


def build() -> str:
    """Compile the oracle library in place (gcc, -O2, no FP contraction, no fast-math)."""
    subprocess.run(BUILD_CMD, check=True)
    return LIB_PATH


# AddressSanitizer + UndefinedBehaviorSanitizer build of the same source (host code only, gcc):
# any report aborts the process.  The library is loaded into an uninstrumented Python, so the
# sanitizer runtime must come first: sanitized_env() gives the environment for that.
SANITIZE_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                  "-fno-sanitize-recover=all", "-ffp-contract=off", "-fPIC", "-shared", "-Wall", "-Wextra"]


def build_sanitized(path: str) -> str:
    """Compile the oracle with ASan and UBSan into `path`."""
    subprocess.run(["gcc", *SANITIZE_FLAGS, "-o", path, _SRC, "-lm"], check=True)
    return path


def sanitized_env(path: str) -> dict:
    """Environment for a child Python that loads the sanitized oracle at `path`."""
    asan = subprocess.run(["gcc", "-print-file-name=libasan.so"], check=True, stdout=subprocess.PIPE,
                          text=True).stdout.strip()
    ubsan = subprocess.run(["gcc", "-print-file-name=libubsan.so"], check=True, stdout=subprocess.PIPE,
                           text=True).stdout.strip()
    env = dict(os.environ, FESTINA_ORACLE_LIB=path, LD_PRELOAD=f"{asan}:{ubsan}",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    return env


class _Lut(C.Structure):
    _fields_ = [("n_models", C.c_int32), ("n_rows", C.c_int32), ("n_sm", C.c_int32),
                ("n_freq", C.c_int32), ("sm_level", C.c_void_p), ("freq_level", C.c_void_p),
                ("pf", C.c_void_p), ("dc", C.c_void_p), ("p0_w", C.c_double)]


class _Gpus(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("n_waves", C.c_int32), ("batch", C.c_void_p),
                ("k_dyn_w", C.c_void_p), ("resident", C.c_void_p), ("cap_pf", C.c_void_p),
                ("cap_dc", C.c_void_p)]


class _Requests(C.Structure):
    _fields_ = [("n_requests", C.c_int32), ("model", C.c_void_p), ("wave", C.c_void_p),
                ("prompt_tokens", C.c_void_p), ("pred_out_tokens", C.c_void_p),
                ("slo_ttft_ms", C.c_void_p), ("slo_tbt_ms", C.c_void_p)]


class _Fleet(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("max_inst", C.c_int32), ("n_inst", C.c_void_p),
                ("inst_model", C.c_void_p), ("inst_prompt_tokens", C.c_void_p),
                ("inst_batch", C.c_void_p), ("inst_sm", C.c_void_p),
                ("inst_slo_ttft_ms", C.c_void_p), ("inst_slo_tbt_ms", C.c_void_p),
                ("hbm_mib", C.c_void_p), ("sm_permille", C.c_void_p), ("util", C.c_void_p),
                ("k_dyn_w", C.c_void_p), ("hbm_cap_mib", C.c_int32), ("sm_cap_permille", C.c_int32)]


class _Batches(C.Structure):
    _fields_ = [("n_batches", C.c_int32), ("max_tasks", C.c_int32), ("n_tasks", C.c_void_p),
                ("task_model", C.c_void_p), ("task_phase", C.c_void_p), ("task_tokens", C.c_void_p),
                ("task_slack_ms", C.c_void_p), ("k_dyn_w", C.c_void_p), ("util", C.c_void_p),
                ("sm_units", C.c_void_p), ("sm_budget", C.c_int32), ("static_power", C.c_int32)]


class _Llms(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("max_inst", C.c_int32), ("n_inst", C.c_void_p),
                ("model", C.c_void_p), ("avg_in_tokens", C.c_void_p), ("avg_out_tokens", C.c_void_p),
                ("batch", C.c_void_p), ("slo_ttft_ms", C.c_void_p), ("slo_tbt_ms", C.c_void_p),
                ("k_dyn_w", C.c_void_p)]


class _Pref(C.Structure):
    _fields_ = [("sm_p", C.c_int32), ("f_p", C.c_int32), ("sm_d", C.c_int32), ("f_d", C.c_int32),
                ("t_p", C.c_double), ("t_d", C.c_double), ("p_p", C.c_double), ("p_d", C.c_double),
                ("sm_pref", C.c_double), ("f_pref", C.c_double), ("feasible", C.c_int)]


class _Avail(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("n_steps", C.c_int32), ("freq_cur", C.c_void_p), ("batch", C.c_void_p),
                ("k_dyn_w", C.c_void_p), ("resident", C.c_void_p), ("t_avail_ms", C.c_void_p),
                ("mem_free_mib", C.c_void_p), ("sm_free", C.c_void_p), ("kv_kib_per_token", C.c_void_p),
                ("k_new_w", C.c_float)]


class _Dispatch(C.Structure):
    _fields_ = [("gpu", C.c_int32), ("freq_level", C.c_int32), ("sm_level", C.c_int32), ("phase", C.c_int32),
                ("energy", C.c_double)]


class _Transfer(C.Structure):
    _fields_ = [("n_gpus", C.c_int32), ("words", C.c_int32), ("resident", C.c_void_p), ("weights_mib", C.c_void_p),
                ("state_mib", C.c_void_p), ("node", C.c_void_p), ("bw_intra_gbs", C.c_float),
                ("bw_inter_gbs", C.c_float)]


class _Moves(C.Structure):
    _fields_ = [("n_requests", C.c_int32), ("src", C.c_void_p), ("model", C.c_void_p),
                ("context_tokens", C.c_void_p), ("remaining_tokens", C.c_void_p), ("kv_kib", C.c_void_p),
                ("token_kib", C.c_void_p)]


class _Plan(C.Structure):
    _fields_ = [("dest", C.c_void_p), ("freq_cur", C.c_void_p), ("sm_cur", C.c_void_p), ("batch", C.c_void_p)]


def lib():
    global _lib
    if _lib is None:
        if "FESTINA_ORACLE_LIB" not in os.environ and (
                not os.path.exists(LIB_PATH) or os.path.getmtime(LIB_PATH) < os.path.getmtime(_SRC)):
            build()
        L = C.CDLL(LIB_PATH)
        P = C.POINTER
        L.festina_oracle_score_placements.argtypes = [P(_Lut), P(_Gpus), P(_Requests), C.c_int32,
                                                      C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.festina_oracle_score_placements.restype = C.c_int
        L.festina_oracle_candidate.argtypes = [P(_Lut), P(_Gpus), P(_Requests), C.c_int32,
                                               C.c_int64, P(C.c_double)]
        L.festina_oracle_candidate.restype = C.c_int
        L.festina_oracle_score_migrations.argtypes = [P(_Lut), P(_Fleet), C.c_int32, C.c_void_p,
                                                      C.c_void_p, C.c_void_p, C.c_void_p]
        L.festina_oracle_score_migrations.restype = C.c_int
        L.festina_oracle_pair.argtypes = [P(_Lut), P(_Fleet), C.c_int32, C.c_int32,
                                          P(C.c_int32), P(C.c_double)]
        L.festina_oracle_pair.restype = C.c_int
        L.festina_oracle_prompt_row.argtypes = [C.c_int32]
        L.festina_oracle_prompt_row.restype = C.c_int
        L.festina_oracle_padded_out.argtypes = [C.c_int32]
        L.festina_oracle_padded_out.restype = C.c_int64
        L.festina_oracle_sweep.argtypes = [P(_Lut), P(_Batches), C.c_int32, C.c_void_p,
                                           C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.festina_oracle_sweep.restype = C.c_int
        L.festina_oracle_sweep_level.argtypes = [P(_Lut), P(_Batches), C.c_int32, C.c_int32,
                                                 P(C.c_double)]
        L.festina_oracle_sweep_level.restype = C.c_int
        L.festina_oracle_min_sm.argtypes = [P(_Lut), P(_Batches), C.c_int32, C.c_int32, C.c_int32]
        L.festina_oracle_min_sm.restype = C.c_int
        L.festina_oracle_preferred.argtypes = [P(_Lut), P(_Llms), C.c_void_p]
        L.festina_oracle_preferred.restype = C.c_int
        L.festina_oracle_phase_cell.argtypes = [P(_Lut), P(_Llms), C.c_int32, C.c_int32, C.c_int32,
                                                C.c_int32, C.c_int32, P(C.c_double), P(C.c_double)]
        L.festina_oracle_phase_cell.restype = C.c_int
        L.festina_oracle_preferred_at.argtypes = [P(_Lut), P(_Llms), C.c_int32, C.c_int32, C.c_int32,
                                                  C.c_int32, C.c_int32, C.c_int32, P(C.c_double), P(C.c_double)]
        L.festina_oracle_preferred_at.restype = C.c_int
        L.festina_oracle_dispatch.argtypes = [P(_Lut), P(_Avail), P(_Requests), C.c_int32, C.c_void_p, C.c_void_p]
        L.festina_oracle_dispatch.restype = C.c_int
        L.festina_oracle_dispatch_waves.argtypes = [P(_Lut), P(_Avail), P(_Requests), C.c_int32, C.c_void_p,
                                                    C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p]
        L.festina_oracle_dispatch_waves.restype = C.c_int
        L.festina_oracle_transfer_costs.argtypes = [P(_Transfer), C.c_int32, C.c_void_p]
        L.festina_oracle_transfer_costs.restype = C.c_int
        L.festina_oracle_request_moves.argtypes = [P(_Lut), P(_Transfer), P(_Plan), P(_Moves), C.c_void_p,
                                                   C.c_void_p, C.c_void_p]
        L.festina_oracle_request_moves.restype = C.c_int
        L.festina_oracle_fleet_ewr.argtypes = [C.c_int32, C.c_int32, C.c_void_p, C.c_void_p, C.c_void_p,
                                               C.c_void_p, C.c_void_p, C.c_void_p]
        L.festina_oracle_fleet_ewr.restype = C.c_int
        _lib = L
    return _lib


# ------------------------------------------------------------------ marshalling
def _arr(a, dtype):
    if a is None:
        return None
    return np.ascontiguousarray(a, dtype=dtype)


def _p(a):
    return None if a is None else a.ctypes.data


class _Pinned:
    """Holds the contiguous arrays alive while the structs point at them."""

    def __init__(self):
        self.keep = []

    def __call__(self, a, dtype):
        a = _arr(a, dtype)
        if a is not None:
            self.keep.append(a)
        return _p(a)


def _lut(d, pin):
    return _Lut(int(d["n_models"]), int(d["n_rows"]), int(d["n_sm"]), int(d["n_freq"]),
                pin(d["sm_level"], np.float32), pin(d["freq_level"], np.float32),
                pin(d["pf"], np.float32), pin(d["dc"], np.float32), float(d["p0_w"]))


def _gpus(d, pin):
    return _Gpus(int(d["n_gpus"]), int(d["n_waves"]), pin(d["batch"], np.int32),
                 pin(d["k_dyn_w"], np.float32), pin(d["resident"], np.uint32),
                 pin(d.get("cap_pf"), np.int8), pin(d.get("cap_dc"), np.int8))


def _requests(d, pin):
    return _Requests(int(d["n_requests"]), pin(d["model"], np.int32), pin(d.get("wave"), np.int32),
                     pin(d["prompt_tokens"], np.int32), pin(d["pred_out_tokens"], np.int32),
                     pin(d["slo_ttft_ms"], np.float32), pin(d["slo_tbt_ms"], np.float32))


def _fleet(d, pin):
    return _Fleet(int(d["n_gpus"]), int(d["max_inst"]), pin(d["n_inst"], np.int32),
                  pin(d["inst_model"], np.int32), pin(d["inst_prompt_tokens"], np.int32),
                  pin(d["inst_batch"], np.int32), pin(d["inst_sm"], np.int32),
                  pin(d["inst_slo_ttft_ms"], np.float32), pin(d["inst_slo_tbt_ms"], np.float32),
                  pin(d["hbm_mib"], np.int32), pin(d["sm_permille"], np.int32),
                  pin(d["util"], np.float32), pin(d["k_dyn_w"], np.float32),
                  int(d["hbm_cap_mib"]), int(d["sm_cap_permille"]))


def _batches(d, pin):
    return _Batches(int(d["n_batches"]), int(d["max_tasks"]), pin(d["n_tasks"], np.int32),
                    pin(d["task_model"], np.int32), pin(d["task_phase"], np.int32),
                    pin(d["task_tokens"], np.int32), pin(d["task_slack_ms"], np.float32),
                    pin(d["k_dyn_w"], np.float32), pin(d["util"], np.float32),
                    pin(d["sm_units"], np.int32), int(d["sm_budget"]), int(d.get("static_power", 0)))


def _llms(d, pin):
    return _Llms(int(d["n_gpus"]), int(d["max_inst"]), pin(d["n_inst"], np.int32), pin(d["model"], np.int32),
                 pin(d["avg_in_tokens"], np.int32), pin(d["avg_out_tokens"], np.int32),
                 pin(d["batch"], np.int32), pin(d["slo_ttft_ms"], np.float32), pin(d["slo_tbt_ms"], np.float32),
                 pin(d["k_dyn_w"], np.float32))


def _avail(d, pin):
    return _Avail(int(d["n_gpus"]), int(d["n_steps"]), pin(d["freq_cur"], np.int32), pin(d["batch"], np.int32),
                  pin(d["k_dyn_w"], np.float32), pin(d["resident"], np.uint32), pin(d["t_avail_ms"], np.float32),
                  pin(d["mem_free_mib"], np.int32), pin(d["sm_free"], np.int32),
                  pin(d["kv_kib_per_token"], np.int32), float(d["k_new_w"]))


def _transfer(d, pin):
    return _Transfer(int(d["n_gpus"]), int(d["words"]), pin(d["resident"], np.uint32), pin(d["weights_mib"], np.int32),
                     pin(d["state_mib"], np.int32), pin(d["node"], np.int32), float(d["bw_intra_gbs"]),
                     float(d["bw_inter_gbs"]))


# ------------------------------------------------------------------ public API
def score_placements(inp: dict, sel=None):
    """Oracle placements for all requests (or the request ids in ``sel``).

    Returns (choice int32, feasible uint8, energy_mj float64), indexed like ``sel``.
    """
    pin = _Pinned()
    lut, gpus, req = _lut(inp["lut"], pin), _gpus(inp["gpus"], pin), _requests(inp["requests"], pin)
    n = int(inp["requests"]["n_requests"]) if sel is None else len(sel)
    sel_a = None if sel is None else _arr(sel, np.int32)
    choice = np.empty(n, np.int32)
    feas = np.empty(n, np.uint8)
    energy = np.empty(n, np.float64)
    rc = lib().festina_oracle_score_placements(C.byref(lut), C.byref(gpus), C.byref(req), n,
                                               _p(sel_a), _p(choice), _p(feas), _p(energy))
    if rc != 0:
        raise ValueError("oracle rejected the placement arguments")
    return choice, feas, energy


def candidate_energy(inp: dict, r: int, idx: int):
    """(eligible, energy_mj) of candidate ``idx`` for request ``r``."""
    pin = _Pinned()
    lut, gpus, req = _lut(inp["lut"], pin), _gpus(inp["gpus"], pin), _requests(inp["requests"], pin)
    e = C.c_double(0.0)
    ok = lib().festina_oracle_candidate(C.byref(lut), C.byref(gpus), C.byref(req), int(r), int(idx),
                                        C.byref(e))
    return bool(ok), float(e.value)


def score_migrations(inp: dict, sel=None):
    """Oracle per-source best destinations (or for the source ids in ``sel``).

    Returns (best_dst int32, saving_w float64, freq_level int32).
    """
    pin = _Pinned()
    lut, fleet = _lut(inp["lut"], pin), _fleet(inp["fleet"], pin)
    n = int(inp["fleet"]["n_gpus"]) if sel is None else len(sel)
    sel_a = None if sel is None else _arr(sel, np.int32)
    best = np.empty(n, np.int32)
    sav = np.empty(n, np.float64)
    lev = np.empty(n, np.int32)
    rc = lib().festina_oracle_score_migrations(C.byref(lut), C.byref(fleet), n, _p(sel_a),
                                               _p(best), _p(sav), _p(lev))
    if rc != 0:
        raise ValueError("oracle rejected the migration arguments")
    return best, sav, lev


def pair_saving(inp: dict, s: int, d: int):
    """(eligible, k_star, saving_w) of moving source ``s`` onto destination ``d``."""
    pin = _Pinned()
    lut, fleet = _lut(inp["lut"], pin), _fleet(inp["fleet"], pin)
    k = C.c_int32(-1)
    sv = C.c_double(0.0)
    ok = lib().festina_oracle_pair(C.byref(lut), C.byref(fleet), int(s), int(d), C.byref(k), C.byref(sv))
    return bool(ok), int(k.value), float(sv.value)


def prompt_row(tokens: int) -> int:
    return int(lib().festina_oracle_prompt_row(int(tokens)))


def padded_out(predicted: int) -> int:
    return int(lib().festina_oracle_padded_out(int(predicted)))


def sweep(inp: dict, sel=None):
    """Oracle local SM/frequency sweep for all batches (or the batch ids in ``sel``).

    Returns (freq_level int32, feasible uint8, energy_mj float64, task_sm int32 [n, max_tasks]).
    """
    pin = _Pinned()
    lut, bat = _lut(inp["lut"], pin), _batches(inp["batches"], pin)
    n = int(inp["batches"]["n_batches"]) if sel is None else len(sel)
    T = int(inp["batches"]["max_tasks"])
    sel_a = None if sel is None else _arr(sel, np.int32)
    lev = np.empty(n, np.int32)
    feas = np.empty(n, np.uint8)
    energy = np.empty(n, np.float64)
    tsm = np.empty((n, T), np.int32)
    rc = lib().festina_oracle_sweep(C.byref(lut), C.byref(bat), n, _p(sel_a), _p(lev), _p(feas),
                                    _p(energy), _p(tsm))
    if rc != 0:
        raise ValueError("oracle rejected the sweep arguments")
    return lev, feas, energy, tsm


def sweep_level(inp: dict, b: int, k: int):
    """(usable, energy_mj) of batch ``b`` at frequency level ``k``."""
    pin = _Pinned()
    lut, bat = _lut(inp["lut"], pin), _batches(inp["batches"], pin)
    e = C.c_double(0.0)
    ok = lib().festina_oracle_sweep_level(C.byref(lut), C.byref(bat), int(b), int(k), C.byref(e))
    return bool(ok), float(e.value)


def min_sm(inp: dict, b: int, t: int, k: int) -> int:
    """Smallest SM level at which task ``t`` of batch ``b`` meets its slack at level ``k`` (-1: none)."""
    pin = _Pinned()
    lut, bat = _lut(inp["lut"], pin), _batches(inp["batches"], pin)
    return int(lib().festina_oracle_min_sm(C.byref(lut), C.byref(bat), int(b), int(t), int(k)))


PREF_FIELDS = ("sm_p", "f_p", "sm_d", "f_d", "t_p", "t_d", "p_p", "p_d", "sm_pref", "f_pref", "feasible")


def preferred(inp: dict) -> dict:
    """Oracle preferred configuration of every instance slot: dict of [G][K] arrays
    (levels int32, durations/powers/averages float64, feasible uint8)."""
    pin = _Pinned()
    lut, q = _lut(inp["lut"], pin), _llms(inp["llms"], pin)
    G, K = int(inp["llms"]["n_gpus"]), int(inp["llms"]["max_inst"])
    buf = (_Pref * max(G * K, 1))()
    if lib().festina_oracle_preferred(C.byref(lut), C.byref(q), C.cast(buf, C.c_void_p)) != 0:
        raise ValueError("oracle rejected the preferred-configuration arguments")
    out = {}
    for f in PREF_FIELDS:
        dt = np.float64 if f in ("t_p", "t_d", "p_p", "p_d", "sm_pref", "f_pref") else np.int32
        out[f] = np.array([getattr(buf[x], f) for x in range(G * K)], dt).reshape(G, K)
    out["feasible"] = out["feasible"].astype(np.uint8)
    return out


def phase_cell(inp: dict, g: int, i: int, decode: bool, j: int, k: int):
    """(feasible, duration_ms, power_w) of one phase of instance (g, i) at cell (j, k)."""
    pin = _Pinned()
    lut, q = _lut(inp["lut"], pin), _llms(inp["llms"], pin)
    t, p = C.c_double(0.0), C.c_double(0.0)
    ok = lib().festina_oracle_phase_cell(C.byref(lut), C.byref(q), int(g), int(i), int(bool(decode)),
                                         int(j), int(k), C.byref(t), C.byref(p))
    return bool(ok), float(t.value), float(p.value)


def fleet_ewr(n_inst, f_pref, t_ms):
    """Eq. energy_waste / energy_optimal / energy_waste_ratio over instance slots [G][K].

    Returns (f_gpu float64 [G], waste_gpu float64 [G], (E_waste, E_optimal, EWR))."""
    n_inst = _arr(n_inst, np.int32)
    f = _arr(f_pref, np.float32)
    t = _arr(t_ms, np.float32)
    G, K = f.shape
    fg = np.empty(G, np.float64)
    wg = np.empty(G, np.float64)
    tot = np.empty(3, np.float64)
    rc = lib().festina_oracle_fleet_ewr(G, K, _p(n_inst), _p(f), _p(t), _p(fg), _p(wg), _p(tot))
    if rc != 0:
        raise ValueError("oracle rejected the EWR arguments")
    return fg, wg, (float(tot[0]), float(tot[1]), float(tot[2]))


def preferred_at(inp: dict, g: int, i: int, jp: int, kp: int, jd: int, kd: int):
    """(feasible, sm_pref, f_pref) of instance (g, i) at the given prefill and decode cells."""
    pin = _Pinned()
    lut, q = _lut(inp["lut"], pin), _llms(inp["llms"], pin)
    sm, f = C.c_double(0.0), C.c_double(0.0)
    ok = lib().festina_oracle_preferred_at(C.byref(lut), C.byref(q), int(g), int(i), int(jp), int(kp), int(jd),
                                           int(kd), C.byref(sm), C.byref(f))
    return bool(ok), float(sm.value), float(f.value)


def dispatch(inp: dict, sel=None):
    """Oracle current-frequency dispatch (Sec. 3.3, Phases One to Three) of all requests (or
    the ids in ``sel``).  Returns (gpu, freq_level, sm_level, phase int32, energy float64)."""
    pin = _Pinned()
    lut, av, req = _lut(inp["lut"], pin), _avail(inp["avail"], pin), _requests(inp["requests"], pin)
    n = int(inp["requests"]["n_requests"]) if sel is None else len(sel)
    sel_a = None if sel is None else _arr(sel, np.int32)
    buf = (_Dispatch * max(n, 1))()
    rc = lib().festina_oracle_dispatch(C.byref(lut), C.byref(av), C.byref(req), n, _p(sel_a), C.cast(buf, C.c_void_p))
    if rc != 0:
        raise ValueError("oracle rejected the dispatch arguments")
    a = np.frombuffer(buf, dtype=np.dtype([("gpu", "<i4"), ("freq_level", "<i4"), ("sm_level", "<i4"),
                                           ("phase", "<i4"), ("energy", "<f8")]), count=n)
    return (a["gpu"].copy(), a["freq_level"].copy(), a["sm_level"].copy(), a["phase"].copy(), a["energy"].copy())


def dispatch_waves(inp: dict, wave_start):
    """Oracle dispatch wave by wave, each wave committed to the GPUs' state before the next
    (requests ordered by wave; wave w = requests wave_start[w] .. wave_start[w+1]-1).
    Returns (gpu, freq_level, sm_level, phase int32, energy float64) and the final state
    {"freq_cur", "batch", "mem_free_mib"}."""
    pin = _Pinned()
    lut, av, req = _lut(inp["lut"], pin), _avail(inp["avail"], pin), _requests(inp["requests"], pin)
    n = int(inp["requests"]["n_requests"])
    ws = _arr(wave_start, np.int32)
    G, S = int(inp["avail"]["n_gpus"]), int(inp["avail"]["n_steps"])
    freq, batch, mem = np.zeros(G, np.int32), np.zeros(G, np.int32), np.zeros((G, S), np.int32)
    buf = (_Dispatch * max(n, 1))()
    rc = lib().festina_oracle_dispatch_waves(C.byref(lut), C.byref(av), C.byref(req), len(ws) - 1, _p(ws),
                                             _p(freq), _p(batch), _p(mem), C.cast(buf, C.c_void_p))
    if rc != 0:
        raise ValueError("oracle rejected the wave dispatch arguments")
    a = np.frombuffer(buf, dtype=np.dtype([("gpu", "<i4"), ("freq_level", "<i4"), ("sm_level", "<i4"),
                                           ("phase", "<i4"), ("energy", "<f8")]), count=n)
    return ((a["gpu"].copy(), a["freq_level"].copy(), a["sm_level"].copy(), a["phase"].copy(), a["energy"].copy()),
            {"freq_cur": freq, "batch": batch, "mem_free_mib": mem})


def transfer_costs(inp: dict) -> np.ndarray:
    """Oracle transfer-cost matrix e_uv (ms, float64, [G][G]) of App. F's device mapping."""
    pin = _Pinned()
    t = _transfer(inp["transfer"], pin)
    G = int(inp["transfer"]["n_gpus"])
    out = np.empty((G, G), np.float64)
    if lib().festina_oracle_transfer_costs(C.byref(t), int(inp["n_models"]), _p(out)) != 0:
        raise ValueError("oracle rejected the transfer arguments")
    return out


def request_moves(inp: dict):
    """Oracle per-request decisions (finish in place / move with KV / move and recompute).

    Returns (decision int32, remaining_ms float64, migrate_ms float64)."""
    pin = _Pinned()
    lut, t = _lut(inp["lut"], pin), _transfer(inp["transfer"], pin)
    pl, mv = inp["plan"], inp["moves"]
    plan = _Plan(pin(pl["dest"], np.int32), pin(pl["freq_cur"], np.int32), pin(pl["sm_cur"], np.int32),
                 pin(pl["batch"], np.int32))
    moves = _Moves(int(mv["n_requests"]), pin(mv["src"], np.int32), pin(mv["model"], np.int32),
                   pin(mv["context_tokens"], np.int32), pin(mv["remaining_tokens"], np.int32),
                   pin(mv["kv_kib"], np.int32), pin(mv["token_kib"], np.int32))
    n = int(mv["n_requests"])
    dec = np.empty(max(n, 1), np.int32)
    rem = np.empty(max(n, 1), np.float64)
    mig = np.empty(max(n, 1), np.float64)
    if lib().festina_oracle_request_moves(C.byref(lut), C.byref(t), C.byref(plan), C.byref(moves), _p(dec), _p(rem),
                                          _p(mig)) != 0:
        raise ValueError("oracle rejected the request-move arguments")
    return dec[:n], rem[:n], mig[:n]
