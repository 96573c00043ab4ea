#!/usr/bin/env python3
"""Benchmark of the batched energy-aware placement and migration search on one GPU.

One step = one pass of the whole hot path over one batch of synthetic input:
  * placement search of the phase-aware bursty workload: 262,144 requests in 64
    arrival waves over 1,024 GPUs, 32 models, 8 SM x 16 frequency levels, capped
    prefill/decode SM splits (every (hosting GPU, SM level, frequency level)
    candidate of every request is scored, masked by SLO and reduced to the
    least-energy feasible one);
  * consolidation scoring of a 2,048-GPU fleet: all 4,192,256 ordered
    source -> destination pairs and the per-source best destination.
Inputs are resident in device memory before the timed region.  The two searches are
independent, so the consolidation scoring is enqueued on a second stream (default priority)
beside the placement search; the timed region ends when both streams have drained.  The
metric is candidate evaluations per second (placement candidates plus migration pairs).

Also reported: the roofline position of the dominant kernel (placement scoring,
timed alone with HIP events recorded around it inside the library), and the CPU
oracle timed on a bounded sample of the same workload on this host.  Outside the
timed steps, ``next_rows`` measures the local schedulers' SM/frequency sweep over
1,024 GPUs x 64 epochs of task batches (one kernel per call), and the preferred
configuration of every LLM instance on a 2,048-GPU fleet plus the fleet's energy waste
ratio, the paper's own current-frequency dispatcher (65,536 requests, 512 GPUs), and the
transfer plan of a 2,048-GPU reconfiguration (cost matrix, per-request moves), the same
way.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu-baseline]
       python bench.py --per-config     (also one JSON line per configuration before the step line;
                                         the step line always carries them as "per_config")
"""
from __future__ import annotations

import argparse
import ctypes as C
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

# MI355X: 256 CUs x 4 SIMD x 16 lanes, 2.4 GHz peak engine clock -> 64 VALU lane-ops/clock/CU
N_CU = 256
LANES_PER_CU_CLOCK = 64
SCLK_HZ = 2.4e9
VALU_PEAK = N_CU * LANES_PER_CU_CLOCK * SCLK_HZ            # 39.32e12 lane-ops/s
HBM_PEAK = 8.0e12                                           # B/s

# Least VALU work per candidate of any exhaustive search: divided by the
# request's Lout, a candidate's energy is Pp * (TTFT / Lout) + Pd * TBT, one fused
# multiply-add of a request term and two GPU terms, and a three-way min folds two
# candidates into the running minimum, half an instruction each.  SLO masks, power terms,
# the per-request scale and the index of the winner are shared or recovered once per
# request or GPU, so they are not counted.  The count runs over distinct candidates: the
# cells of a capped GPU above max(cap_pf, cap_dc) repeat lower cells and need no work.
OPS_PER_CANDIDATE = 1.5
# Migration pair: two budget compares, level-mask AND and test, self test, lowest set bit,
# u_s + u_d, two multiplies, subtract, FMA, compare with the best, three selects.
OPS_PER_PAIR = 15

TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_score_config4_traffic.json")
COUNTERS_FILE = os.path.join(ROOT, "profiles", "k_score_config4_counters.json")
KERNEL_SRC = os.path.join(ROOT, "paper_2606_30391_amd", "csrc", "festina.hip")
SWEEP_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_sweep_traffic.json")
SWEEP_SRC = os.path.join(ROOT, "paper_2606_30391_amd", "csrc", "sweep.hip")
TRANSFER_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_transfer_costs_traffic.json")
TRANSFER_SRC = os.path.join(ROOT, "paper_2606_30391_amd", "csrc", "transfer.hip")
DISPATCH_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_dispatch_traffic.json")
DISPATCH_WAVES_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_dispatch_waves_traffic.json")
MIGRATE_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_migrate_traffic.json")
DISPATCH_SRC = os.path.join(ROOT, "paper_2606_30391_amd", "csrc", "dispatch.hip")
PREFERRED_TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_preferred_traffic.json")
PREFERRED_SRC = os.path.join(ROOT, "paper_2606_30391_amd", "csrc", "preferred.hip")
# Sweep, per (task, SM level, frequency level) cell: one compare of the latency with the
# slack; per (task, frequency level): the SM share add and two FMAs (power, energy).
OPS_PER_SWEEP_CELL = 1
OPS_PER_SWEEP_TASK_LEVEL = 3


# ------------------------------------------------------------------ HIP events (ctypes)
class Hip:
    def __init__(self):
        self.L = C.CDLL("libamdhip64.so")
        self.L.hipEventCreateWithFlags.argtypes = [C.POINTER(C.c_void_p), C.c_uint]
        self.L.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        self.L.hipEventSynchronize.argtypes = [C.c_void_p]
        self.L.hipEventDestroy.argtypes = [C.c_void_p]
        self.L.hipEventRecord.argtypes = [C.c_void_p, C.c_void_p]

    # timing-only events: no system-scope fence (cache writeback/invalidate) on record
    DISABLE_SYSTEM_FENCE = 0x20000000

    def event(self):
        e = C.c_void_p()
        rc = self.L.hipEventCreateWithFlags(C.byref(e), self.DISABLE_SYSTEM_FENCE)
        if rc != 0:
            raise RuntimeError(f"hipEventCreate failed ({rc})")
        return e.value

    def elapsed_ms(self, a, b):
        self.L.hipEventSynchronize(C.c_void_p(b))
        ms = C.c_float()
        rc = self.L.hipEventElapsedTime(C.byref(ms), C.c_void_p(a), C.c_void_p(b))
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(ms.value)

    def destroy(self, e):
        self.L.hipEventDestroy(C.c_void_p(e))

    def record(self, e, stream):
        rc = self.L.hipEventRecord(C.c_void_p(e), C.c_void_p(stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")


# ------------------------------------------------------------------ work counts
def placement_candidates(inp, sel=None):
    """sum over (valid) requests of |hosts(model)| * NS * NF."""
    lut, gp, rq = inp["lut"], inp["gpus"], inp["requests"]
    M = lut["n_models"]
    res = np.asarray(gp["resident"], np.uint32)
    hosts = np.array([int(((res[:, m // 32] >> np.uint32(m % 32)) & 1).sum()) for m in range(M)])
    model = rq["model"] if sel is None else rq["model"][sel]
    ok = (model >= 0) & (model < M)
    return int(hosts[model[ok]].sum()) * lut["n_sm"] * lut["n_freq"]


def distinct_candidates(inp):
    """Candidates that are not repeats: a capped GPU's SM levels above max(cap_pf, cap_dc)
    repeat that level's cells exactly at a higher index (never the lowest-index minimum), so
    only levels 0..max(cap_pf, cap_dc) of each hosting GPU count."""
    lut, gp, rq = inp["lut"], inp["gpus"], inp["requests"]
    M, NS, NF = lut["n_models"], lut["n_sm"], lut["n_freq"]
    G = gp["n_gpus"]
    res = np.asarray(gp["resident"], np.uint32)
    if gp.get("cap_pf") is not None or gp.get("cap_dc") is not None:
        cp = np.full(G, NS - 1) if gp.get("cap_pf") is None else np.asarray(gp["cap_pf"], np.int64)
        cd = np.full(G, NS - 1) if gp.get("cap_dc") is None else np.asarray(gp["cap_dc"], np.int64)
        levels = np.minimum(np.maximum(cp, cd), NS - 1) + 1
    else:
        levels = np.full(G, NS)
    per_model = np.array([int(levels[((res[:, m // 32] >> np.uint32(m % 32)) & 1) == 1].sum()) for m in range(M)])
    model = rq["model"]
    ok = (model >= 0) & (model < M)
    return int(per_model[model[ok]].sum()) * NF


def placement_bytes(inp):
    """Algorithmic HBM bytes of one placement call: request fields in, results out,
    GPU state and each model's tables read once."""
    lut, gp, rq = inp["lut"], inp["gpus"], inp["requests"]
    R, G, W, M = rq["n_requests"], gp["n_gpus"], gp["n_waves"], lut["n_models"]
    req_in = R * (4 * 6)                       # model, wave, prompt, pred, two SLOs
    out = R * (4 + 1 + 4)
    state = W * G * 4 + G * (4 + 4 * ((M + 31) // 32) + (2 if gp.get("cap_pf") is not None else 0))
    tables = 2 * lut["pf"].nbytes
    return req_in + out + state + tables


def sweep_bytes(inp):
    """Algorithmic HBM bytes of one sweep call: every batch's count and GPU terms, every task
    slot's four fields, the results, and the tables read once."""
    bt, lut = inp["batches"], inp["lut"]
    B, T = bt["n_batches"], bt["max_tasks"]
    return B * 12 + B * T * 16 + B * (4 + 1 + 4) + B * T * 4 + 2 * lut["pf"].nbytes


def sweep_work(inp):
    """(cells, algorithmic VALU lane-ops) of one sweep call."""
    bt, lut = inp["batches"], inp["lut"]
    n = np.asarray(bt["n_tasks"])
    tasks = int(n[(n >= 0) & (n <= bt["max_tasks"])].sum())
    cells = tasks * lut["n_sm"] * lut["n_freq"]
    return cells, cells * OPS_PER_SWEEP_CELL + tasks * lut["n_freq"] * OPS_PER_SWEEP_TASK_LEVEL


def src_hash(path=KERNEL_SRC):
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def load_traffic(path=TRAFFIC_FILE, src=KERNEL_SRC):
    """HBM bytes per launch of a kernel from the committed counter runs, or None when
    the kernel source changed since they were taken."""
    try:
        d = json.load(open(path))
    except (OSError, ValueError):
        return None
    if d.get("kernel_src_sha256_16") != src_hash(src):
        return None
    return d.get("hbm_bytes_per_launch")


def load_counters(path=COUNTERS_FILE, src=KERNEL_SRC):
    """VALU issue figures of the scoring kernel from the committed counter run, or None when
    the kernel source changed since it was taken."""
    try:
        d = json.load(open(path))
    except (OSError, ValueError):
        return None
    if d.get("kernel_src_sha256_16") != src_hash(src):
        return None
    return {"valu_issue_busy": d["valu_issue_busy"],
            "valu_lane_ops_per_distinct_candidate": d["valu_lane_ops_per_distinct_candidate"],
            "sclk_ghz_effective": d["sclk_ghz_effective"]}


def timed_calls(hip, torch, fn, calls, warmup):
    """Mean duration (ms) of fn() over `calls` calls, HIP events recorded around each."""
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream().cuda_stream
    evs = [(hip.event(), hip.event()) for _ in range(calls)]
    for a, b in evs:
        hip.record(a, st)
        fn()
        hip.record(b, st)
    torch.cuda.synchronize()
    ms = float(np.mean([hip.elapsed_ms(a, b) for a, b in evs]))
    for a, b in evs:
        hip.destroy(a)
        hip.destroy(b)
    return ms


def timed_batch(hip, torch, fn, calls, head=None):
    """Mean duration (ms) of fn() over `calls` back-to-back calls, one HIP event pair around
    the batch.  `head` enqueues work first so that the device is still busy while the host
    enqueues the batch (the calls then run back to back, not at the host's pace)."""
    fn()
    torch.cuda.synchronize()
    st = torch.cuda.current_stream().cuda_stream
    a, b = hip.event(), hip.event()
    if head is not None:
        head()
    hip.record(a, st)
    for _ in range(calls):
        fn()
    hip.record(b, st)
    torch.cuda.synchronize()
    ms = hip.elapsed_ms(a, b) / calls
    hip.destroy(a)
    hip.destroy(b)
    return ms


def preferred_row(F, W, hip, torch, with_cpu, calls=200, warmup=10):
    """Preferred configurations of every LLM instance (one launch) and the fleet's EWR
    (two launches): durations from HIP events around each call, roofline position, and
    the oracle on the same instances."""
    inp = W.make_llms()
    dp = F.DevicePreferred(inp, "cuda")
    pref_ms = timed_calls(hip, torch, dp.run_preferred, calls, warmup)
    ewr_ms = timed_calls(hip, torch, dp.run_ewr, calls, warmup)
    q, lut = inp["llms"], inp["lut"]
    G, K = q["n_gpus"], q["max_inst"]
    live = int((np.arange(K)[None, :] < q["n_inst"][:, None]).sum())
    cells = 2 * live * lut["n_sm"] * lut["n_freq"]           # both phases of every instance
    nbytes = G * K * (6 * 4) + G * 8 + G * K * (4 * 4 + 7 * 4 + 1) + 2 * lut["pf"].nbytes
    row = {
        "workload": ("preferred configuration of every LLM instance on a 2048-GPU fleet (1-4 instances "
                     "per GPU, 32 models, 8 SM x 16 freq levels, both phases) + the fleet's EWR"),
        "instances": live, "cells": cells, "preferred_kernel_ms": pref_ms, "ewr_ms": ewr_ms,
        "cells_per_s": cells / (pref_ms * 1e-3),
        "roofline": {"kernel": "k_preferred", "bound": "hbm", "achieved": nbytes / (pref_ms * 1e-3) / 1e9,
                     "peak": HBM_PEAK / 1e9, "unit": "GB/s", "frac": nbytes / (pref_ms * 1e-3) / HBM_PEAK,
                     "traffic": load_traffic(PREFERRED_TRAFFIC_FILE, PREFERRED_SRC), "algorithmic_bytes": nbytes},
        "cpu_baseline": None,
    }
    if with_cpu:
        import oracle
        got = dp.results()
        t0 = time.perf_counter()
        ref = oracle.preferred(inp)
        t1 = time.perf_counter()
        row["cpu_baseline"] = {
            "value": cells / (t1 - t0), "unit": "cells/s", "cores": 1, "kind": "oracle",
            "sample": f"all {live} instances ({t1 - t0:.3f} s); single-threaded C, float64, gcc -O2",
            "agreement": {"flags_equal": float(np.mean(got["feasible"] == ref["feasible"])),
                          "cells_equal": float(np.mean((got["sm_p"] == ref["sm_p"]) & (got["f_p"] == ref["f_p"])
                                                       & (got["sm_d"] == ref["sm_d"]) & (got["f_d"] == ref["f_d"])))}}
    return row


def dispatch_row(F, W, hip, torch, with_cpu, calls=200, warmup=10):
    """The paper's own dispatcher (one operating point per GPU, 2% stability tie-break,
    F_max fallback): call time from HIP events, roofline position, and the oracle."""
    inp = W.make_dispatch()
    dd = F.DeviceDispatch(inp, "cuda")
    ms = timed_calls(hip, torch, dd.run, calls, warmup)
    lut, av, rq = inp["lut"], inp["avail"], inp["requests"]
    M, G, R, S = lut["n_models"], av["n_gpus"], rq["n_requests"], av["n_steps"]
    res = np.asarray(av["resident"], np.uint32)
    hosts = np.array([int(((res[:, m // 32] >> np.uint32(m % 32)) & 1).sum()) for m in range(M)])
    evals = int(hosts[rq["model"]].sum())                    # (request, hosting GPU) operating points
    nbytes = R * (5 * 4) + R * (3 * 4 + 1 + 4) + G * (4 * 3 + 4 * ((M + 31) // 32) + S * 12) + M * 4 \
        + 2 * lut["pf"].nbytes
    row = {
        "workload": ("paper's current-frequency dispatcher: 65536 requests, 512 GPUs (1-4 of 32 models each), "
                     "4-step free-memory profiles, 8 SM x 16 freq levels"),
        "requests": R, "evaluations": evals, "kernel_ms": ms, "evaluations_per_s": evals / (ms * 1e-3),
        "roofline": {"kernel": "k_dispatch", "bound": "hbm", "achieved": nbytes / (ms * 1e-3) / 1e9,
                     "peak": HBM_PEAK / 1e9, "unit": "GB/s", "frac": nbytes / (ms * 1e-3) / HBM_PEAK,
                     "traffic": load_traffic(DISPATCH_TRAFFIC_FILE, DISPATCH_SRC), "algorithmic_bytes": nbytes},
        "cpu_baseline": None,
    }
    if with_cpu:
        import oracle
        got = dd.results()
        t0 = time.perf_counter()
        ref = oracle.dispatch(inp)
        t1 = time.perf_counter()
        row["cpu_baseline"] = {
            "value": evals / (t1 - t0), "unit": "evaluations/s", "cores": 1, "kind": "oracle",
            "sample": f"all {R} requests ({t1 - t0:.3f} s); single-threaded C, float64, gcc -O2",
            "agreement": {"all_outputs_equal": float(np.mean(
                (got[0] == ref[0]) & (got[1] == ref[1]) & (got[2] == ref[2]) & (got[3] == ref[3])
                & (got[4] == ref[4].astype(np.float32))))}}
    return row


def dispatch_waves_row(F, W, hip, torch, with_cpu, calls=100, warmup=5):
    """The same dispatcher over configuration 4's 64 arrival waves (262,144 requests, 1,024
    GPUs), each wave committed to the GPUs' batch, memory and frequency before the next:
    call time from HIP events and the oracle."""
    inp = W.make_dispatch_waves(n_requests=262144, n_gpus=1024, n_waves=64)
    ws = inp["wave_start"]
    dd = F.DeviceDispatch(inp, "cuda")
    ms = timed_calls(hip, torch, lambda: dd.run_waves(ws), calls, warmup)
    R, G, n_waves = inp["requests"]["n_requests"], inp["avail"]["n_gpus"], len(ws) - 1
    launches = 3 + int(np.count_nonzero(np.diff(ws)))
    lut, av = inp["lut"], inp["avail"]
    M, S = lut["n_models"], av["n_steps"]
    per_wave = R // n_waves
    # per wave launch: its requests' fields and results, the carried state and the previous
    # wave's commits read once, the folded state written and the next commits cleared, the
    # two tables once
    nbytes = per_wave * (5 * 4 + 3 * 4 + 1 + 4) + G * (4 + 4 * ((M + 31) // 32) + 8 * S) \
        + 2 * G * ((8 + 4 * S) + (8 + 8 * S)) + M * 4 + 2 * lut["pf"].nbytes
    wave_ms = ms / n_waves
    row = {
        "workload": ("paper's current-frequency dispatcher over configuration 4's arrival waves: 262144 requests "
                     "in 64 waves of 4096, 1024 GPUs (1-4 of 32 models each), each wave committed before the next"),
        "requests": R, "waves": n_waves, "launches": launches, "call_ms": ms, "requests_per_s": R / (ms * 1e-3),
        "us_per_wave": ms * 1e3 / n_waves,
        "roofline": {"kernel": "k_dispatch (one wave)", "bound": "hbm", "achieved": nbytes / (wave_ms * 1e-3) / 1e9,
                     "peak": HBM_PEAK / 1e9, "unit": "GB/s", "frac": nbytes / (wave_ms * 1e-3) / HBM_PEAK,
                     "traffic": load_traffic(DISPATCH_WAVES_TRAFFIC_FILE, DISPATCH_SRC), "algorithmic_bytes": nbytes,
                     "note": "latency-bound: a chain of dependent loads and a launch per wave"},
        "cpu_baseline": None,
    }
    if with_cpu:
        import oracle
        got, st = dd.results(), dd.state_results()
        t0 = time.perf_counter()
        ref, ref_st = oracle.dispatch_waves(inp, ws)
        t1 = time.perf_counter()
        row["cpu_baseline"] = {
            "value": R / (t1 - t0), "unit": "requests/s", "cores": 1, "kind": "oracle",
            "sample": f"all {R} requests, {n_waves} waves ({t1 - t0:.3f} s); single-threaded C, float64, gcc -O2",
            "agreement": {"all_outputs_equal": float(np.mean(
                (got[0] == ref[0]) & (got[1] == ref[1]) & (got[2] == ref[2]) & (got[3] == ref[3])
                & (got[4] == ref[4].astype(np.float32)))),
                "final_state_equal": bool(all(np.array_equal(st[k], ref_st[k]) for k in ref_st))}}
    return row


def transfer_row(F, W, hip, torch, with_cpu, calls=200, warmup=10):
    """The transfer plan (App. F): the dense device-mapping cost matrix (the dominant,
    store-bound kernel) and the in-flight requests' decisions."""
    inp = W.make_transfer()
    dt = F.DeviceTransfer(inp, "cuda")
    cost_ms = timed_calls(hip, torch, dt.run_costs, calls, warmup)
    moves_ms = timed_calls(hip, torch, dt.run_moves, calls, warmup)
    tr, M, Q = inp["transfer"], inp["n_models"], inp["moves"]["n_requests"]
    G = tr["n_gpus"]
    nbytes = G * G * 4 + G * (4 * ((M + 31) // 32) + 8) + M * 4     # the matrix written, the fleet read
    row = {
        "workload": "transfer plan of a 2048-GPU reconfiguration: 2048 x 2048 cost matrix, 16384 in-flight requests",
        "pairs": G * G, "requests": Q, "cost_kernel_ms": cost_ms, "moves_ms": moves_ms,
        "pairs_per_s": G * G / (cost_ms * 1e-3),
        "roofline": {"kernel": "k_transfer_costs", "bound": "hbm", "achieved": nbytes / (cost_ms * 1e-3) / 1e9,
                     "peak": HBM_PEAK / 1e9, "unit": "GB/s", "frac": nbytes / (cost_ms * 1e-3) / HBM_PEAK,
                     "traffic": load_traffic(TRANSFER_TRAFFIC_FILE, TRANSFER_SRC), "algorithmic_bytes": nbytes},
        "cpu_baseline": None,
    }
    if with_cpu:
        import oracle
        c, d, r, m = dt.results()
        t0 = time.perf_counter()
        oc = oracle.transfer_costs(inp)
        t1 = time.perf_counter()
        od, orem, omig = oracle.request_moves(inp)
        row["cpu_baseline"] = {
            "value": G * G / (t1 - t0), "unit": "pairs/s", "cores": 1, "kind": "oracle",
            "sample": f"the whole {G} x {G} matrix ({t1 - t0:.3f} s); single-threaded C, float64, gcc -O2",
            "agreement": {"costs_equal": float(np.mean(oc.astype(np.float32) == c)),
                          "decisions_equal": float(np.mean(od == d))}}
    return row


def sweep_row(F, W, hip, torch, with_cpu, calls=200, warmup=10):
    """The local SM/frequency sweep: kernel time from HIP events around each call (one
    launch per call), its roofline position, and the oracle on the same batches."""
    inp = W.make_sweep()
    ds = F.DeviceSweep(inp, "cuda")
    ms = timed_calls(hip, torch, ds.run, calls, warmup)
    bt = inp["batches"]
    cells, ops = sweep_work(inp)
    nbytes = sweep_bytes(inp)
    row = {
        "workload": ("local SM/frequency sweep: 1024 GPUs x 64 epochs = 65536 task batches of up to 8 "
                     "prefill units / decode steps, 32 models, 8 SM x 16 freq levels"),
        "batches": int(bt["n_batches"]), "tasks": int(np.asarray(bt["n_tasks"]).sum()),
        "cells": cells, "kernel_ms": ms, "cells_per_s": cells / (ms * 1e-3),
        "roofline": {"kernel": "k_sweep_8x16", "bound": "hbm", "achieved": nbytes / (ms * 1e-3) / 1e9,
                     "peak": HBM_PEAK / 1e9, "unit": "GB/s", "frac": nbytes / (ms * 1e-3) / HBM_PEAK,
                     "traffic": load_traffic(SWEEP_TRAFFIC_FILE, SWEEP_SRC), "algorithmic_bytes": nbytes,
                     "valu_frac_algorithmic": ops / (ms * 1e-3) / VALU_PEAK},
        "cpu_baseline": None,
    }
    if with_cpu:
        import oracle
        gl, gf, ge, gt = ds.results()
        t0 = time.perf_counter()
        ol, of, oe, ot = oracle.sweep(inp)
        t1 = time.perf_counter()
        row["cpu_baseline"] = {
            "value": cells / (t1 - t0), "unit": "cells/s", "cores": 1, "kind": "oracle",
            "sample": f"all {bt['n_batches']} batches ({t1 - t0:.3f} s); single-threaded C, float64, gcc -O2",
            "agreement": {"flags_equal": float(np.mean(of == gf)), "levels_equal": float(np.mean(ol == gl)),
                          "task_sm_equal": float(np.mean(ot == gt))}}
    return row


# ------------------------------------------------------------------ CPU baseline (oracle)
_WORKER_INP = None


def _worker_init(kind, inp):
    """Pool worker set-up (a fresh interpreter, no GPU): keep the inputs, load the oracle."""
    global _WORKER_INP, _WORKER_KIND
    import oracle
    oracle.lib()
    _WORKER_INP, _WORKER_KIND = inp, kind


def _worker_chunk(sel):
    import oracle
    if _WORKER_KIND == "placement":
        oracle.score_placements(_WORKER_INP, sel)
    else:
        oracle.score_migrations(_WORKER_INP, sel)
    return len(sel)


def oracle_all_cores(kind, inp, sel, workers):
    """The unchanged single-threaded oracle on the same sampled requests (kind "placement")
    or source GPUs ("migration"), split into chunks over `workers` spawned processes; wall
    time of the chunks only (inputs are handed to the workers before the clock starts)."""
    import multiprocessing as mp
    chunks = np.array_split(sel, workers * 8)
    with mp.get_context("spawn").Pool(workers, initializer=_worker_init, initargs=(kind, inp)) as pool:
        pool.map_async(_worker_chunk, [c[:1] for c in chunks[:workers]]).get(timeout=300)   # every worker warm
        t0 = time.perf_counter()
        done = sum(pool.map_async(_worker_chunk, chunks).get(timeout=300))
        t1 = time.perf_counter()
    assert done == len(sel)
    return t1 - t0


def host_cpu():
    """The host's CPU model (first `model name` of /proc/cpuinfo) and its logical CPU counts."""
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "nproc": os.cpu_count(), "usable": len(os.sched_getaffinity(0))}


def best_of(fn, n=3):
    """Least wall time of n calls of fn()."""
    best = None
    for _ in range(n):
        t0 = time.perf_counter()
        fn()
        dt = time.perf_counter() - t0
        best = dt if best is None else min(best, dt)
    return best


def cpu_per_config(W):
    """The single-threaded oracle on the whole of configurations 1-3 (placement) and 5
    (consolidation), best of 3 runs each."""
    import oracle
    out = {}
    for cfg in (1, 2, 3, 5):
        if cfg < 5:
            inp = W.make_placement(cfg)
            work = placement_candidates(inp)
            t = best_of(lambda: oracle.score_placements(inp))
            what = f"all {inp['requests']['n_requests']} requests, {work} candidates"
        else:
            inp = W.make_fleet()
            G = inp["fleet"]["n_gpus"]
            work = G * (G - 1)
            t = best_of(lambda: oracle.score_migrations(inp))
            what = f"all {work} ordered pairs of {G} GPUs"
        out[str(cfg)] = {"value": work / t, "unit": "candidate evaluations/s", "cores": 1, "seconds": t,
                         "sample": what + ", best of 3"}
    return out


def cpu_baseline(place_inp, fleet_inp, gpu_place, gpu_mig, W, stride=4):
    import oracle
    R = place_inp["requests"]["n_requests"]
    sel = np.arange(0, R, stride, dtype=np.int32)
    t0 = time.perf_counter()
    oc, of, oe = oracle.score_placements(place_inp, sel)
    t1 = time.perf_counter()
    ob, osv, ok = oracle.score_migrations(fleet_inp)
    t2 = time.perf_counter()
    cand = placement_candidates(place_inp, sel)
    G = fleet_inp["fleet"]["n_gpus"]
    pairs = G * (G - 1)
    gc, gf, _ = gpu_place
    gb = gpu_mig[0]
    workers = max(1, min(16, os.cpu_count() or 1))        # the machine's CPU share for one GPU
    t_all = oracle_all_cores("placement", place_inp, sel, workers)
    t_mig = oracle_all_cores("migration", fleet_inp, np.arange(G, dtype=np.int32), workers)
    return {
        "value": (cand + pairs) / ((t1 - t0) + (t2 - t1)),
        "unit": "candidate evaluations/s",
        "cores": 1,
        "kind": "oracle",
        "sample": (f"every {stride}th request of the placement workload ({len(sel)} requests, {cand} "
                   f"candidates, {t1 - t0:.2f} s) + all {pairs} migration pairs ({t2 - t1:.2f} s); "
                   f"single-threaded C, float64, gcc -O2"),
        "all_cores": {"value": (cand + pairs) / (t_all + t_mig), "cores": workers,
                      "sample": f"the same {len(sel)} placement requests ({t_all:.2f} s) and all {pairs} migration "
                                f"pairs ({t_mig:.2f} s), each in chunks over {workers} processes",
                      "placement": {"value": cand / t_all, "seconds": t_all},
                      "migration": {"value": pairs / t_mig, "seconds": t_mig}},
        "per_config": cpu_per_config(W),
        "host": host_cpu(),
        "agreement": {"placement_flags_equal": float(np.mean(of == gf[sel])),
                      "placement_choice_equal": float(np.mean(oc == gc[sel])),
                      "migration_dst_equal": float(np.mean(ob == gb))},
    }


# ------------------------------------------------------------------ main
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--per-config", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="first print one line comparing the step (consolidation forked onto a second "
                         "stream and joined back) launched eagerly and replayed from one HIP graph")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the run, copy MIB MiB device-to-device 5 times (a plain copy of known "
                         "size, to scale the HBM byte counters)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} (WORLD_SIZE {world}) is not "
              f"supported: requests are independent, so the search shards by requests across devices "
              f"without communication, and one device's share is what this measures.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_30391_amd import festina as F
    from paper_2606_30391_amd import workloads as W

    F.lib()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    hip = Hip()

    configs = per_config(F, W, hip, torch, verbose=args.per_config)
    if args.graph:
        graph_compare(F, W, torch)

    place = W.make_placement(4)
    fleet = W.make_fleet()
    dp = F.DevicePlacement(place, "cuda")
    dm = F.DeviceMigration(fleet, "cuda")
    torch.cuda.synchronize()

    n_cand = placement_candidates(place)
    n_distinct = distinct_candidates(place)
    G = fleet["fleet"]["n_gpus"]
    n_pairs = G * (G - 1)

    side = torch.cuda.Stream()         # default priority, like the current stream
    for _ in range(args.warmup):
        dp.run()
        dm.run(side)
    torch.cuda.synchronize()

    # Timed steps: placement on the current stream, consolidation on the side stream; events
    # are recorded around the scoring kernel only, in every SAMPLE-th step (each record costs
    # a few microseconds of stream time); the consolidation call is timed afterwards on its
    # own, as a batch.
    K = args.steps
    SAMPLE = 8
    evs = [[hip.event() for _ in range(2)] for _ in range(0, K, SAMPLE)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        dp.run(events=evs[i // SAMPLE] if i % SAMPLE == 0 else None)
        dm.run(side)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    score_ms = float(np.mean([hip.elapsed_ms(e[0], e[1]) for e in evs]))
    for e in evs:
        for x in e:
            hip.destroy(x)
    mig_ms = timed_batch(hip, torch, dm.run, 50, head=lambda: [dp.run() for _ in range(4)])

    step_s = (t1 - t0) / K
    value = (n_cand + n_pairs) / step_s
    achieved = n_distinct * OPS_PER_CANDIDATE / (score_ms * 1e-3)
    gpu_place = dp.results()
    gpu_mig = dm.results()

    counters = load_counters()
    line = {
        "metric": "candidate evaluations/sec + % of HBM/VALU roofline, 1 MI355X",
        "value": value,
        "unit": "candidate evaluations/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": step_s * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        # the same step counted over distinct candidates only (a capped GPU's SM levels above
        # max(cap_pf, cap_dc) repeat lower cells and are not evaluated)
        "value_distinct": (n_distinct + n_pairs) / step_s,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": ("phase-aware bursty placement (262144 requests in 64 waves, 1024 GPUs, 32 models, "
                         "8 SM x 16 freq levels, capped prefill/decode SM splits) + consolidation scoring "
                         "(2048 GPUs, 4192256 ordered pairs)"),
            "placement_candidates": n_cand,
            "distinct_placement_candidates": n_distinct,
            "migration_pairs": n_pairs,
            "parallelism": "single GPU",
        },
        "roofline": {
            "kernel": "k_score (placement scoring + fused argmin)",
            "bound": "alu",
            "achieved": achieved / 1e12,
            "peak": VALU_PEAK / 1e12,
            "unit": "T VALU lane-ops/s",
            "frac": achieved / VALU_PEAK,
            "traffic": load_traffic(),
            "ops_per_candidate": OPS_PER_CANDIDATE,
            "candidates_counted": "distinct (capped GPUs' repeated SM levels excluded)",
            "kernel_ms": score_ms,
            "hbm_frac_algorithmic": placement_bytes(place) / (score_ms * 1e-3) / HBM_PEAK,
            "counters": counters,
            # the same fraction against the peak at the engine clock the counter run measured
            "frac_at_measured_sclk": (None if counters is None else
                                      achieved / (VALU_PEAK * counters["sclk_ghz_effective"] * 1e9 / SCLK_HZ)),
        },
        # the consolidation scoring (the second scoring call), timed alone as a batch of calls
        "migration": {
            "kernel": "k_fleet + k_migrate (consolidation pair scoring + fused per-source argmax)",
            "pairs": n_pairs, "call_ms": mig_ms,
            "roofline": {"bound": "alu", "achieved": n_pairs * OPS_PER_PAIR / (mig_ms * 1e-3) / 1e12,
                         "peak": VALU_PEAK / 1e12, "unit": "T VALU lane-ops/s",
                         "frac": n_pairs * OPS_PER_PAIR / (mig_ms * 1e-3) / VALU_PEAK,
                         "ops_per_pair": OPS_PER_PAIR,
                         "traffic": load_traffic(MIGRATE_TRAFFIC_FILE, KERNEL_SRC)},   # both launches
        },
        "kernels_ms": {"k_score": score_ms, "k_score_candidates_per_s": n_cand / (score_ms * 1e-3),
                       "migration_call": mig_ms,
                       "migration_pairs_per_s_call": n_pairs / (mig_ms * 1e-3)},
        "per_config": configs,
        "cpu_baseline": None,
        "next_rows": {"sweep": sweep_row(F, W, hip, torch, not args.no_cpu_baseline),
                      "preferred": preferred_row(F, W, hip, torch, not args.no_cpu_baseline),
                      "dispatch": dispatch_row(F, W, hip, torch, not args.no_cpu_baseline),
                      "dispatch_waves": dispatch_waves_row(F, W, hip, torch, not args.no_cpu_baseline),
                      "transfer": transfer_row(F, W, hip, torch, not args.no_cpu_baseline)},
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(place, fleet, gpu_place, gpu_mig, W)
    print(json.dumps(line), flush=True)
    if args.copy_calibration > 0:
        n = args.copy_calibration * (1 << 20) // 4
        x = torch.ones(n, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        for _ in range(5):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n * 4, "copies": 5}), flush=True)


def graph_compare(F, W, torch, steps=200, rounds=3):
    """The bench step with the consolidation call forked onto a second stream and joined back,
    timed with events over `steps` steps: launched eagerly, and replayed from one HIP graph
    capture of the same step; `rounds` alternating rounds."""
    dp = F.DevicePlacement(W.make_placement(4), "cuda")
    dm = F.DeviceMigration(W.make_fleet(), "cuda")
    side = torch.cuda.Stream()

    def step():
        cur = torch.cuda.current_stream()
        side.wait_stream(cur)
        dp.run()
        dm.run(side)
        cur.wait_stream(side)

    def per_step_us(fn):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        s.record()
        for _ in range(steps):
            fn()
        e.record()
        torch.cuda.synchronize()
        return s.elapsed_time(e) / steps * 1e3

    for _ in range(10):
        step()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    eager, graph = [], []
    for _ in range(rounds):
        eager.append(per_step_us(step))
        graph.append(per_step_us(g.replay))
    print(json.dumps({"graph_compare": "config-4 placement + config-5 consolidation, forked and joined",
                      "steps": steps, "eager_us_per_step": eager, "graph_replay_us_per_step": graph}), flush=True)


def per_config(F, W, hip, torch, verbose=False):
    """Per configuration: call time, kernel time, rates and the kernel's VALU fraction (one
    JSON line each when verbose); returned as {config: {...}}."""
    out = {}
    for cfg in (1, 2, 3, 4, 5):
        if cfg < 5:
            inp = W.make_placement(cfg)
            dev = F.DevicePlacement(inp, "cuda")
            work = placement_candidates(inp)
            ops = distinct_candidates(inp) * OPS_PER_CANDIDATE
        else:
            inp = W.make_fleet()
            dev = F.DeviceMigration(inp, "cuda")
            G = inp["fleet"]["n_gpus"]
            work = G * (G - 1)
            ops = work * OPS_PER_PAIR
        reps = 10 if cfg == 4 else 50
        for _ in range(5):
            dev.run()
        torch.cuda.synchronize()
        # call time of the plain entry point (each event the timed one records inside the
        # call adds a few microseconds of stream time), then the kernel time from as many
        # calls of the timed entry point
        call_ms, kern_ms = [], []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            dev.run()
            b.record()
            torch.cuda.synchronize()
            call_ms.append(a.elapsed_time(b))
        ev = (hip.event(), hip.event())
        for _ in range(reps):
            dev.run(events=ev)
            torch.cuda.synchronize()
            kern_ms.append(hip.elapsed_ms(*ev))
        for e in ev:
            hip.destroy(e)
        cm, km = float(np.median(call_ms)), float(np.median(kern_ms))
        timed = "k_score (HIP events around the kernel inside the library)"
        if cfg == 5:
            # an event between the two migration kernels costs several microseconds of stream
            # time, more than the kernel itself: time a batch of whole calls instead
            km = timed_batch(hip, torch, dev.run, 50)
            timed = "k_fleet + k_migrate (batch of 50 calls, one event pair)"
        rec = {"work": work, "call_ms": cm, "kernel_ms": km, "kernel_timed": timed,
               "evals_per_s_call": work / (cm * 1e-3), "evals_per_s_kernel": work / (km * 1e-3),
               "valu_frac_kernel": ops / (km * 1e-3) / VALU_PEAK}
        out[str(cfg)] = rec
        if verbose:
            print(json.dumps({"config": cfg, **rec}), flush=True)
    return out


if __name__ == "__main__":
    main()
