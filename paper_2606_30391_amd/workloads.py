"""Seeded synthetic inputs for the batched placement and migration search.

This module only *draws inputs*: request features, GPU state snapshots, fleet
records and the offline profile tables (latency look-up tables).  It holds none
of the search itself: no output-length padding, no prompt bucketing, no power
or energy, no SLO test, no argmin.  Both the HIP path and the CPU oracle consume
what it returns, and neither shares any other code.

The paper's workloads (ShareGPT arrivals, Azure-derived prompt lengths) are not
available here; the laws below stand in for them.  Profile tables follow the
paper's look-up-table axes (Sec. 3.2.1: frequency, SM share, input length) with
a closed-form latency model per model:

* decode step (TBT):  a_m + c_m * b / (s * f)           rows = batch 1..32
* prefill (TTFT):     a_m + cp_m * 256 (p+1) / (s * f)   rows = 256-token prompt buckets
  (the tiny configuration has no prompts and uses the decode table for both)

Tables are evaluated in float64 and rounded once to float32; configurations 3-5
add independent multiplicative noise U(0.95, 1.05) per entry, so nothing may
assume monotone tables.
"""
from __future__ import annotations

import numpy as np

P0_W = 120.0              # static power, W
N_ROWS = 32               # table rows (batch 1..32, or prompt buckets of 256 tokens)
ROW_TOKENS = 256          # prompt tokens per prefill-table row (32 * 256 = 8192)
HBM_CAP_MIB = 288 * 1024  # one MI355X-class GPU: 288 GiB
SM_CAP_PERMILLE = 1000
MAX_INST = 4

CONFIG_SEED_BASE = 30391000

TTFT_SLO_SET = (100.0, 200.0, 400.0)
TBT_SLO_SET = (25.0, 50.0, 100.0)


def config_seed(n: int, extra: int = 0) -> int:
    """Seed of configuration n (1..5); extra parity seeds add 100, 200, 300."""
    return CONFIG_SEED_BASE + n + extra


# --------------------------------------------------------------------------- levels
def sm_levels(ns: int) -> np.ndarray:
    """SM-partition levels s_j = (j+1)/NS (tiny: {.25,.5,.75,1}; others: eighths)."""
    return ((np.arange(ns, dtype=np.float64) + 1.0) / ns).astype(np.float32)


def freq_levels(nf: int) -> np.ndarray:
    """Normalised frequency levels evenly spaced over [0.5, 1.0]."""
    if nf == 1:
        return np.ones(1, dtype=np.float32)
    return (0.5 + 0.5 * np.arange(nf, dtype=np.float64) / (nf - 1)).astype(np.float32)


# --------------------------------------------------------------------------- tables
def _latency_params(rng, m, prefill):
    a = rng.uniform(5.0, 20.0, m)
    c = rng.uniform(0.5, 3.0, m)
    cp = rng.uniform(0.02, 0.1, m) if prefill else None
    return a, c, cp


def _tables(rng, m, s, f, a, c, cp, noise):
    """Return (pf, dc) float32 [M][32][NS][NF] from the closed-form latency model."""
    sf = s.astype(np.float64)[:, None] * f.astype(np.float64)[None, :]        # [NS][NF]
    rows = np.arange(1, N_ROWS + 1, dtype=np.float64)                          # 1..32
    dc = a[:, None, None, None] + c[:, None, None, None] * rows[None, :, None, None] / sf[None, None]
    if cp is None:
        pf = dc.copy()
    else:
        tok = ROW_TOKENS * rows
        pf = a[:, None, None, None] + cp[:, None, None, None] * tok[None, :, None, None] / sf[None, None]
    if noise:
        dc = dc * rng.uniform(0.95, 1.05, dc.shape)
        pf = pf * rng.uniform(0.95, 1.05, pf.shape)
    return np.ascontiguousarray(pf, dtype=np.float32), np.ascontiguousarray(dc, dtype=np.float32)


def _lut(pf, dc, s, f, p0=P0_W):
    m, nr, ns, nf = pf.shape
    return {"n_models": m, "n_rows": nr, "n_sm": ns, "n_freq": nf,
            "sm_level": s, "freq_level": f, "pf": pf, "dc": dc, "p0_w": float(p0)}


def _resident_bits(models_per_gpu, m):
    """Pack per-GPU model lists into [G][ceil(M/32)] uint32 bitmasks."""
    g = len(models_per_gpu)
    words = (m + 31) // 32
    bits = np.zeros((g, words), dtype=np.uint32)
    for gi, ms in enumerate(models_per_gpu):
        for mm in ms:
            bits[gi, mm // 32] |= np.uint32(1) << np.uint32(mm % 32)
    return bits


def _lognormal_tokens(rng, mu, n, lo, hi):
    return np.clip(np.rint(rng.lognormal(mu, 1.0, n)), lo, hi).astype(np.int32)


def _distinct_models(rng, g, m, counts):
    return [np.sort(rng.choice(m, int(k), replace=False)) for k in counts[:g]]


# --------------------------------------------------------------------------- placement
def make_placement(config: int, seed: int | None = None, n_requests: int | None = None,
                   n_gpus: int | None = None) -> dict:
    """Placement inputs of configuration 1-4 (optionally with fewer requests/GPUs).

    Returned dict: {"lut": ..., "gpus": ..., "requests": ..., "meta": ...} of
    numpy arrays laid out as the C ABI expects (structure of arrays).
    """
    if seed is None:
        seed = config_seed(config)
    rng = np.random.default_rng(seed)
    if config == 1:
        M, G, R, NS, NF, W = 2, 8, 64, 4, 8, 1
    elif config == 2:
        M, G, R, NS, NF, W = 8, 64, 4096, 8, 16, 1
    elif config == 3:
        M, G, R, NS, NF, W = 32, 512, 65536, 8, 16, 1
    elif config == 4:
        M, G, R, NS, NF, W = 32, 1024, 262144, 8, 16, 64
    else:
        raise ValueError(f"placement configuration {config} does not exist")
    if n_requests is not None:
        R = int(n_requests)
    if n_gpus is not None:
        G = int(n_gpus)
    s, f = sm_levels(NS), freq_levels(NF)

    # --- profile tables
    a, c, cp = _latency_params(rng, M, prefill=(config != 1))
    pf, dc = _tables(rng, M, s, f, a, c, cp, noise=(config >= 3))
    lut = _lut(pf, dc, s, f)

    # --- GPU state
    cap_pf = cap_dc = None
    if config == 1:
        batch = rng.integers(0, 17, size=(W, G), dtype=np.int32)
        kdyn = rng.uniform(300.0, 500.0, G).astype(np.float32)
        models_per_gpu = [np.arange(M)] * G
        slo_m_ttft = np.full(M, 200.0)
        slo_m_tbt = np.full(M, 50.0)
    else:
        slo_m_ttft = rng.choice(TTFT_SLO_SET, M)
        slo_m_tbt = rng.choice(TBT_SLO_SET, M)
        if config == 2:
            batch = rng.integers(0, 17, size=(W, G), dtype=np.int32)
            kdyn = rng.uniform(300.0, 500.0, G).astype(np.float32)
            models_per_gpu = _distinct_models(rng, G, M, np.full(G, 2))
        else:
            nres = rng.integers(1, 5, size=G)
            models_per_gpu = _distinct_models(rng, G, M, nres)
            kdyn = rng.uniform(300.0, 500.0, G).astype(np.float32)
            if config == 4:
                sig = np.array([0.25, 0.5, 0.75])
                cap_pf = (np.rint(rng.choice(sig, G) * NS) - 1).astype(np.int8)
                cap_dc = (np.rint(rng.choice(sig, G) * NS) - 1).astype(np.int8)
            batch = np.minimum(rng.poisson(4.0, size=(W, G)), 31).astype(np.int32)
    resident = _resident_bits(models_per_gpu, M)
    gpus = {"n_gpus": G, "n_waves": W, "batch": np.ascontiguousarray(batch),
            "k_dyn_w": kdyn, "resident": resident, "cap_pf": cap_pf, "cap_dc": cap_dc}

    # --- requests
    model = rng.integers(0, M, size=R, dtype=np.int32)
    if config == 1:
        prompt = np.zeros(R, dtype=np.int32)          # no prompt phase: decode-row lookup
        pred_out = np.zeros(R, dtype=np.int32)
    else:
        if config == 4:
            long_mask = rng.random(R) < 0.3
            short = _lognormal_tokens(rng, 5.0, R, 16, 8192)
            longp = _lognormal_tokens(rng, 8.0, R, 16, 8192)
            prompt = np.where(long_mask, longp, short).astype(np.int32)
        else:
            prompt = _lognormal_tokens(rng, 6.0, R, 16, 8192)
        pred_out = _lognormal_tokens(rng, 5.0, R, 1, 8192)
    slo_ttft = slo_m_ttft[model].astype(np.float32)
    slo_tbt = slo_m_tbt[model].astype(np.float32)
    if config == 3:
        planted = rng.random(R) < 0.1
        slo_ttft[planted] = 1.0
        slo_tbt[planted] = 1.0
    else:
        planted = np.zeros(R, dtype=bool)
    wave = ((np.arange(R, dtype=np.int64) * W) // max(R, 1)).astype(np.int32)
    requests = {"n_requests": R, "model": model, "wave": wave, "prompt_tokens": prompt,
                "pred_out_tokens": pred_out, "slo_ttft_ms": slo_ttft, "slo_tbt_ms": slo_tbt}
    meta = {"config": config, "seed": seed, "a": a, "c": c, "cp": cp, "planted": planted,
            "models_per_gpu": models_per_gpu}
    return {"lut": lut, "gpus": gpus, "requests": requests, "meta": meta}


# --------------------------------------------------------------------------- migration
def _preferred_sm_level(a, c, cp, slo_ttft, slo_tbt, prompt_tokens, batch, s, f):
    """Instance SM level: the smallest level whose noise-free latencies at the top
    frequency meet both SLOs (else the top level).  This models the local
    scheduler's per-model preferred configuration (App. E, first step) as an
    input; the scoring below never sees the noise-free model."""
    ns = len(s)
    ptok = ROW_TOKENS * np.minimum(np.maximum((prompt_tokens + ROW_TOKENS - 1) // ROW_TOKENS, 1), N_ROWS)
    b = np.minimum(batch + 1, N_ROWS)
    fmax = float(f[-1])
    out = np.full(prompt_tokens.shape, ns - 1, dtype=np.int32)
    done = np.zeros(prompt_tokens.shape, dtype=bool)
    for j in range(ns):
        sj = float(s[j])
        ok = (a + cp * ptok / (sj * fmax) < slo_ttft) & (a + c * b / (sj * fmax) < slo_tbt)
        pick = ok & ~done
        out[pick] = j
        done |= ok
    return out


def make_fleet(seed: int | None = None, n_gpus: int = 2048) -> dict:
    """Consolidation fleet of configuration 5 (optionally fewer GPUs)."""
    if seed is None:
        seed = config_seed(5)
    rng = np.random.default_rng(seed)
    M, NS, NF, G, K = 32, 8, 16, int(n_gpus), MAX_INST
    s, f = sm_levels(NS), freq_levels(NF)
    a, c, cp = _latency_params(rng, M, prefill=True)
    pf, dc = _tables(rng, M, s, f, a, c, cp, noise=True)
    lut = _lut(pf, dc, s, f)
    slo_m_ttft = rng.choice(TTFT_SLO_SET, M)
    slo_m_tbt = rng.choice(TBT_SLO_SET, M)

    n_want = rng.integers(1, K + 1, size=G)
    inst_model = np.zeros((G, K), dtype=np.int32)
    n_inst = np.zeros(G, dtype=np.int32)
    hbm = np.zeros(G, dtype=np.int32)
    foot = np.rint(rng.uniform(8.0, 80.0, size=(G, K)) * 1024.0).astype(np.int64)
    for g in range(G):
        ms = rng.choice(M, int(n_want[g]), replace=False)
        tot = 0
        for i, mm in enumerate(ms):
            if tot + foot[g, i] > HBM_CAP_MIB:
                break
            tot += int(foot[g, i])
            inst_model[g, n_inst[g]] = mm
            n_inst[g] += 1
        hbm[g] = tot
    inst_prompt = _lognormal_tokens(rng, 6.0, G * K, 16, 8192).reshape(G, K)
    inst_batch = np.minimum(rng.poisson(4.0, size=(G, K)), 31).astype(np.int32)
    slo_ttft = slo_m_ttft[inst_model].astype(np.float32)
    slo_tbt = slo_m_tbt[inst_model].astype(np.float32)
    inst_sm = _preferred_sm_level(a[inst_model], c[inst_model], cp[inst_model],
                                  slo_ttft.astype(np.float64), slo_tbt.astype(np.float64),
                                  inst_prompt.astype(np.int64), inst_batch.astype(np.int64), s, f)
    # unused slots hold zeros: they are never read
    unused = np.arange(K)[None, :] >= n_inst[:, None]
    for arr in (inst_model, inst_prompt, inst_batch, inst_sm):
        arr[unused] = 0
    slo_ttft[unused] = 0.0
    slo_tbt[unused] = 0.0
    sm_pm = np.rint(1000.0 * rng.uniform(0.0, 0.6, G)).astype(np.int32)
    util = (sm_pm.astype(np.float64) / 1000.0).astype(np.float32)
    kdyn = rng.uniform(300.0, 500.0, G).astype(np.float32)
    fleet = {"n_gpus": G, "max_inst": K, "n_inst": n_inst, "inst_model": inst_model,
             "inst_prompt_tokens": inst_prompt.astype(np.int32), "inst_batch": inst_batch,
             "inst_sm": inst_sm, "inst_slo_ttft_ms": slo_ttft, "inst_slo_tbt_ms": slo_tbt,
             "hbm_mib": hbm, "sm_permille": sm_pm, "util": util, "k_dyn_w": kdyn,
             "hbm_cap_mib": HBM_CAP_MIB, "sm_cap_permille": SM_CAP_PERMILLE}
    meta = {"config": 5, "seed": seed, "a": a, "c": c, "cp": cp}
    return {"lut": lut, "fleet": fleet, "meta": meta}


# --------------------------------------------------------------------------- tiny random cases
def make_tiny_placement(rng: np.random.Generator, R=None, G=None, M=None, NS=None, NF=None,
                        W=None, caps=None, ties=False, nan_cells=False) -> dict:
    """Small random placement instance for brute-force comparison and parity edge cases."""
    R = int(rng.integers(1, 9)) if R is None else R
    G = int(rng.integers(1, 6)) if G is None else G
    M = int(rng.integers(1, 4)) if M is None else M
    NS = int(rng.integers(1, 5)) if NS is None else NS
    NF = int(rng.integers(1, 7)) if NF is None else NF
    W = int(rng.integers(1, 3)) if W is None else W
    caps = bool(rng.integers(0, 2)) if caps is None else caps
    s, f = sm_levels(NS), freq_levels(NF)
    if ties:
        pf = np.full((M, N_ROWS, NS, NF), np.float32(rng.uniform(5, 30)), dtype=np.float32)
        dc = np.full((M, N_ROWS, NS, NF), np.float32(rng.uniform(5, 30)), dtype=np.float32)
    else:
        pf = rng.uniform(5.0, 60.0, (M, N_ROWS, NS, NF)).astype(np.float32)
        dc = rng.uniform(2.0, 40.0, (M, N_ROWS, NS, NF)).astype(np.float32)
    if nan_cells:
        mask = rng.random(pf.shape) < 0.1
        pf[mask] = np.nan
        dc[rng.random(dc.shape) < 0.05] = np.inf
    lut = _lut(pf, dc, s, f, p0=float(rng.uniform(0.0, 150.0)))
    batch = rng.integers(0, 32, size=(W, G), dtype=np.int32)
    if ties:
        kdyn = np.full(G, np.float32(rng.uniform(300, 500)), dtype=np.float32)
        batch[:] = batch[:, :1]
    else:
        kdyn = rng.uniform(0.0, 500.0, G).astype(np.float32)
    models_per_gpu = [np.flatnonzero(rng.random(M) < 0.7) for _ in range(G)]
    resident = _resident_bits(models_per_gpu, M)
    cap_pf = rng.integers(0, NS, G).astype(np.int8) if caps else None
    cap_dc = rng.integers(0, NS, G).astype(np.int8) if caps else None
    gpus = {"n_gpus": G, "n_waves": W, "batch": batch, "k_dyn_w": kdyn,
            "resident": resident, "cap_pf": cap_pf, "cap_dc": cap_dc}
    prompt = np.where(rng.random(R) < 0.3, 0, rng.integers(1, 9000, R)).astype(np.int32)
    requests = {"n_requests": R, "model": rng.integers(0, M, R).astype(np.int32),
                "wave": rng.integers(0, W, R).astype(np.int32), "prompt_tokens": prompt,
                "pred_out_tokens": rng.integers(0, 300, R).astype(np.int32),
                "slo_ttft_ms": rng.uniform(10.0, 70.0, R).astype(np.float32),
                "slo_tbt_ms": rng.uniform(5.0, 45.0, R).astype(np.float32)}
    return {"lut": lut, "gpus": gpus, "requests": requests,
            "meta": {"models_per_gpu": models_per_gpu}}


def make_tiny_fleet(rng: np.random.Generator, G=None, M=None, NS=None, NF=None,
                    loose=False, huge_budget=False, K=MAX_INST) -> dict:
    """Small random consolidation fleet for brute-force comparison (K instance slots per GPU)."""
    G = int(rng.integers(2, 7)) if G is None else G
    M = int(rng.integers(1, 4)) if M is None else M
    NS = int(rng.integers(1, 5)) if NS is None else NS
    NF = int(rng.integers(1, 9)) if NF is None else NF
    s, f = sm_levels(NS), freq_levels(NF)
    pf = rng.uniform(5.0, 60.0, (M, N_ROWS, NS, NF)).astype(np.float32)
    dc = rng.uniform(2.0, 40.0, (M, N_ROWS, NS, NF)).astype(np.float32)
    lut = _lut(pf, dc, s, f, p0=float(rng.uniform(50.0, 150.0)))
    n_inst = rng.integers(1, K + 1, G).astype(np.int32)
    inst_model = rng.integers(0, M, (G, K)).astype(np.int32)
    inst_prompt = np.where(rng.random((G, K)) < 0.2, 0, rng.integers(1, 9000, (G, K))).astype(np.int32)
    inst_batch = rng.integers(0, 32, (G, K)).astype(np.int32)
    inst_sm = rng.integers(0, NS, (G, K)).astype(np.int32)
    if loose:
        slo_ttft = np.full((G, K), 1e9, dtype=np.float32)
        slo_tbt = np.full((G, K), 1e9, dtype=np.float32)
    else:
        slo_ttft = rng.uniform(20.0, 80.0, (G, K)).astype(np.float32)
        slo_tbt = rng.uniform(10.0, 50.0, (G, K)).astype(np.float32)
    hbm = rng.integers(1000, 200000, G).astype(np.int32)
    sm_pm = rng.integers(0, 700, G).astype(np.int32)
    util = (sm_pm.astype(np.float64) / 1000.0).astype(np.float32)
    kdyn = rng.uniform(300.0, 500.0, G).astype(np.float32)
    fleet = {"n_gpus": G, "max_inst": K, "n_inst": n_inst, "inst_model": inst_model,
             "inst_prompt_tokens": inst_prompt, "inst_batch": inst_batch, "inst_sm": inst_sm,
             "inst_slo_ttft_ms": slo_ttft, "inst_slo_tbt_ms": slo_tbt, "hbm_mib": hbm,
             "sm_permille": sm_pm, "util": util, "k_dyn_w": kdyn,
             "hbm_cap_mib": (1 << 30) if huge_budget else HBM_CAP_MIB,
             "sm_cap_permille": (1 << 30) if huge_budget else SM_CAP_PERMILLE}
    return {"lut": lut, "fleet": fleet, "meta": {}}


# --------------------------------------------------------------------------- local sweep
SWEEP_SEED = CONFIG_SEED_BASE + 50
SWEEP_MAX_TASKS = 8
PREFILL_CHUNK = 2048      # tokens per prefill unit in the sweep workload


def sm_permille(s: np.ndarray) -> np.ndarray:
    """Integer SM share of each level in per-mille of the device (125 per eighth)."""
    return np.rint(1000.0 * s.astype(np.float64)).astype(np.int32)


def make_sweep(seed: int | None = None, n_gpus: int = 1024, n_epochs: int = 64,
               max_tasks: int = SWEEP_MAX_TASKS) -> dict:
    """Batches for the local SM/frequency sweep: one batch per (epoch, GPU).

    Tables as configuration 3 (32 models, 8 SM x 16 frequency levels, +-5% noise).  Each
    GPU hosts 1-4 distinct models and has k ~ U(300, 500).  Per epoch, each hosted model
    has a decode step in the batch with probability 0.7 (decode batch size
    min(Poisson(4) + 1, 32)), and Poisson(0.7) prefill units of hosted models join: a
    prompt from configuration 4's bimodal law (70% lognormal mu=5, 30% mu=8), prefilled in
    chunks of at most 2048 tokens; tasks past max_tasks are dropped.  Slack: decode TBT
    SLO x U(0.9, 1); prefill TTFT SLO x U(0.7, 1).  Utilisation u = min(1, total decode batch / 32).  SM shares in per-mille,
    device budget 1000.
    """
    if seed is None:
        seed = SWEEP_SEED
    rng = np.random.default_rng(seed)
    M, NS, NF, G, E, T = 32, 8, 16, int(n_gpus), int(n_epochs), int(max_tasks)
    s, f = sm_levels(NS), freq_levels(NF)
    a, c, cp = _latency_params(rng, M, prefill=True)
    pf, dc = _tables(rng, M, s, f, a, c, cp, noise=True)
    lut = _lut(pf, dc, s, f)
    slo_m_ttft = rng.choice(TTFT_SLO_SET, M)
    slo_m_tbt = rng.choice(TBT_SLO_SET, M)
    nres = rng.integers(1, 5, size=G)
    models_per_gpu = _distinct_models(rng, G, M, nres)
    kdyn_g = rng.uniform(300.0, 500.0, G).astype(np.float32)

    B = E * G
    n_tasks = np.zeros(B, np.int32)
    model = np.zeros((B, T), np.int32)
    phase = np.zeros((B, T), np.int32)
    tokens = np.zeros((B, T), np.int32)
    slack = np.zeros((B, T), np.float32)
    util = np.zeros(B, np.float32)
    kdyn = np.tile(kdyn_g, E)
    dec_on = rng.random((E, G, MAX_INST)) < 0.7
    dec_b = np.minimum(rng.poisson(4.0, (E, G, MAX_INST)) + 1, N_ROWS)
    n_pre = rng.poisson(0.7, (E, G))
    for e in range(E):
        for g in range(G):
            b = e * G + g
            ms = models_per_gpu[g]
            t = 0
            tot = 0
            for i, mm in enumerate(ms):
                if dec_on[e, g, i] and t < T:
                    model[b, t], phase[b, t], tokens[b, t] = mm, 1, dec_b[e, g, i]
                    slack[b, t] = slo_m_tbt[mm] * rng.uniform(0.9, 1.0)
                    tot += int(dec_b[e, g, i])
                    t += 1
            for _ in range(int(n_pre[e, g])):
                mm = ms[int(rng.integers(0, len(ms)))]
                mu = 8.0 if rng.random() < 0.3 else 5.0
                tok = min(int(np.clip(np.rint(rng.lognormal(mu, 1.0)), 16, 8192)), PREFILL_CHUNK)
                sl = slo_m_ttft[mm] * rng.uniform(0.7, 1.0)
                if t < T:
                    model[b, t], phase[b, t], tokens[b, t], slack[b, t] = mm, 0, tok, sl
                    t += 1
            n_tasks[b] = t
            util[b] = min(1.0, tot / 32.0)
    batches = {"n_batches": B, "max_tasks": T, "n_tasks": n_tasks, "task_model": model,
               "task_phase": phase, "task_tokens": tokens, "task_slack_ms": slack,
               "k_dyn_w": kdyn, "util": util, "sm_units": sm_permille(s), "sm_budget": 1000}
    meta = {"seed": seed, "n_gpus": G, "n_epochs": E, "models_per_gpu": models_per_gpu}
    return {"lut": lut, "batches": batches, "meta": meta}


def make_tiny_sweep(rng: np.random.Generator, B=None, T=None, M=None, NS=None, NF=None,
                    nan_cells=False, zero_power=False) -> dict:
    """Small random sweep instance for pins and parity edge cases."""
    B = int(rng.integers(1, 6)) if B is None else B
    T = int(rng.integers(1, 5)) if T is None else T
    M = int(rng.integers(1, 4)) if M is None else M
    NS = int(rng.integers(1, 5)) if NS is None else NS
    NF = int(rng.integers(1, 7)) if NF is None else NF
    s, f = sm_levels(NS), freq_levels(NF)
    pf = rng.uniform(5.0, 60.0, (M, N_ROWS, NS, NF)).astype(np.float32)
    dc = rng.uniform(2.0, 40.0, (M, N_ROWS, NS, NF)).astype(np.float32)
    if nan_cells:
        pf[rng.random(pf.shape) < 0.1] = np.nan
        dc[rng.random(dc.shape) < 0.05] = np.inf
    lut = _lut(pf, dc, s, f, p0=0.0 if zero_power else float(rng.uniform(0.0, 150.0)))
    n_tasks = rng.integers(0, T + 1, B).astype(np.int32)
    units = sm_permille(s)
    batches = {"n_batches": B, "max_tasks": T, "n_tasks": n_tasks,
               "task_model": rng.integers(0, M, (B, T)).astype(np.int32),
               "task_phase": rng.integers(0, 2, (B, T)).astype(np.int32),
               "task_tokens": rng.integers(1, 9000, (B, T)).astype(np.int32),
               "task_slack_ms": rng.uniform(3.0, 60.0, (B, T)).astype(np.float32),
               "k_dyn_w": (np.zeros(B) if zero_power else rng.uniform(0.0, 500.0, B)).astype(np.float32),
               "util": rng.uniform(0.0, 1.0, B).astype(np.float32),
               "sm_units": units, "sm_budget": int(rng.integers(1, 1000 * T + 2))}
    return {"lut": lut, "batches": batches, "meta": {}}


# --------------------------------------------------------------------------- preferred configuration
LLMS_SEED = CONFIG_SEED_BASE + 60


def make_llms(seed: int | None = None, n_gpus: int = 2048) -> dict:
    """Active LLM instances for the preferred-configuration search and the EWR reduction.

    Configuration 5's fleet law: tables as configuration 3 (32 models, 8 SM x 16 frequency
    levels, +-5% noise), each GPU hosts 1-4 distinct models with k ~ U(300, 500); per
    instance the average prompt over the last window is lognormal(6, 1) tokens (clipped
    16-8192), the average output lognormal(5, 1) (clipped 1-8192), the decode batch
    min(Poisson(4), 31), and the SLOs are the model's.
    """
    if seed is None:
        seed = LLMS_SEED
    rng = np.random.default_rng(seed)
    M, NS, NF, G, K = 32, 8, 16, int(n_gpus), MAX_INST
    s, f = sm_levels(NS), freq_levels(NF)
    a, c, cp = _latency_params(rng, M, prefill=True)
    pf, dc = _tables(rng, M, s, f, a, c, cp, noise=True)
    lut = _lut(pf, dc, s, f)
    slo_m_ttft = rng.choice(TTFT_SLO_SET, M)
    slo_m_tbt = rng.choice(TBT_SLO_SET, M)
    n_inst = rng.integers(1, K + 1, size=G).astype(np.int32)
    model = np.zeros((G, K), np.int32)
    for g in range(G):
        model[g, :n_inst[g]] = rng.choice(M, int(n_inst[g]), replace=False)
    avg_in = _lognormal_tokens(rng, 6.0, G * K, 16, 8192).reshape(G, K)
    avg_out = _lognormal_tokens(rng, 5.0, G * K, 1, 8192).reshape(G, K)
    batch = np.minimum(rng.poisson(4.0, size=(G, K)), 31).astype(np.int32)
    kdyn = rng.uniform(300.0, 500.0, G).astype(np.float32)
    unused = np.arange(K)[None, :] >= n_inst[:, None]
    for arr in (model, avg_in, avg_out, batch):
        arr[unused] = 0
    slo_ttft = slo_m_ttft[model].astype(np.float32)
    slo_tbt = slo_m_tbt[model].astype(np.float32)
    slo_ttft[unused] = 0.0
    slo_tbt[unused] = 0.0
    llms = {"n_gpus": G, "max_inst": K, "n_inst": n_inst, "model": model, "avg_in_tokens": avg_in,
            "avg_out_tokens": avg_out, "batch": batch, "slo_ttft_ms": slo_ttft, "slo_tbt_ms": slo_tbt,
            "k_dyn_w": kdyn}
    return {"lut": lut, "llms": llms, "meta": {"seed": seed}}


def make_tiny_llms(rng: np.random.Generator, G=None, K=None, M=None, NS=None, NF=None,
                   nan_cells=False, zero_out=False) -> dict:
    """Small random set of LLM instances for pins and parity edge cases."""
    G = int(rng.integers(1, 5)) if G is None else G
    K = int(rng.integers(1, 4)) if K is None else K
    M = int(rng.integers(1, 4)) if M is None else M
    NS = int(rng.integers(1, 5)) if NS is None else NS
    NF = int(rng.integers(1, 7)) if NF is None else NF
    s, f = sm_levels(NS), freq_levels(NF)
    pf = rng.uniform(5.0, 60.0, (M, N_ROWS, NS, NF)).astype(np.float32)
    dc = rng.uniform(2.0, 40.0, (M, N_ROWS, NS, NF)).astype(np.float32)
    if nan_cells:
        pf[rng.random(pf.shape) < 0.1] = np.nan
        dc[rng.random(dc.shape) < 0.05] = np.inf
    lut = _lut(pf, dc, s, f, p0=float(rng.uniform(0.0, 150.0)))
    llms = {"n_gpus": G, "max_inst": K, "n_inst": rng.integers(0, K + 1, G).astype(np.int32),
            "model": rng.integers(0, M, (G, K)).astype(np.int32),
            "avg_in_tokens": rng.integers(1, 9000, (G, K)).astype(np.int32),
            "avg_out_tokens": (np.zeros((G, K)) if zero_out else rng.integers(0, 400, (G, K))).astype(np.int32),
            "batch": rng.integers(0, 32, (G, K)).astype(np.int32),
            "slo_ttft_ms": rng.uniform(8.0, 70.0, (G, K)).astype(np.float32),
            "slo_tbt_ms": rng.uniform(4.0, 45.0, (G, K)).astype(np.float32),
            "k_dyn_w": rng.uniform(0.0, 500.0, G).astype(np.float32)}
    return {"lut": lut, "llms": llms, "meta": {}}


# --------------------------------------------------------------------------- current-frequency dispatch
DISPATCH_SEED = CONFIG_SEED_BASE + 70
N_AVAIL_STEPS = 4


def make_dispatch(seed: int | None = None, n_requests: int = 65536, n_gpus: int = 512) -> dict:
    """Requests and GPU state for the paper's own dispatcher (current frequency, one
    operating point per GPU, 2% stability tie-break, F_max fallback).

    Configuration 3's laws for the tables (32 models, 8 SM x 16 frequency levels, +-5%
    noise), the GPUs (1-4 models, k ~ U(300, 500), batch min(Poisson(4), 31)) and the
    requests (prompts lognormal(6, 1), outputs lognormal(5, 1), model SLOs).  Added: each
    GPU's current frequency level (uniform), a 4-step free-memory profile from its local
    scheduler (now: U(0, 2048) MiB free; each later step after Exp(30 ms) frees U(256, 4096)
    MiB more, up to 288 GiB) with its free SM level (now: uniform in -1..7, -1 = none;
    each step frees 0-3 levels more, up to 7), a KV-cache size per model of 128-640 KiB per
    token, and k = 400 W for a newly activated GPU.
    """
    if seed is None:
        seed = DISPATCH_SEED
    rng = np.random.default_rng(seed)
    M, NS, NF, G, R, S = 32, 8, 16, int(n_gpus), int(n_requests), N_AVAIL_STEPS
    s, f = sm_levels(NS), freq_levels(NF)
    a, c, cp = _latency_params(rng, M, prefill=True)
    pf, dc = _tables(rng, M, s, f, a, c, cp, noise=True)
    lut = _lut(pf, dc, s, f)
    slo_m_ttft = rng.choice(TTFT_SLO_SET, M)
    slo_m_tbt = rng.choice(TBT_SLO_SET, M)
    nres = rng.integers(1, 5, size=G)
    models_per_gpu = _distinct_models(rng, G, M, nres)
    kdyn = rng.uniform(300.0, 500.0, G).astype(np.float32)
    batch = np.minimum(rng.poisson(4.0, size=G), 31).astype(np.int32)
    freq_cur = rng.integers(0, NF, G).astype(np.int32)
    t = np.zeros((G, S))
    mem = np.zeros((G, S), np.int64)
    sm = np.zeros((G, S), np.int32)
    mem[:, 0] = rng.integers(0, 2049, G)
    sm[:, 0] = rng.integers(-1, NS, G)
    for k in range(1, S):
        t[:, k] = t[:, k - 1] + rng.exponential(30.0, G)
        mem[:, k] = np.minimum(mem[:, k - 1] + rng.integers(256, 4097, G), HBM_CAP_MIB)
        sm[:, k] = np.minimum(sm[:, k - 1] + rng.integers(0, 4, G), NS - 1)
    avail = {"n_gpus": G, "n_steps": S, "freq_cur": freq_cur, "batch": batch, "k_dyn_w": kdyn,
             "resident": _resident_bits(models_per_gpu, M), "t_avail_ms": t.astype(np.float32),
             "mem_free_mib": mem.astype(np.int32), "sm_free": sm,
             "kv_kib_per_token": rng.integers(128, 641, M).astype(np.int32), "k_new_w": 400.0}
    model = rng.integers(0, M, size=R, dtype=np.int32)
    prompt = _lognormal_tokens(rng, 6.0, R, 16, 8192)
    pred_out = _lognormal_tokens(rng, 5.0, R, 1, 8192)
    requests = {"n_requests": R, "model": model, "wave": None, "prompt_tokens": prompt,
                "pred_out_tokens": pred_out, "slo_ttft_ms": slo_m_ttft[model].astype(np.float32),
                "slo_tbt_ms": slo_m_tbt[model].astype(np.float32)}
    return {"lut": lut, "avail": avail, "requests": requests,
            "meta": {"seed": seed, "models_per_gpu": models_per_gpu}}


def wave_bounds(n_requests: int, n_waves: int) -> np.ndarray:
    """Offsets of n_waves arrival waves of near-equal size over requests ordered by wave
    (wave w holds requests bounds[w] .. bounds[w+1]-1), as the placement workloads assign
    waves: request r arrives in wave floor(r * W / R)."""
    R, Wn = int(n_requests), int(n_waves)
    wave = (np.arange(R, dtype=np.int64) * Wn) // max(R, 1)
    return np.searchsorted(wave, np.arange(Wn + 1), side="left").astype(np.int32)


def make_dispatch_waves(seed: int | None = None, n_requests: int = 65536, n_gpus: int = 512,
                        n_waves: int = 64) -> dict:
    """The dispatcher workload of make_dispatch with its requests split into n_waves arrival
    waves (configuration 4's 64 waves), for the wave-by-wave dispatch: same GPUs, tables
    and request laws; ``wave_start`` holds the wave offsets."""
    inp = make_dispatch(seed=seed, n_requests=n_requests, n_gpus=n_gpus)
    ws = wave_bounds(n_requests, n_waves)
    inp["requests"]["wave"] = (np.searchsorted(ws, np.arange(n_requests), side="right") - 1).astype(np.int32)
    inp["wave_start"] = ws
    return inp


def make_tiny_dispatch(rng: np.random.Generator, R=None, G=None, M=None, NS=None, NF=None, S=None,
                       ties=False) -> dict:
    """Small random dispatch instance for pins and parity edge cases.  With ``ties`` every
    GPU shares one table value and power coefficient, so energies tie exactly or lie
    within 2% and the stability tie-break decides."""
    R = int(rng.integers(1, 9)) if R is None else R
    G = int(rng.integers(1, 7)) if G is None else G
    M = int(rng.integers(1, 3)) if M is None else M
    NS = int(rng.integers(1, 5)) if NS is None else NS
    NF = int(rng.integers(1, 6)) if NF is None else NF
    S = int(rng.integers(1, 4)) if S is None else S
    s, f = sm_levels(NS), freq_levels(NF)
    pf = rng.uniform(5.0, 60.0, (M, N_ROWS, NS, NF)).astype(np.float32)
    dc = rng.uniform(2.0, 40.0, (M, N_ROWS, NS, NF)).astype(np.float32)
    kd = rng.uniform(0.0, 500.0, G)
    if ties:
        pf[:] = np.float32(rng.uniform(5, 30))
        dc[:] = np.float32(rng.uniform(2, 20))
        kd = np.full(G, rng.uniform(0.0, 5.0))      # dynamic power small: energies within 2%
    lut = _lut(pf, dc, s, f, p0=float(np.float32(rng.uniform(50.0, 150.0))))   # the ABI's P0 is float32
    t = np.cumsum(rng.exponential(10.0, (G, S)), axis=1)
    t[:, 0] = 0.0
    mem = np.cumsum(rng.integers(0, 400, (G, S)), axis=1)
    sm = np.minimum(np.cumsum(rng.integers(0, 2, (G, S)), axis=1) + rng.integers(-1, NS, G)[:, None], NS - 1)
    models_per_gpu = [np.flatnonzero(rng.random(M) < 0.8) for _ in range(G)]
    avail = {"n_gpus": G, "n_steps": S, "freq_cur": rng.integers(0, NF, G).astype(np.int32),
             "batch": rng.integers(0, 32, G).astype(np.int32), "k_dyn_w": kd.astype(np.float32),
             "resident": _resident_bits(models_per_gpu, M), "t_avail_ms": t.astype(np.float32),
             "mem_free_mib": mem.astype(np.int32), "sm_free": sm.astype(np.int32),
             "kv_kib_per_token": rng.integers(1, 200, M).astype(np.int32),
             "k_new_w": float(np.float32(rng.uniform(0, 500)))}
    requests = {"n_requests": R, "model": rng.integers(0, M, R).astype(np.int32), "wave": None,
                "prompt_tokens": np.where(rng.random(R) < 0.2, 0, rng.integers(1, 3000, R)).astype(np.int32),
                "pred_out_tokens": rng.integers(0, 300, R).astype(np.int32),
                "slo_ttft_ms": rng.uniform(10.0, 90.0, R).astype(np.float32),
                "slo_tbt_ms": rng.uniform(5.0, 45.0, R).astype(np.float32)}
    return {"lut": lut, "avail": avail, "requests": requests, "meta": {}}


# --------------------------------------------------------------------------- transfer plan
TRANSFER_SEED = CONFIG_SEED_BASE + 80
GPUS_PER_NODE = 8
XGMI_LINK_GBS = 153.6      # one GPU-to-GPU xGMI link inside a node
NIC_GBS = 50.0             # 400 Gb/s between nodes


def make_transfer(seed: int | None = None, n_gpus: int = 2048, requests_per_gpu: int = 8) -> dict:
    """A 2,048-GPU fleet about to be reconfigured (configuration 5's shape), for the transfer
    cost matrix of the device mapping and the per-request move decisions.

    Tables as configuration 3; each GPU hosts 1-4 distinct models of 32, whose weights take
    U(8, 80) GiB; GPUs sit 8 to a node (xGMI links of 153.6 GB/s inside a node, 50 GB/s
    between nodes); each GPU has U(0, 16) GiB of request state selected for migration.  The
    plan keeps half of the GPUs' state in place and sends the other half to a random
    permutation of those GPUs.  Each GPU has ~8 in-flight requests of its models: context
    lognormal(6, 1) prompt tokens plus U{0..500} generated, remaining tokens lognormal(5, 1),
    KV cache 128-640 KiB per token by model, 4 bytes per token of token state, and each GPU
    an operating point (uniform SM and frequency level) and decode batch min(Poisson(4), 31).
    """
    if seed is None:
        seed = TRANSFER_SEED
    rng = np.random.default_rng(seed)
    M, NS, NF, G = 32, 8, 16, int(n_gpus)
    s, f = sm_levels(NS), freq_levels(NF)
    a, c, cp = _latency_params(rng, M, prefill=True)
    pf, dc = _tables(rng, M, s, f, a, c, cp, noise=True)
    lut = _lut(pf, dc, s, f)
    nres = rng.integers(1, 5, size=G)
    models_per_gpu = _distinct_models(rng, G, M, nres)
    weights = np.rint(rng.uniform(8.0, 80.0, M) * 1024).astype(np.int32)
    state = rng.integers(0, 16 * 1024 + 1, G).astype(np.int32)
    transfer = {"n_gpus": G, "words": (M + 31) // 32, "resident": _resident_bits(models_per_gpu, M),
                "weights_mib": weights, "state_mib": state,
                "node": (np.arange(G) // GPUS_PER_NODE).astype(np.int32),
                "bw_intra_gbs": XGMI_LINK_GBS, "bw_inter_gbs": NIC_GBS}
    dest = np.arange(G, dtype=np.int32)
    moving = np.flatnonzero(rng.random(G) < 0.5)
    dest[moving] = moving[rng.permutation(len(moving))]
    plan = {"dest": dest, "freq_cur": rng.integers(0, NF, G).astype(np.int32),
            "sm_cur": rng.integers(0, NS, G).astype(np.int32),
            "batch": np.minimum(rng.poisson(4.0, G), 31).astype(np.int32)}
    Q = G * int(requests_per_gpu)
    src = rng.integers(0, G, Q).astype(np.int32)
    model = np.array([models_per_gpu[g][int(rng.integers(0, len(models_per_gpu[g])))] for g in src], np.int32)
    ctx = (_lognormal_tokens(rng, 6.0, Q, 16, 8192) + rng.integers(0, 501, Q)).clip(1, 8192).astype(np.int32)
    kv_tok = rng.integers(128, 641, M)
    moves = {"n_requests": Q, "src": src, "model": model, "context_tokens": ctx,
             "remaining_tokens": _lognormal_tokens(rng, 5.0, Q, 0, 8192),
             "kv_kib": (kv_tok[model] * ctx).astype(np.int32), "token_kib": ((ctx * 4 + 1023) // 1024).astype(np.int32)}
    return {"lut": lut, "n_models": M, "transfer": transfer, "plan": plan, "moves": moves,
            "meta": {"seed": seed, "models_per_gpu": models_per_gpu}}


def make_tiny_transfer(rng: np.random.Generator, G=None, M=None, NS=None, NF=None, Q=None) -> dict:
    """Small random transfer instance for pins and parity edge cases."""
    G = int(rng.integers(1, 9)) if G is None else G
    M = int(rng.integers(1, 5)) if M is None else M
    NS = int(rng.integers(1, 5)) if NS is None else NS
    NF = int(rng.integers(1, 6)) if NF is None else NF
    Q = int(rng.integers(0, 20)) if Q is None else Q
    s, f = sm_levels(NS), freq_levels(NF)
    pf = rng.uniform(5.0, 600.0, (M, N_ROWS, NS, NF)).astype(np.float32)
    dc = rng.uniform(2.0, 40.0, (M, N_ROWS, NS, NF)).astype(np.float32)
    lut = _lut(pf, dc, s, f)
    models_per_gpu = [np.flatnonzero(rng.random(M) < 0.5) for _ in range(G)]
    transfer = {"n_gpus": G, "words": (M + 31) // 32, "resident": _resident_bits(models_per_gpu, M),
                "weights_mib": rng.integers(0, 90000, M).astype(np.int32),
                "state_mib": rng.integers(0, 20000, G).astype(np.int32),
                "node": (np.arange(G) // int(rng.integers(1, 5))).astype(np.int32),
                "bw_intra_gbs": float(np.float32(rng.uniform(50, 400))),
                "bw_inter_gbs": float(np.float32(rng.uniform(5, 100)))}
    plan = {"dest": rng.permutation(G).astype(np.int32), "freq_cur": rng.integers(0, NF, G).astype(np.int32),
            "sm_cur": rng.integers(0, NS, G).astype(np.int32), "batch": rng.integers(0, 32, G).astype(np.int32)}
    ctx = rng.integers(1, 9000, Q).astype(np.int32)
    moves = {"n_requests": Q, "src": rng.integers(0, G, Q).astype(np.int32),
             "model": rng.integers(0, M, Q).astype(np.int32), "context_tokens": ctx,
             "remaining_tokens": rng.integers(0, 600, Q).astype(np.int32),
             "kv_kib": (rng.integers(0, 800, Q) * ctx // 8).astype(np.int32),
             "token_kib": ((ctx * 4 + 1023) // 1024).astype(np.int32)}
    return {"lut": lut, "n_models": M, "transfer": transfer, "plan": plan, "moves": moves, "meta": {}}
