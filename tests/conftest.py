import json
import os
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
HERE = os.path.dirname(os.path.abspath(__file__))
if HERE not in sys.path:
    sys.path.insert(0, HERE)

GOLDEN = os.path.join(HERE, "golden")


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def load_golden(name):
    with open(os.path.join(GOLDEN, name)) as fh:
        return json.load(fh)


def _tables(spec):
    M, NS, NF = spec["n_models"], spec["n_sm"], spec["n_freq"]
    pf = np.full((M, 32, NS, NF), spec["fill"], np.float32)
    dc = np.full((M, 32, NS, NF), spec["fill"], np.float32)
    for m, row, j, k, v in spec["pf_cells"]:
        pf[m, row, j, k] = v
    for m, row, j, k, v in spec["dc_cells"]:
        dc[m, row, j, k] = v
    return {"n_models": M, "n_rows": 32, "n_sm": NS, "n_freq": NF,
            "sm_level": np.array(spec["sm_level"], np.float32),
            "freq_level": np.array(spec["freq_level"], np.float32),
            "pf": pf, "dc": dc, "p0_w": float(spec["p0_w"])}


def golden_placement(variant=None):
    """Inputs of the hand-worked placement example (optionally its capped variant)."""
    d = load_golden("placement_worked_example.json")
    lut = _tables(d["lut"])
    G = d["gpus"]["n_gpus"]
    batch = np.array(d["gpus"]["batch"], np.int32)
    gpus = {"n_gpus": G, "n_waves": 1, "batch": batch,
            "k_dyn_w": np.array(d["gpus"]["k_dyn_w"], np.float32),
            "resident": np.ones((G, 1), np.uint32), "cap_pf": None, "cap_dc": None}
    q = d["request"]
    req = {"n_requests": 1, "model": np.array([q["model"]], np.int32), "wave": None,
           "prompt_tokens": np.array([q["prompt_tokens"]], np.int32),
           "pred_out_tokens": np.array([q["pred_out_tokens"]], np.int32),
           "slo_ttft_ms": np.array([q["slo_ttft_ms"]], np.float32),
           "slo_tbt_ms": np.array([q["slo_tbt_ms"]], np.float32)}
    exp = d["expected"]
    if variant == "capped":
        v = d["capped_variant"]
        gpus["cap_pf"] = np.array(v["cap_pf"], np.int8)
        gpus["cap_dc"] = np.array(v["cap_dc"], np.int8)
        if v["drop_gpu0"]:
            gpus["batch"] = batch.copy()
            gpus["batch"][0, 0] = -1
        exp = v["expected"]
    return {"lut": lut, "gpus": gpus, "requests": req}, exp, d


def golden_migration():
    d = load_golden("migration_worked_example.json")
    lut = _tables(d["lut"])
    fs = d["fleet"]
    G, K = fs["n_gpus"], fs["max_inst"]
    z = lambda dt: np.zeros((G, K), dt)
    fl = {"n_gpus": G, "max_inst": K, "n_inst": np.zeros(G, np.int32), "inst_model": z(np.int32),
          "inst_prompt_tokens": z(np.int32), "inst_batch": z(np.int32), "inst_sm": z(np.int32),
          "inst_slo_ttft_ms": z(np.float32), "inst_slo_tbt_ms": z(np.float32),
          "hbm_mib": np.array(fs["hbm_mib"], np.int32), "sm_permille": np.array(fs["sm_permille"], np.int32),
          "util": np.array(fs["util"], np.float32), "k_dyn_w": np.array(fs["k_dyn_w"], np.float32),
          "hbm_cap_mib": fs["hbm_cap_mib"], "sm_cap_permille": fs["sm_cap_permille"]}
    for g, insts in enumerate(fs["instances"]):
        fl["n_inst"][g] = len(insts)
        for i, (m, pt, b, j, st, sb) in enumerate(insts):
            fl["inst_model"][g, i] = m
            fl["inst_prompt_tokens"][g, i] = pt
            fl["inst_batch"][g, i] = b
            fl["inst_sm"][g, i] = j
            fl["inst_slo_ttft_ms"][g, i] = st
            fl["inst_slo_tbt_ms"][g, i] = sb
    return {"lut": lut, "fleet": fl}, d["expected"], d


@pytest.fixture
def rng():
    return np.random.default_rng(12345)


def golden_sweep(variant=None):
    """Inputs of the hand-worked sweep example (optionally one of its variants by name)."""
    d = load_golden("sweep_worked_example.json")
    spec = dict(d["lut"])
    bt = dict(d["batch"])
    exp = d["expected"]
    slack = [t["slack_ms"] for t in bt["tasks"]]
    if variant is not None:
        v = [x for x in d["variants"] if x["name"] == variant][0]
        ch = v["change"]
        if "p0_w" in ch:
            spec["p0_w"] = ch["p0_w"]
        bt["sm_units"] = ch.get("sm_units", bt["sm_units"])
        bt["sm_budget"] = ch.get("sm_budget", bt["sm_budget"])
        bt["static_power"] = ch.get("static_power", 0)
        slack = ch.get("slack_ms", slack)
        exp = v["expected"]
    lut = _tables(spec)
    T = len(bt["tasks"])
    batches = {"n_batches": 1, "max_tasks": T, "n_tasks": np.array([T], np.int32),
               "task_model": np.array([[t["model"] for t in bt["tasks"]]], np.int32),
               "task_phase": np.array([[t["phase"] for t in bt["tasks"]]], np.int32),
               "task_tokens": np.array([[t["tokens"] for t in bt["tasks"]]], np.int32),
               "task_slack_ms": np.array([slack], np.float32),
               "k_dyn_w": np.array([bt["k_dyn_w"]], np.float32),
               "util": np.array([bt["util"]], np.float32),
               "sm_units": np.array(bt["sm_units"], np.int32), "sm_budget": int(bt["sm_budget"]),
               "static_power": int(bt.get("static_power", 0))}
    return {"lut": lut, "batches": batches}, exp, d


def golden_preferred(variant=None):
    """Inputs of the hand-worked preferred-configuration example (one instance), or of one
    of its variants by name."""
    d = load_golden("preferred_worked_example.json")
    lut = _tables(d["lut"])
    q = dict(d["instance"])
    exp = d["expected"]
    if variant is not None:
        v = [x for x in d["variants"] if x["name"] == variant][0]
        q.update(v["change"])
        exp = v["expected"]
    one = lambda v, dt: np.array([[v]], dt)
    llms = {"n_gpus": 1, "max_inst": 1, "n_inst": np.array([1], np.int32),
            "model": one(q["model"], np.int32), "avg_in_tokens": one(q["avg_in_tokens"], np.int32),
            "avg_out_tokens": one(q["avg_out_tokens"], np.int32), "batch": one(q["batch"], np.int32),
            "slo_ttft_ms": one(q["slo_ttft_ms"], np.float32), "slo_tbt_ms": one(q["slo_tbt_ms"], np.float32),
            "k_dyn_w": np.array([q["k_dyn_w"]], np.float32)}
    return {"lut": lut, "llms": llms}, exp, d


def golden_dispatch(variant=None):
    """Inputs of the hand-worked dispatch example (optionally one of its variants by name)."""
    d = load_golden("dispatch_worked_example.json")
    lut = _tables(d["lut"])
    av = dict(d["avail"])
    q = dict(d["request"])
    exp = d["expected"]
    if variant is not None:
        v = [x for x in d["variants"] if x["name"] == variant][0]
        for k, val in v["change"].items():
            (q if k in q else av)[k] = val
        exp = v["expected"]
    G = len(av["freq_cur"])
    avail = {"n_gpus": G, "n_steps": len(av["t_avail_ms"][0]), "freq_cur": np.array(av["freq_cur"], np.int32),
             "batch": np.array(av["batch"], np.int32), "k_dyn_w": np.array(av["k_dyn_w"], np.float32),
             "resident": np.ones((G, 1), np.uint32), "t_avail_ms": np.array(av["t_avail_ms"], np.float32),
             "mem_free_mib": np.array(av["mem_free_mib"], np.int32), "sm_free": np.array(av["sm_free"], np.int32),
             "kv_kib_per_token": np.array(av["kv_kib_per_token"], np.int32), "k_new_w": float(av["k_new_w"])}
    req = {"n_requests": 1, "model": np.array([q["model"]], np.int32), "wave": None,
           "prompt_tokens": np.array([q["prompt_tokens"]], np.int32),
           "pred_out_tokens": np.array([q["pred_out_tokens"]], np.int32),
           "slo_ttft_ms": np.array([q["slo_ttft_ms"]], np.float32),
           "slo_tbt_ms": np.array([q["slo_tbt_ms"]], np.float32)}
    return {"lut": lut, "avail": avail, "requests": req}, exp, d


def golden_transfer():
    """Inputs of the hand-worked transfer example."""
    d = load_golden("transfer_worked_example.json")
    M = d["n_models"]
    G = len(d["resident"])
    res = np.zeros((G, 1), np.uint32)
    for g, ms in enumerate(d["resident"]):
        for m in ms:
            res[g, 0] |= np.uint32(1 << m)
    transfer = {"n_gpus": G, "words": 1, "resident": res, "weights_mib": np.array(d["weights_mib"], np.int32),
                "state_mib": np.array(d["state_mib"], np.int32), "node": np.array(d["node"], np.int32),
                "bw_intra_gbs": d["bw_intra_gbs"], "bw_inter_gbs": d["bw_inter_gbs"]}
    plan = {k: np.array(v, np.int32) for k, v in d["plan"].items()}
    mv = d["moves"]
    moves = {"n_requests": len(mv)}
    for k in ("src", "model", "context_tokens", "remaining_tokens", "kv_kib", "token_kib"):
        moves[k] = np.array([x[k] for x in mv], np.int32)
    return {"lut": _tables(d["lut"]), "n_models": M, "transfer": transfer, "plan": plan, "moves": moves}, d
