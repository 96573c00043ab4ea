"""bench.py: the one-GPU contract (more GPUs exit with a message, before any GPU work) and,
on a GPU, the schema of the JSON line a short run prints."""
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BENCH = os.path.join(ROOT, "bench.py")


@pytest.mark.parametrize("args,env", [(["--gpus", "2"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_exits_with_a_message(args, env):
    e = dict(os.environ, **env)
    p = subprocess.run([sys.executable, BENCH, *args], capture_output=True, text=True, env=e, timeout=120)
    assert p.returncode == 2
    assert "one GPU only" in p.stderr
    assert p.stdout == ""


def _has_gpu():
    try:
        import torch
        return torch.cuda.is_available()
    except ImportError:
        return False


@pytest.mark.gpu
@pytest.mark.skipif(not _has_gpu(), reason="needs a GPU")
def test_short_run_prints_one_line_with_the_contract_fields():
    print("[gpu] bench.py --steps 3 --warmup 1", flush=True)
    p = subprocess.run([sys.executable, "-u", BENCH, "--steps", "3", "--warmup", "1"],
                       capture_output=True, text=True, timeout=600, cwd=ROOT)
    assert p.returncode == 0, p.stderr[-2000:]
    lines = [l for l in p.stdout.splitlines() if l.startswith("{")]
    assert len(lines) == 1, p.stdout[-2000:]
    b = json.loads(lines[0])
    assert b["metric"] == "candidate evaluations/sec + % of HBM/VALU roofline, 1 MI355X"
    assert b["unit"] == "candidate evaluations/s" and b["n_gpus"] == 1
    assert b["steps"] == 3 and b["warmup"] == 1
    assert b["higher_is_better"] is True and b["scaling"] == "weak" and b["vs_baseline"] is None
    assert b["dtype"] == "f32" and b["data"] == "synthetic"
    assert b["ms_per_step"] > 0 and b["value"] > 0
    cfg = b["config"]
    assert "workload" in cfg and cfg["placement_candidates"] > cfg["distinct_placement_candidates"] > 0
    assert cfg["migration_pairs"] == 2048 * 2047
    work = cfg["placement_candidates"] + cfg["migration_pairs"]
    assert abs(b["value"] * b["ms_per_step"] * 1e-3 / work - 1) < 1e-6      # value = work / step time
    r = b["roofline"]
    assert r["bound"] == "alu" and r["unit"] == "T VALU lane-ops/s"
    assert 0 < r["frac"] <= 1 and abs(r["frac"] - r["achieved"] / r["peak"]) < 1e-9
    assert abs(r["achieved"] * 1e12 * r["kernel_ms"] * 1e-3
               - r["ops_per_candidate"] * cfg["distinct_placement_candidates"]) < 1e-3 * r["achieved"] * 1e12 * r["kernel_ms"] * 1e-3
    assert r["traffic"] is None or r["traffic"] > 0
    if r["counters"] is not None:
        clk = r["counters"]["sclk_ghz_effective"]
        assert 0.5 < clk < 3.0
        assert abs(r["frac_at_measured_sclk"] - r["frac"] * 2.4 / clk) < 1e-9
    ks = b["kernels_ms"]
    assert abs(ks["k_score_candidates_per_s"] * ks["k_score"] * 1e-3 / cfg["placement_candidates"] - 1) < 1e-6
    mg = b["migration"]
    assert mg["pairs"] == cfg["migration_pairs"] and mg["call_ms"] > 0
    mr = mg["roofline"]
    assert mr["bound"] == "alu" and 0 < mr["frac"] <= 1 and abs(mr["frac"] - mr["achieved"] / mr["peak"]) < 1e-9
    assert mr["traffic"] is None or mr["traffic"] > 0
    c = b["cpu_baseline"]
    assert c["kind"] == "oracle" and c["cores"] >= 1 and c["value"] > 0 and c["unit"] == b["unit"]
    assert c["agreement"]["placement_flags_equal"] == 1.0 and c["agreement"]["migration_dst_equal"] == 1.0
    assert c["host"]["nproc"] >= c["host"]["usable"] >= 1
    for row in ("sweep", "preferred", "dispatch", "transfer"):
        assert row in b["next_rows"] and b["next_rows"][row]["roofline"]["frac"] > 0
    wv = b["next_rows"]["dispatch_waves"]
    assert wv["waves"] == 64 and wv["launches"] == 67 and wv["call_ms"] > 0
    if wv["cpu_baseline"] is not None:
        assert wv["cpu_baseline"]["agreement"]["all_outputs_equal"] == 1.0
        assert wv["cpu_baseline"]["agreement"]["final_state_equal"]
