"""Build the HIP library in place (hipcc, gfx950)."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRCS = [os.path.join(HERE, "csrc", n) for n in ("festina.hip", "sweep.hip", "preferred.hip", "dispatch.hip",
                                                       "transfer.hip")]
LIB = os.path.join(HERE, "libfestina.so")

# -packed-fp32-ops: no v_pk_*_f32 from the compiler (plain fp32 VALU only)
HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-I", os.path.join(ROOT, "include")]


def build_hip(verbose: bool = False) -> str:
    cmd = ["hipcc", *HIPCC_FLAGS, "-o", LIB + ".tmp", *SRCS]
    proc = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    out = proc.stdout.decode()
    noise = "packed-fp32-ops"
    msgs = "\n".join(l for l in out.splitlines() if noise not in l and l.strip())
    if proc.returncode != 0:
        raise RuntimeError(f"hipcc failed ({proc.returncode}):\n{out}")
    if verbose and msgs:
        print(msgs)
    os.replace(LIB + ".tmp", LIB)
    return LIB


if __name__ == "__main__":
    print(build_hip(verbose=True))
