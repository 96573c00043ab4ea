"""Build the HIP library in place (hipcc, gfx950).

Beside the library the build records a SHA-256 over its sources, the public header and
the compiler flags (``libfestina.so.sources``); the binding refuses to load a library whose
record does not match the sources in the tree, so a stale binary is never used.
"""
from __future__ import annotations

import hashlib
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRCS = [os.path.join(HERE, "csrc", n) for n in ("festina.hip", "sweep.hip", "preferred.hip", "dispatch.hip",
                                                       "transfer.hip")]
LIB = os.path.join(HERE, "libfestina.so")
HASH_FILE = LIB + ".sources"
HEADER = os.path.join(ROOT, "include", "festina.h")

# -packed-fp32-ops: no v_pk_*_f32 from the compiler (plain fp32 VALU only)
HIPCC_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared", "-Wall",
               "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
               "-I", os.path.join(ROOT, "include")]


def source_hash() -> str:
    """SHA-256 over the library's sources, the public header and the compiler flags."""
    h = hashlib.sha256()
    for path in (*SRCS, HEADER):
        with open(path, "rb") as f:
            h.update(os.path.basename(path).encode() + b"\0" + f.read() + b"\0")
    h.update(" ".join(HIPCC_FLAGS[:-2]).encode())   # the include path is left out: it names the tree
    return h.hexdigest()


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
    with open(HASH_FILE + ".tmp", "w") as f:
        f.write(source_hash() + "\n")
    os.replace(HASH_FILE + ".tmp", HASH_FILE)
    return LIB


if __name__ == "__main__":
    print(build_hip(verbose=True))
