"""Static properties of the gfx950 device code, checked on the CPU (hipcc cross-compiles).

* The dispatcher and transfer-plan kernels promise outputs bit-identical to a float64
  evaluation of their formulas in the order written, which holds only while no multiply
  and add are fused: their device code must hold no fused float64 multiply-add
  (v_fma_f64 / v_fmac_f64), which `#pragma clang fp contract(off)` guarantees.
"""
import os
import re
import subprocess

import pytest

from paper_2606_30391_amd.build import HIPCC_FLAGS, HERE

CSRC = os.path.join(HERE, "csrc")


def _device_asm(name, tmp_path):
    flags = [f for f in HIPCC_FLAGS if f not in ("-shared",)]
    out = tmp_path / (name + ".s")
    cmd = ["hipcc", *flags, "--cuda-device-only", "-S", os.path.join(CSRC, name + ".hip"), "-o", str(out)]
    proc = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    assert proc.returncode == 0, proc.stdout.decode()[-2000:]
    return out.read_text()


def _kernel_bodies(asm):
    """{kernel symbol: its instructions} from the device assembly."""
    bodies, cur = {}, None
    for line in asm.splitlines():
        m = re.match(r"^(_Z\w+):\s*(;.*)?$", line)
        if m:
            cur = m.group(1)
            bodies[cur] = []
            continue
        if cur is not None:
            s = line.strip()
            if s.startswith("s_endpgm"):
                cur = None
            elif s and not s.startswith((";", ".")):
                bodies[cur].append(s)
    return bodies


@pytest.mark.parametrize("name", ["dispatch", "transfer"])
def test_float64_kernels_have_no_fused_multiply_add(name, tmp_path):
    bodies = _kernel_bodies(_device_asm(name, tmp_path))
    assert bodies, "no kernels found in the device assembly"
    fused = {k: [i for i in v if i.startswith(("v_fma_f64", "v_fmac_f64"))] for k, v in bodies.items()}
    assert not any(fused.values()), {k: v[:3] for k, v in fused.items() if v}
    assert any(i.startswith("v_mul_f64") for v in bodies.values() for i in v)   # the float64 path is there
