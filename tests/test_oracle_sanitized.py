"""The oracle's pin suites again, against an AddressSanitizer + UndefinedBehaviorSanitizer
build of the same C source (gcc, host code only): an out-of-bounds access, a use of freed
memory, a signed overflow or any other undefined behaviour in the oracle aborts the child
run.  The oracle's results are also checked by the pins themselves, unchanged."""
import os
import subprocess
import sys

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PIN_SUITES = ["test_oracle_placement_pins.py", "test_oracle_migration_pins.py", "test_oracle_sweep_pins.py",
              "test_oracle_preferred_pins.py", "test_oracle_dispatch_pins.py", "test_oracle_dispatch_waves_pins.py",
              "test_oracle_transfer_pins.py"]


def test_pin_suites_under_asan_and_ubsan(tmp_path):
    lib = oracle.build_sanitized(str(tmp_path / "libfestina_oracle_asan.so"))
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
           *[os.path.join(HERE, f) for f in PIN_SUITES]]
    proc = subprocess.run(cmd, cwd=ROOT, env=oracle.sanitized_env(lib), stdout=subprocess.PIPE,
                          stderr=subprocess.STDOUT, text=True, timeout=900)
    tail = proc.stdout[-4000:]
    assert proc.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in proc.stdout and "runtime error:" not in proc.stdout, tail
    assert " passed" in tail, tail


@pytest.mark.parametrize("body, report", [
    # heap buffer overflow (a size known only at run time): AddressSanitizer
    ("#include <stdlib.h>\nint bad(int i) { int *a = malloc((size_t)(i - 5) * sizeof(int)); a[i] = 7; int r = a[0]; "
     "free(a); return r; }\n", "AddressSanitizer"),
    # signed overflow: UndefinedBehaviorSanitizer
    ("int bad(int i) { int x = 2147483600; return x + i * 1000; }\n", "runtime error:"),
])
def test_sanitized_build_reports_a_planted_fault(tmp_path, body, report):
    """The sanitized build and its environment do catch faults: a tiny C file with a planted
    fault, built with the same flags and loaded the same way, aborts with the report."""
    src = tmp_path / "bad.c"
    src.write_text(body)
    lib = tmp_path / "libbad.so"
    subprocess.run(["gcc", *oracle.SANITIZE_FLAGS, "-o", str(lib), str(src)], check=True)
    code = f"import ctypes; L = ctypes.CDLL({str(lib)!r}); print(L.bad(9))"
    proc = subprocess.run([sys.executable, "-c", code], env=oracle.sanitized_env(str(lib)),
                          stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, timeout=120)
    assert proc.returncode != 0, proc.stdout
    assert report in proc.stdout, proc.stdout
