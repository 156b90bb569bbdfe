"""The float64 oracle and its ctypes wrapper under AddressSanitizer and
UndefinedBehaviorSanitizer: the oracle is rebuilt with both (every finding
fatal) and the oracle's own pin tests run against that build in a child
process with the sanitizer runtimes preloaded.  A use-after-free in the
wrapper (arrays released while the C code still reads them) or an
out-of-bounds access in the C code ends that process with a report."""
import os
import subprocess
import sys

import pytest

from oracle import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = ["tests/test_oracle_pins.py", "tests/test_oracle_joint.py", "tests/test_oracle_mqap.py",
        "tests/test_oracle_adam.py", "tests/test_oracle_prerank.py"]


def runtime(name):
    path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True).stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_pins_pass_under_asan_and_ubsan(tmp_path):
    asan, ubsan = runtime("libasan.so"), runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("gcc sanitizer runtimes not available")
    lib = oracle.build(force=True, sanitize=True, out=str(tmp_path / "libams_oracle_asan.so"))
    env = dict(os.environ, AMS_ORACLE_LIB=lib, LD_PRELOAD=f"{asan}:{ubsan}",
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1", PYTHONPATH=ROOT)
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                        *PINS], cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error:" not in r.stderr, tail
