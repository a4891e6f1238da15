"""The oracle's pin suites run again against a build of the oracle with
AddressSanitizer and UndefinedBehaviorSanitizer: an out-of-bounds access, a use of
freed memory or undefined arithmetic anywhere the pins reach aborts the run.  The
pins check what the oracle computes; this checks how (a stray read can still
produce plausible numbers).  CPU only."""
import os
import shutil
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _libasan():
    if shutil.which("gcc") is None:
        return None
    path = subprocess.check_output(["gcc", "-print-file-name=libasan.so"], text=True).strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.mark.skipif(_libasan() is None, reason="gcc's AddressSanitizer runtime is not installed")
def test_oracle_pins_under_asan_and_ubsan():
    lib = oracle.build(force=True, sanitize=True)
    env = dict(os.environ)
    env.update(LD_PRELOAD=_libasan(), DCD_ORACLE_LIB=lib,
               # the interpreter's own allocations are not freed at exit
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1",
               OMP_NUM_THREADS="4")
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
           "tests/test_oracle_pins.py", "tests/test_parity_gates.py"]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=900)
    out = r.stdout[-4000:] + r.stderr[-4000:]
    assert r.returncode == 0, out
    assert "passed" in r.stdout and "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out
