"""The oracle's pins once more, against a build of the oracle instrumented
with AddressSanitizer and UndefinedBehaviorSanitizer (every report fatal):
an out-of-bounds read or write, a use after free or an undefined operation
anywhere in the C the pins exercise ends the run with a report.  The checked
library runs in a child process that preloads the ASan runtime (leak
detection off: the interpreter itself keeps memory until exit)."""
import os
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _asan_runtime():
    try:
        p = subprocess.run(["gcc", "-print-file-name=libasan.so"], capture_output=True, text=True, check=True)
    except (OSError, subprocess.CalledProcessError):
        return None
    path = p.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_oracle_pins_under_asan_and_ubsan(tmp_path):
    rt = _asan_runtime()
    if rt is None:
        pytest.skip("no AddressSanitizer runtime for gcc here")
    lib = oracle.build(path=str(tmp_path / "liboracle_checked.so"), sanitize=True)
    env = dict(os.environ, LD_PRELOAD=rt, SINGA_ORACLE_LIB=lib,
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
           os.path.join(ROOT, "tests", "test_oracle_pins.py"), os.path.join(ROOT, "tests", "test_oracle_net.py")]
    p = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    out = p.stdout + p.stderr
    assert p.returncode == 0, out[-4000:]
    assert "Sanitizer" not in out, out[-4000:]
    assert " passed" in out
