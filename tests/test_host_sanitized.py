"""The host-side tests again, against the cache core built with
AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The sanitizer runtimes must be loaded before Python starts, so the tests run
in a child interpreter with them preloaded; any report (out-of-bounds
access, use after free, undefined behaviour) fails the child run. The
hipRTC compilation test is left out (it exercises the compiler, not this
library, and is slow under the sanitizers).
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name):
    try:
        path = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True,
                              text=True, timeout=60).stdout.strip()
    except (OSError, subprocess.SubprocessError):
        return None
    return path if os.path.isabs(path) and os.path.exists(path) else None


def test_host_core_under_sanitizers():
    asan, ubsan = _runtime("libasan.so"), _runtime("libubsan.so")
    if not asan or not ubsan:
        pytest.skip("gcc sanitizer runtimes not found")
    env = dict(os.environ, TRI_FAKE_SANITIZE="1", LD_PRELOAD=f"{asan}:{ubsan}",
               ASAN_OPTIONS="detect_leaks=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
           "-k", "not generated_source_compiles",
           "tests/test_host_cache.py", "tests/test_host_tuning.py", "tests/test_host_fuzz.py"]
    r = subprocess.run(cmd, cwd=ROOT, env=env, capture_output=True, text=True, timeout=1200)
    tail = (r.stdout + r.stderr)[-4000:]
    assert r.returncode == 0, tail
    assert "ERROR: AddressSanitizer" not in tail and "runtime error:" not in tail, tail
