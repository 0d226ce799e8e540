"""AddressSanitizer + UndefinedBehaviorSanitizer run (CPU, no GPU).

tests/emu/sanitize_driver.cpp runs the kernels' row bodies in the CPU
emulation on small cascades of every flag combination, and the C ABI's
host-side validation and size arithmetic on bad, extreme and boundary
arguments, all compiled with -fsanitize=address,undefined for the host.  A
sanitizer report or a failed check fails the test."""

import os
import shutil
import subprocess
import sys

import pytest

sys.path.insert(0, os.path.join(os.path.dirname(__file__), "emu"))


def test_emulation_and_host_validation_under_asan_ubsan():
    if shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"):
        pytest.skip("hipcc not available")
    import build_sanitize
    exe = build_sanitize.build()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    proc = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    out = proc.stdout + proc.stderr
    assert "ERROR: AddressSanitizer" not in out, out[-4000:]
    assert "runtime error:" not in out, out[-4000:]
    assert proc.returncode == 0, out[-4000:]
    assert "sanitize driver ok" in proc.stdout
