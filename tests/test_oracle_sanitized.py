"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only):
oracle/sanitize_driver.c compiles spk_oracle.c with both sanitizers and runs
every oracle function on small seeded inputs and edge cases (empty and
silent inputs, NaN / inf / -0 values, T = 1 and 254, strides, padding,
truncated spike lists, both winner modes, several STDP configurations) in
exactly sized heap buffers.  Any out-of-bounds access, leak or undefined
arithmetic fails the run."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
DRIVER = os.path.join(ROOT, "oracle", "sanitize_driver.c")


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
def test_oracle_is_clean_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_sanitized")
    subprocess.check_call(["gcc", "-std=c11", "-O1", "-g", "-ffp-contract=off",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                           "-fno-omit-frame-pointer", "-Wall", "-o", exe, DRIVER, "-lm"])
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    out = r.stdout + r.stderr
    assert r.returncode == 0, out[-4000:]
    assert "runtime error" not in out and "AddressSanitizer" not in out, out[-4000:]
    assert "all calls ran" in out
