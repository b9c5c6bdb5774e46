"""The oracle's C library under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only): tests/asan/oracle_asan_driver.c calls every entry point on edge
sizes (empty, single row, budgets beyond the length, NaN scores, the layer
limit of the budget split, prefill chunks past the cache) with buffers of
exactly the contracted sizes; any out-of-bounds access, leak or undefined
operation fails the run.  Built with gcc (host code only)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_oracle_under_sanitizers(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_asan")
    cmd = [gcc, "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=undefined", "-ffp-contract=off",
           os.path.join(ROOT, "tests", "asan", "oracle_asan_driver.c"), os.path.join(ROOT, "oracle", "lethe_oracle.c"),
           "-lm", "-o", exe]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:halt_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0 and run.stdout.strip() == "ok", run.stdout + run.stderr
