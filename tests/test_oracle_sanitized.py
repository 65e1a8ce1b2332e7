"""The CPU oracle under AddressSanitizer and UndefinedBehaviorSanitizer.

oracle/sanitize_check.c calls every oracle function on small problems (a
divisible grid with GQA, a padded grid, a padded grid with text tokens; bf16
and fp32 rounding; top-k, mass and per-sequence selection; block lists with
empty rows) with exactly-sized heap buffers.  A sanitized build must run
clean and print the same checksums as a plain build of the same sources."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ORACLE = os.path.join(os.path.dirname(HERE), "oracle")
SOURCES = [os.path.join(ORACLE, "sanitize_check.c"), os.path.join(ORACLE, "vsa2_oracle.c")]


def _build(tmp_path, name, flags):
    exe = str(tmp_path / name)
    subprocess.check_call(["gcc", "-std=c11", "-fopenmp", "-Wall", "-Wextra", *flags, "-o", exe, *SOURCES, "-lm"])
    return exe


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_runs_clean_under_asan_and_ubsan(tmp_path):
    plain = _build(tmp_path, "check_plain", ["-O1"])
    san = _build(tmp_path, "check_san", ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                                         "-fno-sanitize-recover=all"])
    env = dict(os.environ, OMP_NUM_THREADS="4", ASAN_OPTIONS="detect_leaks=1:abort_on_error=0")
    a = subprocess.run([plain], capture_output=True, text=True, env=env, timeout=300)
    b = subprocess.run([san], capture_output=True, text=True, env=env, timeout=300)
    assert a.returncode == 0, a.stderr[-2000:]
    assert b.returncode == 0, b.stderr[-4000:]
    assert "runtime error" not in b.stderr and "AddressSanitizer" not in b.stderr, b.stderr[-4000:]
    assert a.stdout.endswith("done\n") and a.stdout == b.stdout
