"""The CPU oracle's C code under AddressSanitizer and UndefinedBehaviorSanitizer
(gcc, host code only): tests/native/oracle_sanitize.c compiles qg_oracle.c
into a driver that calls every entry point over padded rows, random finite
bf16 patterns, tiny and subnormal values, signed zeros, the extremes and
non-finite input. Any out-of-bounds access, leak or undefined operation
aborts the run."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "native", "oracle_sanitize.c")
FLAGS = ["-O1", "-g", "-std=c11", "-ffp-contract=off", "-fno-omit-frame-pointer", "-Wall",
         "-Wno-unknown-pragmas", "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]


def test_oracle_is_clean_under_sanitizers(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_sanitize")
    build = subprocess.run(["gcc", *FLAGS, "-o", exe, SRC, "-lm"], capture_output=True, text=True)
    if build.returncode != 0 and "sanitize" in build.stderr and "cannot find" in build.stderr:
        pytest.skip("sanitizer runtime not installed: " + build.stderr[-200:])
    assert build.returncode == 0, build.stderr[-2000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, timeout=120, env=env)
    assert run.returncode == 0, (run.stdout + run.stderr)[-3000:]
    assert "oracle sanitizer run done" in run.stdout
    assert "runtime error" not in run.stderr and "AddressSanitizer" not in run.stderr
