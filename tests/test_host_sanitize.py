"""The library's host tables (placement, straggler masks, the delay model, the
real-valued cyclic code, decode coefficients, the minimum-norm solver) built
with g++ under AddressSanitizer and UndefinedBehaviorSanitizer and exercised by
tests/host_sanitize.cpp, which checks results as well as memory and arithmetic
errors.  These sources are plain C++, so no GPU or HIP compiler is involved."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2607_20739_amd", "csrc")


def test_host_tables_pass_under_address_and_undefined_behaviour_sanitizers(tmp_path):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ is not available")
    exe = str(tmp_path / "host_sanitize")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
           "-fno-sanitize-recover=all", "-I", CSRC, os.path.join(ROOT, "tests", "host_sanitize.cpp"),
           os.path.join(CSRC, "pgc_codes.cpp"), "-o", exe]
    build = subprocess.run(cmd, capture_output=True, text=True)
    assert build.returncode == 0, build.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    run = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert run.returncode == 0, run.stderr[-4000:]
    assert "all checks passed" in run.stdout
