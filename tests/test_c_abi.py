"""The C ABI from a plain C99 program (no Python binding): include/pgc.h compiles
with gcc -std=c99 -Wall -Werror, the program links against libpgc.so, and the
host-only entry points it calls return what the oracle and the paper's printed
example give.  No GPU is used."""

import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import pgc_oracle as O
from oracle import rng as R

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_DIR = os.path.join(ROOT, "paper_2607_20739_amd")


@pytest.fixture(scope="module")
def c_output(tmp_path_factory):
    gcc = shutil.which("gcc")
    if gcc is None or not os.path.exists(os.path.join(LIB_DIR, "libpgc.so")):
        pytest.fail("needs gcc and the built libpgc.so")
    exe = str(tmp_path_factory.mktemp("cabi") / "abi_host")
    subprocess.run([gcc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-I", os.path.join(ROOT, "include"),
                    os.path.join(HERE, "c", "abi_host.c"), "-L", LIB_DIR, "-lpgc",
                    "-Wl,-rpath," + LIB_DIR, "-o", exe], check=True, capture_output=True, text=True)
    res = subprocess.run([exe], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    lines = {}
    for line in res.stdout.splitlines():
        key, _, rest = line.partition(" ")
        lines[key] = rest
    assert "done" in lines and not any(k == "status" for k in lines), res.stdout
    return lines


def _ints(s):
    return [int(v) for v in s.split()]


def test_fr_placement_and_schedule_from_c(c_output):
    # Sec. III prints this placement for n = 4, c = 2: W0, W1 hold D0, D1; W2, W3 hold D2, D3.
    assert _ints(c_output["placement_fr"]) == [0, 1, 0, 1, 2, 3, 2, 3]
    P = O.placement(O.FR, 4, 2)
    assert _ints(c_output["schedule_fr_t2"]) == [P[i][O.evaluated_slot(2, 2)] for i in range(4)]


def test_decode_coefficients_from_c_match_the_oracle(c_output):
    assert _ints(c_output["survivors_fr"]) == [1, 2, 3]
    d, scale = O.decode_weights(O.FR, 4, 2, [1, 2, 3])
    got = c_output["decode_fr"].split()
    assert [float(v) for v in got[:3]] == d.tolist() and float(got[4]) == scale
    assert _ints(c_output["placement_cr"]) == [k for row in O.placement(O.CR, 5, 3) for k in row]
    assert _ints(c_output["survivors_cr"]) == [0, 2, 4]
    d, scale = O.decode_weights(O.CR, 5, 3, [0, 2, 4])
    got = c_output["decode_cr"].split()
    assert [float(v) for v in got[:3]] == d.tolist() and float(got[4]) == scale


def test_errors_and_context_free_calls_from_c(c_output):
    status, _, msg = c_output["step_unbound"].partition(" ")
    assert int(status) == -5 and "workspace" in msg            # PGC_ESTATE
    assert int(c_output["too_many"].split()[0]) == -2           # PGC_ESTRAGGLERS
    assert int(c_output["init_bad"]) == -1                      # PGC_EINVAL: c does not divide n for FR
    assert int(c_output["splitmix64_0_0"]) == R.splitmix64(0, 0)
    assert _ints(c_output["mask_exact_8_2_t3"]) == R.straggler_mask((5 << 32) | 1, 3, R.POLICY_EXACT, 8, 2).tolist()
    assert int(c_output["workspace_fr"]) > 0
