"""The PGC step driven by a plain C program through include/pgc.h (device
memory from the HIP C runtime API; no Python binding, no torch on the GPU),
checked after every step against the fp64 oracle on the same inputs."""

import os
import shutil
import subprocess

import numpy as np
import pytest

from workloads import Workload, make_inputs, POLICY_UNIFORM_COUNT

from _parity import FP32_TOL, normwise_error, oracle_masks, oracle_run

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_DIR = os.path.join(ROOT, "paper_2607_20739_amd")
SCHEME = {"FR": 0, "CR": 1, "CR_REAL": 2}
MODEL = {"logistic": 0, "lsq": 1}

CASES = [
    Workload("c_abi_cr_logistic", "CR", "logistic", n=6, c=3, N=6 * 500, d=260, lr=0.1, steps=9,
             policy=POLICY_UNIFORM_COUNT, cap=2, seed=81),
    Workload("c_abi_fr_lsq", "FR", "lsq", n=8, c=4, N=8 * 300, d=1024, lr=0.02, steps=9,
             policy=POLICY_UNIFORM_COUNT, cap=3, seed=82),
]


@pytest.fixture(scope="module")
def c_program(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("cabi_gpu") / "abi_gpu")
    gcc = shutil.which("gcc")
    assert gcc is not None
    subprocess.run([gcc, "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                    "-I", "/opt/rocm/include", os.path.join(HERE, "c", "abi_gpu.c"), "-L", LIB_DIR, "-lpgc",
                    "-L", "/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath," + LIB_DIR, "-Wl,-rpath,/opt/rocm/lib",
                    "-o", exe], check=True, capture_output=True, text=True)
    return exe


@pytest.mark.parametrize("w", CASES, ids=[w.name for w in CASES])
def test_c_program_trajectory_matches_oracle(c_program, w, tmp_path):
    print("\n[gpu case] C caller %s" % w.name, flush=True)
    X, y, beta0 = make_inputs(w)          # drawn on the host; the C program copies them to the GPU
    Xh, yh, bh = X.numpy(), y.numpy(), beta0.numpy()
    masks = oracle_masks(w)
    (tmp_path / "in.bin").write_bytes(np.concatenate([Xh.ravel(), yh, bh]).astype(np.float32).tobytes())
    (tmp_path / "masks.bin").write_bytes(np.stack(masks).astype(np.uint8).tobytes())
    res = subprocess.run([c_program, str(SCHEME[w.scheme]), str(MODEL[w.model]), str(w.n), str(w.c), str(w.d),
                          str(w.N), str(w.steps), repr(w.lr), str(tmp_path / "in.bin"), str(tmp_path / "masks.bin"),
                          str(tmp_path / "out.bin")], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stdout + res.stderr
    out = np.frombuffer((tmp_path / "out.bin").read_bytes(), dtype=np.float32).reshape(w.steps, 2, w.d)
    ref = oracle_run(w, Xh, yh, bh, masks)
    for t, o in enumerate(ref):
        assert normwise_error(out[t, 0], o.ghat) <= FP32_TOL, "step %d ghat" % t
        assert normwise_error(out[t, 1], o.beta) <= FP32_TOL, "step %d w" % t
