"""Build libpgc.so (the C-ABI library of include/pgc.h) for gfx950 with hipcc.

Usage: python -m paper_2607_20739_amd.build   (or build() from Python)

Every HIP and C++ source under csrc/ is compiled with
  --offload-arch=gfx950 -O3 -std=c++17 -fPIC
  -Xclang -target-feature -Xclang -packed-fp32-ops
(the last pair keeps the compiler from emitting packed fp32 VALU instructions;
the host pass reports the feature as unknown, which is harmless) and linked
into paper_2607_20739_amd/libpgc.so next to this file, linked against ROCm's
roctx library for the per-step profiler ranges.
"""

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libpgc.so")
SOURCES = sorted(f for f in os.listdir(CSRC) if f.endswith((".cpp", ".hip")))
ARCH = "gfx950"
ROCM_LIB = "/opt/rocm/lib"   # librocprofiler-sdk-roctx (per-step profiler ranges)


def hipcc():
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the HIP library cannot be built")
    return path


def common_flags():
    return ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-Wall",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", INCLUDE, "-I", CSRC]


def _compile(src):
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [hipcc()] + common_flags() + ["-c", os.path.join(CSRC, src), "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("compiling %s failed:\n%s\n%s" % (src, " ".join(cmd), res.stderr))
    return obj


def build(verbose=False):
    """Compile and link libpgc.so; returns its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(SOURCES)) as pool:
        objs = list(pool.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs + [
        "-L" + ROCM_LIB, "-Wl,-rpath," + ROCM_LIB, "-lrocprofiler-sdk-roctx"]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError("linking libpgc.so failed:\n%s\n%s" % (" ".join(cmd), res.stderr))
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
