"""Host-side checks of bench.py: its argument guards, its algorithmic-work
accounting, and when it reports measured HBM traffic.  No GPU needed."""

import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from workloads import ORDER, WORKLOADS  # noqa: E402


def run_bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120)


def test_bench_measures_one_gpu_only():
    res = run_bench("--gpus", "2")
    assert res.returncode == 2
    assert "one GPU" in res.stderr
    assert res.stdout == ""


def test_bench_rejects_an_empty_timed_region():
    for args in (("--steps", "0"), ("--repeat", "0"), ("--warmup", "0")):
        res = run_bench(*args)
        assert res.returncode == 2, args
        assert "--steps" in res.stderr and "--repeat" in res.stderr


def test_bench_defaults_to_the_largest_workload():
    """With no --workload / --config the bench runs the 64 GiB PGC-CR workload."""
    w = WORKLOADS[bench.DEFAULT_WORKLOAD]
    assert bench.DEFAULT_WORKLOAD == ORDER[-1]
    assert (w.scheme, w.model, w.n, w.c, w.d, w.N) == ("CR", "logistic", 128, 8, 8192, 2097152)
    assert w.N * w.d * 4 == 64 << 30


@pytest.mark.parametrize("name", [n for n in ORDER if WORKLOADS[n].model != "mlp"])
def test_linear_step_bytes_follow_the_per_row_accounting(name):
    w = WORKLOADS[name]
    # Each evaluated row: d fp32 features and one fp32 label, read once; plus w.
    # FR evaluates one partition per group (N / c rows); CR every partition.
    rows = w.N // w.c if w.scheme == "FR" else w.N
    grad, step = bench.algorithmic_bytes(w)
    assert grad == rows * (4 * w.d + 4) + 4 * w.d
    assert step > grad
    # The rest of the step (ring, coded words, w) is under 1% of the stream
    # except for the cache-resident d = 64 case.
    if w.d >= 1024:
        assert (step - grad) < 0.01 * grad


def test_mlp_gemm_flops_are_two_per_multiply_add():
    w = WORKLOADS["cr_mlp_n64_c4_784x1024x10"]
    assert bench.mlp_gemm_flops(w) == 2.0 * 1048576 * 784 * 1024


def test_traffic_is_reported_only_for_the_kernel_source_it_was_measured_on(monkeypatch):
    with open(bench.TRAFFIC_FILE) as f:
        data = json.load(f)
    name = "crreal_lsq_n8_c3_d1024"
    entry = data[name]
    monkeypatch.setattr(bench, "kernel_source_hash", lambda bound: entry["kernel_source_sha256_16"])
    assert bench.read_traffic(name, "hbm") == entry["bytes_per_launch"]
    monkeypatch.setattr(bench, "kernel_source_hash", lambda bound: "0" * 16)
    assert bench.read_traffic(name, "hbm") is None
    assert bench.read_traffic("no_such_workload", "hbm") is None


def test_recorded_traffic_covers_the_algorithmic_bytes():
    """Counters read at least what the kernel must stream (X and y once)."""
    with open(bench.TRAFFIC_FILE) as f:
        data = json.load(f)
    for name, entry in data.items():
        w = WORKLOADS[name]
        if w.model == "mlp":
            must_read = w.N * w.d * 2   # bf16 X
        else:
            must_read = bench.algorithmic_bytes(w)[0] - 4 * w.d
        assert entry["read_bytes"] >= 0.999 * must_read, name


def test_cpu_baseline_reports_the_oracle_rate_on_a_bounded_sample():
    from workloads import make_inputs
    w = WORKLOADS["fr_logistic_n4_c2_d64"]
    X, y, beta0 = make_inputs(w)
    res = bench.cpu_baseline(w, X, y, beta0, budget_s=1.0)
    assert res["kind"] == "oracle" and res["unit"] == "steps/s"
    assert res["value"] > 0 and res["cores"] >= 1
    assert "oracle" in res["sample"] and "rows" not in res["sample"]   # small X: every row is used
