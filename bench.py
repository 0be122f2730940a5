#!/usr/bin/env python3
"""Throughput of the PGC step on one MI355X.

One "step" is one pipelined PGC step (t >= 1) of the whole hot path: the
per-partition gradients of every evaluated partition, the ring write, the
encode of every worker's coded gradient, the masked decode and the update,
over the full synthetic dataset resident in HBM.  The default workload is the
largest: PGC-CR (Sec. V-B), logistic regression, n = 128, c = 8, d = 8192,
N = 2,097,152 rows (64 GiB of fp32 features).

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--repeat R]
                  [--workload NAME | --config K] [--lr LR] [--seed S] [--steps-log PATH]

Prints one JSON line.  `value` is steps/s, the median of R timed passes of K
steps each; `roofline` is the gradient kernel (the dominant one) against the
8 TB/s HBM peak, timed with HIP events around its launches inside the timed
passes (every launch, or one in --time-every when there are more than 100 of
them; an event pair adds ~6 us to the step it brackets), with the whole step's
fraction beside it; `cpu_baseline` is the fp64 oracle on the host cores over a
bounded sample of the same workload.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0
DEFAULT_WORKLOAD = "cr_logistic_n128_c8_d8192"
# Timed launches of the dominant kernel to aim for when --time-every is not given.
TIMED_LAUNCH_TARGET = 100
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCES = {"hbm": os.path.join(ROOT, "paper_2607_20739_amd", "csrc", "pgc_linear.hip"),
                  "mfma": os.path.join(ROOT, "paper_2607_20739_amd", "csrc", "pgc_mlp.hip")}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash(bound):
    """Hash of the source file that holds the dominant kernel of a workload."""
    with open(KERNEL_SOURCES[bound], "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def rows_per_step(w):
    """Rows the pipelined step streams: all N for CR, one partition per FR group."""
    return w.N // w.c if w.scheme == "FR" else w.N


def algorithmic_bytes(w):
    """(gradient-kernel bytes per launch, whole-step bytes) of a pipelined step.

    Linear models: each evaluated row once (4d bytes of features + 4 of label)
    plus w.  MLP: each evaluated row's bf16 features and int32 label.  The
    whole step adds the fresh-gradient writes, one read of every ring slot the
    encode combines, the coded-gradient writes, the decoded vector and the
    update's read and write of w.
    """
    q = w.q
    rows = rows_per_step(w)
    n_eval = w.n // w.c if w.scheme == "FR" else w.n
    planes_read = w.n if w.scheme == "FR" else w.n * w.c
    n_coded = w.n // w.c if w.scheme == "FR" else w.n
    if w.model == "mlp":
        grad = rows * (2 * w.d + 4) + 4 * q
    else:
        grad = rows * (4 * w.d + 4) + 4 * q
    step = grad + 4 * q * (n_eval + planes_read + n_coded + 1 + 2)
    return grad, step


def mlp_gemm_flops(w):
    """Algorithmic FLOPs of one launch of the forward (X W1) or the weight-gradient
    (X^T dZ1) GEMM: 2 * rows * d_in * hidden each."""
    return 2.0 * rows_per_step(w) * w.d * w.hidden


def read_traffic(workload, bound):
    """HBM bytes per launch of the dominant kernel measured by rocprofv3 counters,
    if they were taken on the current kernel source; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            data = json.load(f)
    except (OSError, ValueError):
        return None
    entry = data.get(workload)
    if not entry or entry.get("kernel_source_sha256_16") != kernel_source_hash(bound):
        return None
    return entry.get("bytes_per_launch")


def cpu_baseline(w, X, y, beta0, budget_s):
    """The oracle, as it stands, on the host over the first steps of the same run.

    The oracle runs the whole workload when its fp64 copy of X fits in 8 GiB.
    Larger linear workloads run on a prefix of every partition's rows (the
    same n, c, d, masks and lr), with the rate scaled to the full row count:
    their step is per-row gradient work plus an encode / decode over n c d
    values, well under 1% of a full step at those sizes."""
    from threadpoolctl import threadpool_info
    from oracle import pgc_oracle as O
    from oracle import rng as R
    schemes = {"FR": O.FR, "CR": O.CR, "CR_REAL": O.CR_REAL}
    B = None
    if w.scheme == "CR_REAL":
        B = O.cyclic_encoding_matrix(w.n, w.c, R.null_space_generator(w.code_seed, w.c - 1, w.n))
    max_steps = 100000
    m = w.N // w.n
    shape = (w.d, w.hidden, w.classes) if w.model == "mlp" else None
    rows = m if w.N * w.d * 8 <= (8 << 30) else max(1, (4 << 30) // (w.n * w.d * 8))
    Xs = X.view(w.n, m, w.d)[:, :rows].reshape(w.n * rows, w.d).float().cpu().numpy()
    ys = y.view(w.n, m)[:, :rows].reshape(-1).cpu().numpy()
    bs = beta0.cpu().numpy()

    def run(steps):
        masks = [R.straggler_mask(w.mask_seed, t, w.policy, w.n, w.cap, w.p) for t in range(steps)]
        t0 = time.perf_counter()
        O.run(schemes[w.scheme], w.model, w.n, w.c, Xs, ys, bs, w.lr, masks, B=B, shape=shape,
              keep_coded=False, keep_alpha=False)
        return time.perf_counter() - t0

    # Marginal cost of a step from runs of 1 and 3 steps (their difference
    # cancels the one-time fp64 copy of X).
    t_one, t_three = run(1), run(3)
    per_step = max((t_three - t_one) / 2, 1e-6)
    if per_step * 30 > budget_s:
        # Slow steps (the MLP at full size): report that marginal rate.
        steps, elapsed = 2, t_three - t_one
        log("oracle: ~%.1f s per step from runs of 1 and 3 steps" % per_step)
        what = ("fp64 numpy oracle, marginal cost of a step from runs of steps t=0 and t=0..2 of the "
                "same workload and masks (%.1f s and %.1f s wall)" % (t_one, t_three))
    else:
        # Size the sample from two probes (10 and 30 steps): their difference is
        # the marginal cost of a step, the rest the one-time setup (the oracle's
        # fp64 copy of X).  The estimate is floored at a quarter of the longer
        # probe's average, so a noisy difference cannot inflate the sample.
        t_short, t_long = run(10), run(30)
        per_step = max((t_long - t_short) / 20, t_long / 30 / 4, 1e-6)
        setup = max(t_short - 10 * per_step, 0.0)
        steps = int(max(2, min(max_steps, (budget_s - setup) / per_step)))
        log("oracle: %d of %d rows per partition, ~%.1f ms per step, ~%.1f s setup; timing %d steps"
            % (rows, m, per_step * 1e3, setup, steps))
        elapsed = run(steps)
        what = ("fp64 numpy oracle over steps t=0..%d of the same workload and masks (%.1f s wall, "
                "including its one-time fp64 copy of X)" % (steps - 1, elapsed))
    threads = [i["num_threads"] for i in threadpool_info() if i.get("user_api") == "blas"]
    cores = min(max(threads) if threads else 1, len(os.sched_getaffinity(0)))
    if rows < m:
        what += ("; run on the first %d of the %d rows of every partition, rate scaled by %d/%d"
                 % (rows, m, rows, m))
    return {"value": steps / elapsed * rows / m, "unit": "steps/s", "cores": cores, "kind": "oracle",
            "sample": what}


def copy_calibration(nbytes):
    """Launch torch's copy kernel on nbytes bytes 20 times: it reads and writes
    exactly nbytes per launch, which scales the FETCH_SIZE / WRITE_SIZE counters."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(20):
        dst.copy_(src)
    torch.cuda.synchronize()
    log("copied %d bytes 20 times" % (src.numel() * 4))
    return 0


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps per pass (default: about 1 s of steps, between 20 and 100,000)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps before the timed ones (default: at least 20 and at least "
                         "0.25 s of steps, so the GPU's clocks have ramped up)")
    ap.add_argument("--repeat", type=int, default=3,
                    help="timed passes of --steps steps each; value is their median")
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--config", type=int, default=0, metavar="K",
                    help="run the K-th listed workload instead (1 = the small case, 5 = the default)")
    ap.add_argument("--lr", type=float, default=None, help="override the workload's learning rate")
    ap.add_argument("--seed", type=int, default=None, help="override the workload's data and mask seed")
    ap.add_argument("--steps-log", default="", metavar="PATH",
                    help="write one JSON line per step of the untimed repeat pass (t, stragglers, "
                         "survivors, decode scale, step time) and, when they take at most 512 MiB, "
                         "every step's decoded gradient and weights to PATH.npz (tests/"
                         "steps_log_errors.py adds the per-step errors against the oracle)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="wall-time budget of the oracle baseline (0 disables it)")
    ap.add_argument("--all-kernel-times", action="store_true",
                    help="time every kernel with HIP events (adds event overhead to the step)")
    ap.add_argument("--time-every", type=int, default=None,
                    help="bracket one launch in this many of each timed kernel with HIP events "
                         "(an event pair costs ~6 us of step time; default: every launch when the "
                         "timed passes hold at most %d, else enough to time about that many)"
                         % TIMED_LAUNCH_TARGET)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES bytes 20 times and exit "
                         "(a known-size reference for the HBM byte counters)")
    args = ap.parse_args()
    if args.copy_calibration:
        return copy_calibration(args.copy_calibration)
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        return 2
    if ((args.steps is not None and args.steps < 1) or (args.warmup is not None and args.warmup < 1)
            or args.repeat < 1):
        print("--steps, --warmup and --repeat must be >= 1 (the first warm-up step is the pipeline "
              "fill t = 0)", file=sys.stderr)
        return 2

    import torch
    import paper_2607_20739_amd as P
    from dataclasses import replace
    from workloads import ORDER, WORKLOADS, make_inputs

    name = args.workload
    if args.config:
        if not 1 <= args.config <= len(ORDER):
            print("--config must be 1..%d" % len(ORDER), file=sys.stderr)
            return 2
        name = ORDER[args.config - 1]
    if name not in WORKLOADS:
        print("unknown workload %r (known: %s)" % (name, ", ".join(ORDER)), file=sys.stderr)
        return 2
    w = WORKLOADS[name]
    if args.lr is not None:
        w = replace(w, lr=args.lr)
    if args.seed is not None:
        w = replace(w, seed=args.seed)
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        return 1
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    log("workload %s: generating inputs" % w.name)
    X, y, beta0 = make_inputs(w, device=dev)
    masks = []

    def mask(t):
        while len(masks) <= t:
            masks.append(P.pgc_make_mask(w.mask_seed, len(masks), w.policy, w.n, w.cap, w.p))
        return masks[t]
    sess = P.PGCSession(w.scheme, w.n, w.c, w.model, w.N, w.d, hidden=w.hidden, classes=w.classes,
                        code_seed=w.code_seed, device=dev)
    wv = beta0.clone()
    t_warm = time.perf_counter()
    if args.warmup is not None:
        warmup = args.warmup
        for t in range(warmup):
            sess.step(X, y, wv, mask(t), w.lr)
    else:
        warmup = 0
        while warmup < 20 or time.perf_counter() - t_warm < 0.25:
            for _ in range(20):
                sess.step(X, y, wv, mask(warmup), w.lr)
                warmup += 1
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    warm_s = time.perf_counter() - t_warm
    steps = args.steps
    if steps is None:
        # About one second of steps per pass (the warm-up's rate, which
        # includes the slower t = 0 step, errs on the short side).
        steps = int(min(100000, max(20, round(warmup / max(warm_s, 1e-9)))))
    log("warm-up: %d steps (t = 0 fills the pipeline); timing %d passes of %d steps"
        % (warmup, args.repeat, steps))
    total = warmup + args.repeat * steps
    mask(total - 1)   # every step's straggler mask, drawn before the timed passes

    stream = torch.cuda.current_stream(dev)
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    # HIP events bracket only the dominant kernel(s) inside the timed region.
    timed_kernels = ([P.PGC_KERNEL_MLP_FORWARD, P.PGC_KERNEL_MLP_WGRAD] if w.model == "mlp"
                     else [P.PGC_KERNEL_GRADIENT])
    if args.all_kernel_times:
        timed_kernels = True
    period = args.time_every
    if period is None:
        period = max(1, (args.repeat * steps) // TIMED_LAUNCH_TARGET)
    P.pgc_set_timing(sess.ctx, timed_kernels)
    P.pgc_set_timing_period(sess.ctx, max(1, period))
    pass_ms = []
    t = warmup
    for _ in range(args.repeat):
        torch.cuda.synchronize()
        start.record(stream)
        for _ in range(steps):
            sess.step(X, y, wv, mask(t), w.lr)
            t += 1
        stop.record(stream)
        torch.cuda.synchronize()
        pass_ms.append(start.elapsed_time(stop))
    kernels = {"gradient": P.PGC_KERNEL_GRADIENT, "reduce": P.PGC_KERNEL_REDUCE, "code": P.PGC_KERNEL_CODE,
               "mlp_cast": P.PGC_KERNEL_MLP_CAST, "mlp_forward": P.PGC_KERNEL_MLP_FORWARD,
               "mlp_head": P.PGC_KERNEL_MLP_HEAD, "mlp_wgrad": P.PGC_KERNEL_MLP_WGRAD}
    per_launch, timed_launches = {}, {}
    for kname, kid in kernels.items():
        ms, launches = P.pgc_kernel_time(sess.ctx, kid)
        if launches:
            per_launch[kname] = ms / launches
            timed_launches[kname] = launches
    P.pgc_set_timing(sess.ctx, [])
    if not bool(torch.isfinite(wv).all()):
        print("non-finite weights after the timed steps", file=sys.stderr)
        return 1

    # The warm-up step t = 0 (every worker evaluates all of its partitions),
    # timed on its own after starting the session over.  The same session
    # then repeats every step untimed, reading the decoded gradient out after
    # each one; its final weights must equal the timed passes' bit for bit.
    sess.restart()
    w_check = beta0.clone()
    torch.cuda.synchronize()
    start.record(stream)
    sess.step(X, y, w_check, mask(0), w.lr)
    stop.record(stream)
    torch.cuda.synchronize()
    warmup_step_ms = start.elapsed_time(stop)
    steps_log = open(args.steps_log, "w") if args.steps_log else None
    # Every step's decoded gradient and weights, where they fit in 512 MiB.
    keep_vectors = steps_log is not None and 2 * total * w.q * 4 <= (512 << 20)
    step_ms, ghats, ws = [warmup_step_ms], [], []

    def keep(t):
        if keep_vectors:
            ghats.append(sess.decoded().cpu())
            ws.append(w_check.cpu())

    keep(0)
    for t in range(1, total):
        if steps_log:
            start.record(stream)
        sess.step(X, y, w_check, mask(t), w.lr)
        if steps_log:
            stop.record(stream)
        sess.decoded()
        if steps_log:
            torch.cuda.synchronize()
            step_ms.append(start.elapsed_time(stop))
            keep(t)
    torch.cuda.synchronize()
    if steps_log:
        for t in range(total):
            survivors, _, scale = sess.decode_coeffs(mask(t))
            rec = {"t": t, "stragglers": [int(i) for i in mask(t).nonzero()[0]],
                   "survivors": [int(i) for i in survivors], "decode_scale": scale, "step_ms": step_ms[t]}
            steps_log.write(json.dumps(rec) + "\n")
        steps_log.close()
        if keep_vectors:
            import numpy as np
            np.savez(args.steps_log + ".npz", ghat=torch.stack(ghats).numpy(), w=torch.stack(ws).numpy(),
                     workload=w.name, lr=w.lr, seed=w.seed)
    reproduced = bool(torch.equal(w_check, wv))
    if not reproduced:
        log("the repeated pass did not reproduce the timed passes' weights bit for bit")
    del w_check

    ms_per_step = sorted(pass_ms)[len(pass_ms) // 2] / steps
    steps_per_s = 1000.0 / ms_per_step
    grad_bytes, step_bytes = algorithmic_bytes(w)
    step_gbs = step_bytes / (ms_per_step * 1e-3) / 1e9
    if w.model == "mlp":
        dominant = max(("mlp_forward", "mlp_wgrad"), key=lambda k: per_launch[k])
        achieved = mlp_gemm_flops(w) / (per_launch[dominant] * 1e-3) / 1e12
        roofline = {"bound": "mfma", "kernel": dominant, "achieved": achieved,
                    "peak": BF16_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                    "frac": achieved / BF16_MFMA_PEAK_TFLOPS, "traffic": read_traffic(w.name, "mfma"),
                    "timed_launches": timed_launches[dominant]}
    else:
        achieved = grad_bytes / (per_launch["gradient"] * 1e-3) / 1e9
        roofline = {"bound": "hbm", "kernel": "linear_gradient_kernel", "achieved": achieved,
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                    "traffic": read_traffic(w.name, "hbm"),
                    "timed_launches": timed_launches["gradient"],
                    "step_achieved": step_gbs, "step_frac": step_gbs / HBM_PEAK_GBS}
    log("step %.4f ms (passes: %s ms); per launch (ms): %s" % (
        ms_per_step, ", ".join("%.2f" % p for p in pass_ms),
        ", ".join("%s %.4f" % kv for kv in per_launch.items())))

    baseline = None
    if args.cpu_seconds > 0:
        log("oracle baseline on the host (budget %.0f s)" % args.cpu_seconds)
        baseline = cpu_baseline(w, X, y, beta0, args.cpu_seconds)

    rows = rows_per_step(w)
    out = {
        "metric": "PGC steps/sec & samples/sec at 1 MI355X; achieved HBM GB/s vs peak",
        "value": steps_per_s,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.model == "mlp" else "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "scheme": w.scheme, "loss": w.model, "n": w.n, "c": w.c,
                   "N": w.N, "d": w.d, "q": w.q, "lr": w.lr, "seed": w.seed},
        "repeat": args.repeat,
        "pass_ms": pass_ms,
        "samples_per_s": {"unique_rows": rows * steps_per_s, "worker_samples": w.N * steps_per_s},
        "step_hbm_gbs": step_gbs,
        "kernel_ms_per_launch": per_launch,
        "warmup_step_ms": warmup_step_ms,
        "timed_pass_reproduced": reproduced,
        "roofline": roofline,
        "cpu_baseline": baseline,
    }
    print(json.dumps(out), flush=True)
    sess.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
