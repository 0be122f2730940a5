#!/usr/bin/env python3
"""Comparison studies on the PGC kernels of one MI355X.

  python studies.py baselines   GPU cost per step of DGD, IS-SGD, GC and PGC
                                (the per-step comparison of Fig. 3, 7 and 10a,
                                measured on the simulated workers' kernels)
  python studies.py naive-cr    decoding coefficients and loss of naive PGC-CR
                                beside PGC-FR and PGC-CR, n = 12, c = 6 (Sec. V-A)
  python studies.py delays      simulated cluster time per step under exponential
                                worker delays, and simulated time to a target
                                loss (Sec. VI-B)

Every scheme runs through the same library entry points and kernels as the
PGC step; DGD is FR with c = 1, GC is a context with pipelining switched off
(GC-CR being the real-valued cyclic code, exact under stragglers), IS-SGD
averages the survivors' uncoded gradients.  The training loss is a diagnostic
computed with torch outside the hot path.  Each study prints one JSON line per
case and, with --out, writes a markdown summary.
"""

import argparse
import json
import math
import os
import sys

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from workloads import Workload, make_inputs, POLICY_EXACT  # noqa: E402

# name: (library scheme, partitions per worker as a function of s, pipelined,
#        stragglers it tolerates as a function of s)
SCHEMES = {
    "DGD": ("FR", lambda s: 1, True, lambda s: 0),
    "IS-SGD": ("IS_SGD", lambda s: 1, True, lambda s: s),
    "GC-FR": ("FR", lambda s: s + 1, False, lambda s: s),
    "GC-CR": ("CR_REAL", lambda s: s + 1, False, lambda s: s),
    "PGC-FR": ("FR", lambda s: s + 1, True, lambda s: s),
    "PGC-CR": ("CR", lambda s: s + 1, True, lambda s: s),
    "naive PGC-CR": ("CR_REAL", lambda s: s + 1, True, lambda s: s),
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def scheme_setup(name, s):
    lib_scheme, c_of, pipelined, s_of = SCHEMES[name]
    return lib_scheme, c_of(s), pipelined, s_of(s)


def worker_partitions(name, s, t):
    """Partitions one worker evaluates at step t (the warm-up step evaluates all c)."""
    _, c, pipelined, _ = scheme_setup(name, s)
    return c if (not pipelined or t == 0) else 1


def rows_streamed(name, s, N):
    """Feature rows the all-workers simulation reads in a steady step.  FR
    groups share one evaluation; without pipelining every copy of a partition
    is evaluated at the same weights, so the c copies are computed once."""
    lib_scheme, c, pipelined, _ = scheme_setup(name, s)
    return N // c if (lib_scheme == "FR" and pipelined) else N


def worker_rows(name, s, m):
    """Feature rows one worker reads per steady step: c partitions for GC, one otherwise."""
    return worker_partitions(name, s, 1) * m


def decoding_alpha(ctx, n, c, mask, B):
    """Effective weight alpha[m, k] of partition k's gradient as sent by the
    m-th survivor j_m: n * scale * d_m * B[j_m, k], so that for an exact
    decoder sum_m alpha[m, k] = 1 (Sec. V-A), and PGC-CR's weight is 1 / mu.
    Returns (alpha over the held (survivor, partition) pairs, survivors)."""
    import numpy as np
    import paper_2607_20739_amd as P
    surv, d, scale = P.pgc_decode_coeffs(ctx, mask, n)
    held = B[surv] != 0.0
    alpha = n * scale * d[:, None] * B[surv]
    return np.where(held, alpha, np.nan), surv


def logistic_loss(X, y, w):
    import torch
    z = X @ w
    return float((torch.nn.functional.softplus(z) - y * z).mean())


def train(name, s, w_data, X, y, beta0, masks, lr, record_alpha=False, loss_every=1):
    """Run one scheme on the GPU; returns per-step losses (before each step and
    after the last) and, for record_alpha, the per-step alpha extremes."""
    import numpy as np
    import torch
    import paper_2607_20739_amd as P
    lib_scheme, c, pipelined, _ = scheme_setup(name, s)
    n = w_data.n
    sess = P.PGCSession(lib_scheme, n, c, "logistic", w_data.N, w_data.d, code_seed=w_data.code_seed,
                        device=X.device, pipelined=pipelined)
    B = P.pgc_encoding_matrix(sess.ctx, n)
    wv = beta0.clone()
    losses, alphas = [], []
    try:
        for t, mask in enumerate(masks):
            if t % loss_every == 0:
                losses.append((t, logistic_loss(X, y, wv)))
            if record_alpha:
                a, _ = decoding_alpha(sess.ctx, n, c, mask, B)
                alphas.append((float(np.nanmax(a)), float(np.nanmin(a))))
            sess.step(X, y, wv, mask, lr)
        losses.append((len(masks), logistic_loss(X, y, wv)))
        torch.cuda.synchronize()
    finally:
        sess.close()
    return losses, alphas


def delay_masks(n, s_tol, steps, seed, mean, t_p, name, s):
    """Masks and simulated step durations of the delay model for one scheme."""
    import paper_2607_20739_amd as P
    masks, secs = [], []
    for t in range(steps):
        mask, _, sec = P.pgc_delay_step(seed, t, n, s_tol, mean, worker_partitions(name, s, t) * t_p)
        masks.append(mask)
        secs.append(sec)
    return masks, secs


# ----------------------------------------------------------------------------
# baselines: GPU cost per step
# ----------------------------------------------------------------------------

def timed_steps(P, torch, sess, X, y, beta0, masks, warmup, steps, lr=0.01):
    """GPU milliseconds per step over `steps` steps after `warmup` untimed ones."""
    dev = X.device
    wv = beta0.clone()
    for t in range(warmup):
        sess.step(X, y, wv, masks[t], lr)
    stream = torch.cuda.current_stream(dev)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for t in range(warmup, warmup + steps):
        sess.step(X, y, wv, masks[t], lr)
    stop.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(stop) / steps


def study_baselines(args, out):
    import numpy as np
    import torch
    import paper_2607_20739_amd as P
    n, d, m = args.n, args.d, args.rows_per_partition
    N = n * m
    dev = torch.device("cuda", 0)
    data = Workload("study_baselines", "FR", "logistic", n=n, c=1, N=N, d=d, lr=0.01, steps=1,
                    policy=POLICY_EXACT, cap=0, seed=11, code_seed=11)
    X, y, beta0 = make_inputs(data, device=dev)
    total = args.warmup + args.steps
    worker_ms = {}

    def one_worker_ms(r):
        # One worker's step on its own GPU: full-batch gradient of its r rows.
        if r not in worker_ms:
            sess = P.PGCSession("FR", 1, 1, "logistic", r, d, device=dev)
            masks = [np.zeros(1, np.uint8)] * total
            try:
                worker_ms[r] = float(np.median([timed_steps(P, torch, sess, X[:r], y[:r], beta0, masks,
                                                            args.warmup, args.steps)
                                                for _ in range(args.repeats)]))
            finally:
                sess.close()
        return worker_ms[r]

    rows = []
    for s in args.s:
        for name in SCHEMES:
            lib_scheme, c, pipelined, s_tol = scheme_setup(name, s)
            if name == "DGD" and s != args.s[0]:
                continue
            sess = P.PGCSession(lib_scheme, n, c, "logistic", N, d, code_seed=11, device=dev,
                                pipelined=pipelined)
            masks = [P.pgc_make_mask(7, t, POLICY_EXACT, n, s_tol) for t in range(total)]
            try:
                reps = [timed_steps(P, torch, sess, X, y, beta0, masks, args.warmup, args.steps)
                        for _ in range(args.repeats)]
            finally:
                sess.close()
            ms = float(np.median(reps))
            r = rows_streamed(name, s, N)
            wr = worker_rows(name, s, m)
            rec = {"study": "baselines", "scheme": name, "s": s if s_tol else 0, "c": c, "n": n, "d": d,
                   "N": N, "ms_per_step": ms, "ms_repeats": reps, "rows_per_step": r,
                   "hbm_gbs": r * (4 * d + 4) / (ms * 1e-3) / 1e9,
                   "partitions_per_worker": worker_partitions(name, s, 1), "worker_rows": wr,
                   "worker_ms_per_step": one_worker_ms(wr)}
            print(json.dumps(rec), flush=True)
            rows.append(rec)
    dgd = next(r for r in rows if r["scheme"] == "DGD")
    lines = ["All n = %d workers simulated on one GPU (d = %d, %d rows per partition, median of %d x %d steps), "
             "and one worker's own step on a GPU of its own." % (n, d, m, args.repeats, args.steps), "",
             "| scheme | s | c | all workers: rows read / step | GPU ms / step | vs DGD | HBM GB/s "
             "| one worker: partitions / step | rows / step | GPU ms / step | vs DGD |",
             "|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in rows:
        lines.append("| %s | %d | %d | %d | %.4f | %.2f | %.0f | %d | %d | %.4f | %.2f |" % (
            r["scheme"], r["s"], r["c"], r["rows_per_step"], r["ms_per_step"], r["ms_per_step"] / dgd["ms_per_step"],
            r["hbm_gbs"], r["partitions_per_worker"], r["worker_rows"], r["worker_ms_per_step"],
            r["worker_ms_per_step"] / dgd["worker_ms_per_step"]))
    return lines


# ----------------------------------------------------------------------------
# naive-cr: decoding coefficients and loss, n = 12, c = 6
# ----------------------------------------------------------------------------

def window_extremes(values, every, pick):
    """pick() over each window of `every` consecutive steps."""
    return [round(pick(values[i:i + every]), 3) for i in range(0, len(values), every)]


NAIVE_CR_N, NAIVE_CR_S = 12, 5
NAIVE_CR_MASK_SEED = (12 << 32) | 1


def naive_cr_workload(rows_per_partition, d, lr, steps):
    """Data of the naive-CR study: n = 12 workers, c = 6, logistic labels."""
    n, s = NAIVE_CR_N, NAIVE_CR_S
    return Workload("study_naive_cr", "CR_REAL", "logistic", n=n, c=s + 1, N=n * rows_per_partition, d=d,
                    lr=lr, steps=steps, policy=POLICY_EXACT, cap=s, seed=12, code_seed=12)


def study_naive_cr(args, out):
    import numpy as np
    import torch
    n, s = NAIVE_CR_N, NAIVE_CR_S
    dev = torch.device("cuda", 0)
    data = naive_cr_workload(args.rows_per_partition, args.d, args.lr, args.steps)
    # Drawn on the host, so the fp64 control (tests/naive_cr_oracle.py) can
    # draw the very same data without a GPU.
    X, y, beta0 = (t.to(dev) for t in make_inputs(data, device="cpu"))
    results = {}
    for name in ["PGC-FR", "PGC-CR", "naive PGC-CR"]:
        masks, _ = delay_masks(n, s, args.steps, NAIVE_CR_MASK_SEED, 1.0, 1.0, name, s)
        losses, alphas = train(name, s, data, X, y, beta0, masks, args.lr, record_alpha=True)
        amax = [a for a, _ in alphas]
        amin = [b for _, b in alphas]
        lv = [l for _, l in losses]
        finite = [l for l in lv if math.isfinite(l)]
        rec = {"study": "naive-cr", "scheme": name, "n": n, "c": s + 1, "steps": args.steps, "lr": args.lr,
               "loss_first": lv[0], "loss_last": lv[-1], "loss_max": max(finite) if finite else None,
               "alpha_max": max(amax), "alpha_min": min(amin),
               "steps_with_abs_alpha_over_10": int(sum(1 for a, b in alphas if max(a, -b) > 10.0)),
               "loss_trace": [round(l, 6) if math.isfinite(l) else None for l in lv[::max(1, args.steps // 50)]],
               "alpha_max_trace": window_extremes(amax, max(1, args.steps // 50), max),
               "alpha_min_trace": window_extremes(amin, max(1, args.steps // 50), min)}
        print(json.dumps(rec), flush=True)
        results[name] = rec
    lines = ["n = 12, c = 6, s = 5 (the 5 slowest of 12 exponential delays each step), logistic loss, "
             "d = %d, %d rows per partition, lr %.2f, %d steps." % (args.d, args.rows_per_partition, args.lr,
                                                                  args.steps), "",
             "| scheme | loss at t=0 | final loss | max loss | max alpha | min alpha | steps with max abs alpha > 10 |",
             "|---|---|---|---|---|---|---|"]
    for name, r in results.items():
        lines.append("| %s | %.4f | %s | %s | %.4g | %.4g | %d |" % (
            name, r["loss_first"], "%.4g" % r["loss_last"] if math.isfinite(r["loss_last"]) else "non-finite",
            "%.4g" % r["loss_max"] if r["loss_max"] is not None else "-", r["alpha_max"], r["alpha_min"],
            r["steps_with_abs_alpha_over_10"]))
    every = max(1, args.steps // 50)
    lines += ["", "Trace: loss at the start of each window of %d steps; extreme alpha of naive PGC-CR "
              "over the window:" % every, "",
              "| t | loss PGC-FR | loss PGC-CR | loss naive PGC-CR | max alpha | min alpha |",
              "|---|---|---|---|---|---|"]
    tr = {k: v["loss_trace"] for k, v in results.items()}
    naive = results["naive PGC-CR"]
    for i in range(len(naive["alpha_max_trace"])):
        lines.append("| %d | %s | %s | %s | %.4g | %.4g |" % tuple(
            [i * every] + ["%.4f" % tr[k][i] if tr[k][i] is not None else "non-finite"
                           for k in ["PGC-FR", "PGC-CR", "naive PGC-CR"]]
            + [naive["alpha_max_trace"][i], naive["alpha_min_trace"][i]]))
    return lines


# ----------------------------------------------------------------------------
# delays: simulated time per step and time to loss
# ----------------------------------------------------------------------------

def study_delays(args, out):
    import numpy as np
    n = args.n
    lines = ["Simulated time per step, normalised to DGD (%d draws; compute per partition %.2f s)." % (
        args.draws, args.partition_seconds), "",
             "| mean delay (s) | s | " + " | ".join(k for k in SCHEMES if k != "naive PGC-CR") + " |",
             "|---|---|" + "---|" * (len(SCHEMES) - 1)]
    for mean in args.means:
        for s in args.s:
            per = {}
            for name in SCHEMES:
                if name == "naive PGC-CR":
                    continue
                _, _, _, s_tol = scheme_setup(name, s)
                _, secs = delay_masks(n, s_tol, args.draws + 1, (21 << 32) | 1, mean, args.partition_seconds,
                                      name, s)
                per[name] = float(np.mean(secs[1:]))
            rec = {"study": "delays-per-step", "n": n, "s": s, "mean_delay_s": mean,
                   "partition_seconds": args.partition_seconds, "seconds_per_step": per,
                   "vs_dgd": {k: v / per["DGD"] for k, v in per.items()}}
            print(json.dumps(rec), flush=True)
            lines.append("| %.1f | %d | " % (mean, s) + " | ".join(
                "%.0f%%" % (100.0 * per[k] / per["DGD"]) for k in per) + " |")
    if args.no_train:
        return lines

    import torch
    dev = torch.device("cuda", 0)
    s, mean = args.train_s, args.means[0]
    data = Workload("study_delays", "FR", "logistic", n=n, c=s + 1, N=n * args.rows_per_partition, d=args.d,
                    lr=args.lr, steps=args.steps, policy=POLICY_EXACT, cap=s, seed=13, code_seed=13)
    X, y, beta0 = make_inputs(data, device=dev)
    runs = {}
    for name in SCHEMES:
        if name == "naive PGC-CR":
            continue
        _, _, _, s_tol = scheme_setup(name, s)
        masks, secs = delay_masks(n, s_tol, args.steps, (13 << 32) | 1, mean, args.partition_seconds, name, s)
        losses, _ = train(name, s, data, X, y, beta0, masks, args.lr)
        clock = np.concatenate([[0.0], np.cumsum(secs)])
        runs[name] = (np.array([l for _, l in losses]), clock)
    dgd_loss = runs["DGD"][0]
    target = dgd_loss[-1] + args.target_frac * (dgd_loss[0] - dgd_loss[-1])
    lines += ["", "Time to loss %.4f (DGD's final loss plus %.0f%% of its decrease), s = %d, mean delay %.1f s, "
              "%d steps, lr %.2f:" % (target, 100 * args.target_frac, s, mean, args.steps, args.lr), "",
              "| scheme | steps to target | simulated seconds to target | vs DGD | final loss |",
              "|---|---|---|---|---|"]
    dgd_time = None
    for name, (lv, clock) in runs.items():
        hit = np.nonzero(lv <= target)[0]
        step = int(hit[0]) if hit.size else None
        sec = float(clock[step]) if step is not None else None
        if name == "DGD":
            dgd_time = sec
        rec = {"study": "delays-time-to-loss", "scheme": name, "s": s, "mean_delay_s": mean, "target_loss": target,
               "steps_to_target": step, "seconds_to_target": sec, "final_loss": float(lv[-1])}
        print(json.dumps(rec), flush=True)
        lines.append("| %s | %s | %s | %s | %.4f |" % (
            name, step if step is not None else "not reached", "%.1f" % sec if sec is not None else "-",
            "%.2f" % (sec / dgd_time) if sec is not None and dgd_time else "-", lv[-1]))
    return lines


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("study", choices=["baselines", "naive-cr", "delays"])
    ap.add_argument("--n", type=int, default=12)
    ap.add_argument("--d", type=int, default=None)
    ap.add_argument("--rows-per-partition", type=int, default=None)
    ap.add_argument("--s", type=int, nargs="+", default=[1, 2, 3])
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--repeats", type=int, default=3, help="baselines: timed repeats per case (median kept)")
    ap.add_argument("--lr", type=float, default=None)
    ap.add_argument("--means", type=float, nargs="+", default=[1.0, 2.0], help="mean delays in seconds")
    ap.add_argument("--partition-seconds", type=float, default=1.0,
                    help="simulated compute time of one partition gradient on one worker")
    ap.add_argument("--draws", type=int, default=2000, help="simulated steps per per-step-time estimate")
    ap.add_argument("--train-s", type=int, default=2)
    ap.add_argument("--target-frac", type=float, default=0.05)
    ap.add_argument("--no-train", action="store_true", help="delays: only the simulated per-step times")
    ap.add_argument("--out", default=None, help="write a markdown summary here")
    args = ap.parse_args()
    defaults = {"baselines": dict(d=1024, rows_per_partition=65536, steps=100, lr=0.01),
                "naive-cr": dict(d=256, rows_per_partition=4096, steps=300, lr=0.5),
                "delays": dict(d=256, rows_per_partition=4096, steps=300, lr=0.5)}[args.study]
    for k, v in defaults.items():
        if getattr(args, k) is None:
            setattr(args, k, v)
    needs_gpu = args.study != "delays" or not args.no_train
    if needs_gpu:
        import torch
        if not torch.cuda.is_available():
            print("no GPU visible", file=sys.stderr)
            return 1
    fn = {"baselines": study_baselines, "naive-cr": study_naive_cr, "delays": study_delays}[args.study]
    lines = fn(args, args.out)
    argv, skip = [], False
    for a in sys.argv[1:]:
        if skip:
            skip = False
        elif a == "--out":
            skip = True
        elif not a.startswith("--out="):
            argv.append(a)
    cmd = "python studies.py " + " ".join(argv)
    text = "\n".join(["# Study: %s" % args.study, "", "Command: `%s`" % cmd, ""] + lines) + "\n"
    if args.out:
        os.makedirs(os.path.dirname(os.path.abspath(args.out)), exist_ok=True)
        with open(args.out, "w") as f:
            f.write(text)
    log(text)
    return 0


if __name__ == "__main__":
    sys.exit(main())
