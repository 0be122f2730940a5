#!/usr/bin/env python3
"""fp64 control of the naive PGC-CR study (test infrastructure).

The study (`studies.py naive-cr`) trains PGC-FR, PGC-CR and the naive
pipelined cyclic code with real coefficients (Sec. V-A) on the GPU at n = 12,
c = 6, dropping the 5 slowest of 12 exponential delays each step, and finds
that only the naive code's loss leaves the basin.  Its decoding weights reach
|alpha| ~ 1e5, which also multiplies the fp32 rounding of the ring.  This
module runs the same three schemes in the fp64 oracle on the same data and
straggler sets, so the divergence can be attributed: if the oracle diverges
too, it comes from stale copies weighted by large coefficients (the effect
Sec. V-A and Fig. 6 describe), not from fp32 arithmetic.

  python tests/naive_cr_oracle.py [--steps T] [--rows-per-partition M] [--d D]
                                  [--lr LR] [--gpu-json PATH] [--out PATH]

--gpu-json takes the JSON lines `studies.py naive-cr` printed, to put the GPU's
loss beside the oracle's in the table written to --out.
"""

import argparse
import json
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from oracle import pgc_oracle as O  # noqa: E402
from oracle import rng as R  # noqa: E402

N_WORKERS, S = 12, 5
MASK_SEED = (12 << 32) | 1
SCHEMES = {"PGC-FR": O.FR, "PGC-CR": O.CR, "naive PGC-CR": O.CR_REAL}


def study_inputs(rows_per_partition, d, lr, steps):
    """The study's data, drawn on the host exactly as studies.py draws it."""
    from studies import naive_cr_workload
    from workloads import make_inputs
    w = naive_cr_workload(rows_per_partition, d, lr, steps)
    X, y, beta0 = make_inputs(w, device="cpu")
    return w, X.numpy().astype(np.float64), y.numpy().astype(np.float64), beta0.numpy().astype(np.float64)


def study_masks(steps):
    """The 5 slowest of 12 exponential delays (mean 1 s) at every step."""
    return [R.delay_step(MASK_SEED, t, N_WORKERS, S, 1.0)[0] for t in range(steps)]


def run_scheme(name, w, X, y, beta0, masks):
    """Loss before every step and after the last, and the extreme reported
    decoding weights n * scale * d_m * B[j_m, k] over held pairs per step."""
    scheme = SCHEMES[name]
    n, c = w.n, w.c
    B = None
    if scheme == O.CR_REAL:
        B = O.cyclic_encoding_matrix(n, c, R.null_space_generator(w.code_seed, c - 1, n))
    recs = O.run(scheme, "logistic", n, c, X, y, beta0, w.lr, masks, B=B, keep_coded=False, keep_alpha=True)
    place = O.placement(scheme, n, c)
    losses = [O.full_loss("logistic", X, y, beta0)]
    amax, amin = [], []
    for r in recs:
        losses.append(O.full_loss("logistic", X, y, r.beta) if np.all(np.isfinite(r.beta)) else math.inf)
        held = [n * r.scale * r.alpha[m, k] for m, j in enumerate(r.survivors) for k in place[j]]
        amax.append(max(held))
        amin.append(min(held))
    return losses, amax, amin


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--steps", type=int, default=300)
    ap.add_argument("--rows-per-partition", type=int, default=4096)
    ap.add_argument("--d", type=int, default=256)
    ap.add_argument("--lr", type=float, default=0.5)
    ap.add_argument("--gpu-json", default=None)
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    w, X, y, beta0 = study_inputs(args.rows_per_partition, args.d, args.lr, args.steps)
    masks = study_masks(args.steps)
    gpu = {}
    if args.gpu_json:
        with open(args.gpu_json) as f:
            for line in f:
                if line.strip().startswith("{"):
                    rec = json.loads(line)
                    if rec.get("study") == "naive-cr":
                        gpu[rec["scheme"]] = rec
    res = {}
    for name in SCHEMES:
        losses, amax, amin = run_scheme(name, w, X, y, beta0, masks)
        finite = [v for v in losses if math.isfinite(v)]
        res[name] = {"losses": losses, "alpha_max": max(amax), "alpha_min": min(amin)}
        print(json.dumps({"scheme": name, "loss_first": losses[0], "loss_last": losses[-1],
                          "loss_max": max(finite), "alpha_max": max(amax), "alpha_min": min(amin)}), flush=True)
    every = max(1, args.steps // 50)
    argv, skip = [], False
    for a in sys.argv[1:]:
        if skip:
            skip = False
        elif a == "--out":
            skip = True
        elif not a.startswith("--out="):
            argv.append(a)
    cmd = "python tests/naive_cr_oracle.py " + " ".join(argv)
    lines = ["# fp64 control of the naive PGC-CR study", "",
             "Command: `%s` (writes this file with `--out`)." % cmd.strip(), "",
             "The oracle (plain numpy, fp64) runs PGC-FR, PGC-CR and naive PGC-CR (real coefficients, "
             "Sec. V-A) on the data and straggler sets of `studies.py naive-cr`: n = 12, c = 6, the 5 slowest "
             "of 12 exponential delays dropped each step, logistic loss, d = %d, %d rows per partition, lr %.2f, "
             "%d steps." % (args.d, args.rows_per_partition, args.lr, args.steps), "",
             "| scheme | oracle final loss | oracle max loss | oracle max alpha | oracle min alpha |"
             + (" GPU final loss | GPU max loss |" if gpu else ""),
             "|---|---|---|---|---|" + ("---|---|" if gpu else "")]
    for name, r in res.items():
        fin = [v for v in r["losses"] if math.isfinite(v)]
        row = "| %s | %.4g | %.4g | %.4g | %.4g |" % (name, r["losses"][-1], max(fin), r["alpha_max"], r["alpha_min"])
        if gpu:
            g = gpu.get(name, {})
            row += " %s | %s |" % ("%.4g" % g["loss_last"] if g.get("loss_last") is not None else "-",
                                   "%.4g" % g["loss_max"] if g.get("loss_max") is not None else "-")
        lines.append(row)
    lines += ["", "Loss at the start of each window of %d steps (oracle%s):" % (every, " / GPU" if gpu else ""), "",
              "| t | PGC-FR | PGC-CR | naive PGC-CR |", "|---|---|---|---|"]
    for i, t in enumerate(range(0, args.steps, every)):
        cells = []
        for name in SCHEMES:
            o = res[name]["losses"][t]
            cell = "%.4f" % o if math.isfinite(o) else "non-finite"
            if gpu and name in gpu and i < len(gpu[name]["loss_trace"]):
                g = gpu[name]["loss_trace"][i]
                cell += " / " + ("%.4f" % g if g is not None else "non-finite")
            cells.append(cell)
        lines.append("| %d | %s |" % (t, " | ".join(cells)))
    text = "\n".join(lines) + "\n"
    if args.out:
        with open(args.out, "w") as f:
            f.write(text)
    print(text)
    return 0


if __name__ == "__main__":
    sys.exit(main())
