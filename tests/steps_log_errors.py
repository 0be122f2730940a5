#!/usr/bin/env python3
"""Per-step errors of a bench.py run against the fp64 oracle (test infrastructure).

  python tests/steps_log_errors.py LOG [--teacher-forced] [--device cuda|cpu]

LOG is the JSON-lines file `bench.py --steps-log LOG` wrote and LOG.npz the
decoded gradient and weights of every step beside it.  The inputs are drawn
again from the workload's seed on `device` (the bench draws them on the GPU),
the oracle runs the logged straggler masks, and LOG is rewritten with, per step:
  err_ghat, err_w   normwise errors max_i |gpu_i - oracle_i| / max_i |oracle_i|
                    of the two independent trajectories;
  tf_err_ghat       (--teacher-forced) the step's decoded gradient against the
                    oracle's decoded gradient at the GPU's own iterates, which
                    separates one step's error from the drift between the two
                    trajectories.
Prints the worst of each.
"""

import argparse
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from oracle import pgc_oracle as O  # noqa: E402
from oracle import rng as R  # noqa: E402

SCHEMES = {"FR": O.FR, "CR": O.CR, "CR_REAL": O.CR_REAL, "IS_SGD": O.IS_SGD}


def normwise(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    scale = np.max(np.abs(b))
    diff = np.max(np.abs(a - b))
    return float(diff / scale) if scale > 0 else float(diff)


def annotate(log_path, w, X, y, beta0, teacher_forced=False):
    """Add the error columns to log_path; returns the rewritten records."""
    with open(log_path) as f:
        recs = [json.loads(line) for line in f if line.strip()]
    vec = np.load(log_path + ".npz")
    ghat_gpu, w_gpu = vec["ghat"], vec["w"]
    if len(recs) != len(ghat_gpu):
        raise ValueError("log has %d steps, vectors %d" % (len(recs), len(ghat_gpu)))
    masks = []
    for r in recs:
        m = np.zeros(w.n, np.uint8)
        m[r["stragglers"]] = 1
        masks.append(m)
    B = None
    if w.scheme == "CR_REAL":
        B = O.cyclic_encoding_matrix(w.n, w.c, R.null_space_generator(w.code_seed, w.c - 1, w.n))
    shape = (w.d, w.hidden, w.classes) if w.model == "mlp" else None
    Xh = np.asarray(X, dtype=np.float64)
    yh = np.asarray(y, dtype=np.float64)
    ref = O.run(SCHEMES[w.scheme], w.model, w.n, w.c, Xh, yh, beta0, w.lr, masks, B=B, shape=shape,
                keep_coded=False, keep_alpha=False)
    iterates = {0: np.asarray(beta0, np.float64)}
    memo = {}
    for t, (r, o) in enumerate(zip(recs, ref)):
        r["err_ghat"] = normwise(ghat_gpu[t], o.ghat)
        r["err_w"] = normwise(w_gpu[t], o.beta)
        if teacher_forced:
            tf = O.teacher_forced_ghat(SCHEMES[w.scheme], w.model, w.n, w.c, Xh, yh, iterates, t, masks[t],
                                       B=B, shape=shape, memo=memo)
            r["tf_err_ghat"] = normwise(ghat_gpu[t], tf)
            iterates[t + 1] = w_gpu[t].astype(np.float64)
            for key in [k for k in memo if k[1] < t + 2 - w.c]:
                del memo[key]
    with open(log_path, "w") as f:
        for r in recs:
            f.write(json.dumps(r) + "\n")
    return recs


def main():
    import torch
    from dataclasses import replace
    from workloads import WORKLOADS, make_inputs
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("log")
    ap.add_argument("--teacher-forced", action="store_true")
    ap.add_argument("--device", default="cuda")
    args = ap.parse_args()
    meta = np.load(args.log + ".npz")
    w = replace(WORKLOADS[str(meta["workload"])], lr=float(meta["lr"]), seed=int(meta["seed"]))
    X, y, beta0 = make_inputs(w, device=args.device)
    Xh = X.float().cpu().numpy()
    recs = annotate(args.log, w, Xh, y.cpu().numpy(), beta0.cpu().numpy(), args.teacher_forced)
    del X
    out = {"workload": w.name, "lr": w.lr, "steps": len(recs),
           "worst_err_ghat": max(r["err_ghat"] for r in recs), "worst_err_w": max(r["err_w"] for r in recs)}
    if args.teacher_forced:
        out["worst_tf_err_ghat"] = max(r["tf_err_ghat"] for r in recs)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
