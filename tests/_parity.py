"""Shared helpers of the GPU parity tests: run the HIP path and the oracle on the
same seeded inputs and compare them step by step."""

import numpy as np

from oracle import pgc_oracle as O
from oracle import rng as R

SCHEMES = {"FR": O.FR, "CR": O.CR, "CR_REAL": O.CR_REAL, "IS_SGD": O.IS_SGD}

# Floating-point bar of the fp32 path (normwise, per step, per vector):
#   max_i |gpu_i - oracle_i| / max_i |oracle_i| <= 1e-5.
FP32_TOL = 1e-5


def normwise_error(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    scale = np.max(np.abs(b))
    return float(np.max(np.abs(a - b)) / scale) if scale > 0 else float(np.max(np.abs(a - b)))


def elementwise_error(a, b, floor=1e-3):
    """max_i |a_i - b_i| / max(|b_i|, floor * max_j |b_j|): the elementwise
    relative error, with an absolute floor so that entries near zero do not
    make it meaningless.  Reported beside the normwise bar, not gated."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    scale = np.maximum(np.abs(b), floor * np.max(np.abs(b)))
    scale = np.where(scale > 0, scale, 1.0)
    return float(np.max(np.abs(a - b) / scale))


def oracle_masks(w, steps=None):
    steps = w.steps if steps is None else steps
    return [R.straggler_mask(w.mask_seed, t, w.policy, w.n, w.cap, w.p) for t in range(steps)]


def oracle_code_matrix(w):
    if w.scheme != "CR_REAL":
        return None
    return O.cyclic_encoding_matrix(w.n, w.c, R.null_space_generator(w.code_seed, w.c - 1, w.n))


def oracle_run(w, X, y, beta0, masks, lr=None, keep_coded=False, pipelined=True, progress_every=0):
    """The oracle's trajectory; with progress_every > 0 it prints a line every
    that many steps (long full-size runs)."""
    shape = (w.d, w.hidden, w.classes) if w.model == "mlp" else None

    def report(t, rec):
        if progress_every and (t + 1) % progress_every == 0:
            print("  oracle: %d of %d steps done" % (t + 1, len(masks)), flush=True)
    return O.run(SCHEMES[w.scheme], w.model, w.n, w.c, X, y, beta0, w.lr if lr is None else lr,
                 masks, B=oracle_code_matrix(w), shape=shape, keep_coded=keep_coded,
                 keep_alpha=False, pipelined=pipelined, on_step=report)


def gpu_session(w, device="cuda", pipelined=True):
    import paper_2607_20739_amd as P
    return P.PGCSession(w.scheme, w.n, w.c, w.model, w.N, w.d, hidden=w.hidden, classes=w.classes,
                        code_seed=w.code_seed, device=device, pipelined=pipelined)


def gpu_masks(w, steps=None):
    import paper_2607_20739_amd as P
    steps = w.steps if steps is None else steps
    return [P.pgc_make_mask(w.mask_seed, t, w.policy, w.n, w.cap, w.p) for t in range(steps)]


def gpu_run(w, X, y, beta0, masks, lr=None, keep=("ghat", "w"), read_coded=False, pipelined=True):
    """Run the HIP path; returns one dict per step with host copies of the kept vectors."""
    import torch
    sess = gpu_session(w, X.device, pipelined=pipelined)
    wv = beta0.clone()
    out = []
    try:
        for mask in masks:
            sess.step(X, y, wv, mask, w.lr if lr is None else lr)
            rec = {}
            if "ghat" in keep:
                rec["ghat"] = sess.decoded().cpu().numpy()
            if "w" in keep:
                rec["w"] = wv.cpu().numpy()
            if read_coded:
                rec["coded"] = np.stack([sess.coded(j).cpu().numpy() for j in range(sess.n_coded)])
            out.append(rec)
        torch.cuda.synchronize()
    finally:
        sess.close()
    return out, wv
