"""pgc_step_noalloc (the step with its scratch in the library's fixed device
array, for callers that cannot allocate) against pgc_step, through the C ABI.

Calls in a row on one GPU, each with a smaller problem than the one before:
the fixed array keeps the earlier call's contents, and a later call must not
depend on them.  The two entry points run the same kernels on the same grid, so the
decoded gradients and weights must agree bit for bit (well within the fp32
bar of 1e-5).
"""

import numpy as np
import pytest
import torch

import paper_2607_20739_amd as P
from workloads import Workload, make_inputs, POLICY_BERNOULLI, POLICY_EXACT, POLICY_UNIFORM_COUNT

from _parity import FP32_TOL, gpu_masks, gpu_session, normwise_error

pytestmark = pytest.mark.gpu

# The first problem's partial sums fill the fixed array exactly (1024 blocks
# of 8192 floats = 32 MiB); the second is far smaller.
LARGE = Workload("noalloc_cr_logistic_d8192", "CR", "logistic", n=16, c=4, N=16 * 2048, d=8192,
                 lr=0.05, steps=7, policy=POLICY_BERNOULLI, cap=3, p=0.2, seed=71)
SMALL = Workload("noalloc_real_lsq_d1000", "CR_REAL", "lsq", n=6, c=3, N=6 * 300, d=1000,
                 lr=0.02, steps=6, policy=POLICY_UNIFORM_COUNT, cap=2, seed=72, code_seed=4)
# FR: every pipelined step evaluates one partition per group (a strided subset).
TINY_FR = Workload("noalloc_fr_logistic_d64", "FR", "logistic", n=4, c=2, N=4 * 512, d=64,
                   lr=0.1, steps=6, policy=POLICY_EXACT, cap=1, seed=73)


def _announce(what):
    print("\n[gpu case] " + what, flush=True)


def _run(w, noalloc):
    X, y, beta0 = make_inputs(w, device="cuda")
    sess = gpu_session(w)
    try:
        wv = beta0.clone()
        out = []
        for mask in gpu_masks(w):
            if noalloc:
                P.pgc_step_noalloc(sess.ctx, X, y, wv, mask, w.lr, w.n)
            else:
                P.pgc_step(sess.ctx, X, y, wv, mask, w.lr, w.n)
            out.append((sess.decoded().cpu().numpy(), wv.cpu().numpy()))
        torch.cuda.synchronize()
        return out
    finally:
        sess.close()


def test_noalloc_step_matches_pgc_step_on_two_calls_in_a_row():
    problems = (LARGE, SMALL, TINY_FR)
    sizes = []
    for w in problems:
        sess = gpu_session(w)
        try:
            sizes.append(P.pgc_workspace_bytes(sess.ctx))
        finally:
            sess.close()
    assert sizes == sorted(sizes, reverse=True) and len(set(sizes)) == len(sizes), sizes   # each call smaller
    for w in problems:
        _announce("%s n=%d c=%d d=%d N=%d" % (w.name, w.n, w.c, w.d, w.N))
        ref = _run(w, noalloc=False)
        got = _run(w, noalloc=True)
        assert len(ref) == len(got) == w.steps
        for t, ((g_ref, w_ref), (g, wv)) in enumerate(zip(ref, got)):
            assert normwise_error(g, g_ref) <= FP32_TOL, "step %d ghat" % t
            assert normwise_error(wv, w_ref) <= FP32_TOL, "step %d w" % t
            assert np.array_equal(g, g_ref) and np.array_equal(wv, w_ref), "step %d not bitwise" % t


def test_noalloc_step_rejects_what_does_not_fit():
    _announce("noalloc rejections")
    # d = 32768 on 1024 blocks: 128 MiB of partial sums, beyond the fixed array.
    big = Workload("noalloc_too_big", "CR", "lsq", n=4, c=2, N=4 * 2048, d=32768, lr=0.01, steps=1,
                   policy=POLICY_UNIFORM_COUNT, cap=1, seed=73)
    mlp = Workload("noalloc_mlp", "CR", "mlp", n=4, c=2, N=4 * 64, d=64, lr=0.05, steps=1,
                   policy=POLICY_UNIFORM_COUNT, cap=1, seed=74, hidden=256, classes=10)
    for w in (big, mlp):
        X, y, beta0 = make_inputs(w, device="cuda")
        sess = gpu_session(w)
        try:
            wv = beta0.clone()
            with pytest.raises(P.PGCError) as e:
                P.pgc_step_noalloc(sess.ctx, X, y, wv, np.zeros(w.n, np.uint8), w.lr, w.n)
            assert e.value.status == P.PGC_EINVAL
            assert sess.t == 0
            torch.cuda.synchronize()
            assert torch.equal(wv, beta0)
        finally:
            sess.close()
