"""GPU checks of the library's auxiliary entry points: per-kernel timing and its
sampling period, and argument errors that need a bound workspace."""

import numpy as np
import pytest
import torch

import paper_2607_20739_amd as P
from workloads import WORKLOADS, Workload, make_inputs, POLICY_EXACT

from _parity import gpu_masks, gpu_session

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    P.lib()


def test_kernel_timing_counts_every_period_th_launch():
    w = WORKLOADS["fr_logistic_n4_c2_d64"]
    print("\n[gpu case] timing period", flush=True)
    X, y, beta0 = make_inputs(w, device="cuda")
    masks = gpu_masks(w, 10)
    sess = gpu_session(w)
    try:
        wv = beta0.clone()
        P.pgc_set_timing(sess.ctx, [P.PGC_KERNEL_GRADIENT, P.PGC_KERNEL_CODE])
        P.pgc_set_timing_period(sess.ctx, 3)
        for t in range(10):
            sess.step(X, y, wv, masks[t], w.lr)
        for kernel in (P.PGC_KERNEL_GRADIENT, P.PGC_KERNEL_CODE):
            ms, launches = P.pgc_kernel_time(sess.ctx, kernel)
            assert launches == 4                    # launches 1, 4, 7 and 10
            assert ms > 0.0
        ms, launches = P.pgc_kernel_time(sess.ctx, P.PGC_KERNEL_MLP_FORWARD)
        assert (ms, launches) == (0.0, 0)           # not launched by a linear model
        # Setting the kernels again clears the totals and restarts the sampling.
        P.pgc_set_timing(sess.ctx, True)
        for t in range(2):
            sess.step(X, y, wv, masks[t], w.lr)
        assert P.pgc_kernel_time(sess.ctx, P.PGC_KERNEL_GRADIENT)[1] == 1
        with pytest.raises(P.PGCError) as e:
            P.pgc_set_timing_period(sess.ctx, 0)
        assert e.value.status == P.PGC_EINVAL
    finally:
        sess.close()


def test_step_and_readout_argument_errors():
    w = Workload("api_mlp", "CR", "mlp", n=4, c=2, N=4 * 64, d=64, lr=0.05, steps=2,
                 policy=POLICY_EXACT, cap=1, seed=3, hidden=256, classes=10)
    print("\n[gpu case] argument errors", flush=True)
    X, y, beta0 = make_inputs(w, device="cuda")
    sess = gpu_session(w)
    try:
        wv = beta0.clone()
        mask = np.zeros(w.n, np.uint8)
        # X of the MLP must be 16-byte aligned: an offset of one bf16 element is not.
        buf = torch.empty(X.numel() + 8, dtype=torch.bfloat16, device="cuda")
        Xu = buf[1:1 + X.numel()].view_as(X)
        Xu.copy_(X)
        with pytest.raises(P.PGCError) as e:
            P.pgc_step(sess.ctx, Xu.data_ptr(), y, wv, mask, w.lr, w.n)
        assert e.value.status == P.PGC_EINVAL
        assert sess.t == 0
        sess.step(X, y, wv, mask, w.lr)
        out = torch.empty(sess.q, dtype=torch.float32, device="cuda")
        for call, args in [(P.pgc_read_ring, (w.n, 0, out)), (P.pgc_read_ring, (0, w.c, out)),
                           (P.pgc_read_coded, (sess.n_coded, out))]:
            with pytest.raises(P.PGCError) as e:
                call(sess.ctx, *args)
            assert e.value.status == P.PGC_EINVAL
        assert sess.t == 1
    finally:
        sess.close()
