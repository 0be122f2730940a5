"""GPU parity of the two-layer MLP path (bf16 MFMA) against the fp64 oracle.

The oracle evaluates the network with the same bf16 inputs and bf16-rounded
W1, W2 (reading R3); the GPU additionally rounds H, dZ2 and dZ1 to bf16 for
its MFMAs, which the 2e-2 normwise bar covers.
"""

import numpy as np
import pytest
import torch

import paper_2607_20739_amd as P
from oracle import pgc_oracle as O
from workloads import WORKLOADS, Workload, make_inputs, POLICY_BERNOULLI, POLICY_EXACT, \
    POLICY_UNIFORM_COUNT

from _parity import elementwise_error, gpu_masks, gpu_run, gpu_session, normwise_error, oracle_masks, \
    oracle_run

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


def _announce(what):
    print("\n[gpu case] " + what, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    P.lib()


def _host_inputs(X, y, beta0):
    return X.float().cpu().numpy(), y.cpu().numpy(), beta0.cpu().numpy()


def _check_trajectory(w):
    X, y, beta0 = make_inputs(w, device="cuda")
    masks_gpu = gpu_masks(w)
    masks_or = oracle_masks(w)
    assert [m.tolist() for m in masks_gpu] == [m.tolist() for m in masks_or]
    recs_gpu, _ = gpu_run(w, X, y, beta0, masks_gpu)
    recs_or = oracle_run(w, *_host_inputs(X, y, beta0), masks_or)
    worst = worst_elem = 0.0
    for t, (g, o) in enumerate(zip(recs_gpu, recs_or)):
        assert np.all(np.isfinite(g["ghat"])) and np.all(np.isfinite(g["w"]))
        e_g = normwise_error(g["ghat"], o.ghat)
        e_w = normwise_error(g["w"], o.beta)
        worst = max(worst, e_g, e_w)
        worst_elem = max(worst_elem, elementwise_error(g["ghat"], o.ghat), elementwise_error(g["w"], o.beta))
        assert e_g <= BF16_TOL, "step %d: decoded gradient error %.3g" % (t, e_g)
        assert e_w <= BF16_TOL, "step %d: weight error %.3g" % (t, e_w)
    print("  worst normwise error over %d steps: %.3g (elementwise, floor 1e-3 of the max: %.3g)"
          % (len(recs_gpu), worst, worst_elem), flush=True)


SMALL = [
    # ragged partitions (m = 100, padded to 128 rows) and two classes short of 16
    Workload("mlp_cr_small_ragged", "CR", "mlp", n=4, c=2, N=4 * 100, d=64, lr=0.05, steps=6,
             policy=POLICY_EXACT, cap=1, seed=31, hidden=256, classes=10),
    # d_in not a multiple of the K step (40 = 32 + 8), three classes, FR
    Workload("mlp_fr_small", "FR", "mlp", n=4, c=2, N=4 * 64, d=40, lr=0.05, steps=6,
             policy=POLICY_EXACT, cap=1, seed=32, hidden=256, classes=3),
    # hidden = 512 (two forward column blocks, four head waves), c = n
    Workload("mlp_cr_c_eq_n", "CR", "mlp", n=3, c=3, N=3 * 160, d=120, lr=0.02, steps=7,
             policy=POLICY_UNIFORM_COUNT, cap=2, seed=33, hidden=512, classes=16),
    # several tiles of every kernel: d_in = 456 spans three 224-wide feature tiles of the
    # weight gradient (the last ragged), hidden = 768 three forward column tiles, m = 600
    # two 384-row forward tiles (the last ragged, with a partial second epilogue pass)
    Workload("mlp_cr_multi_tile", "CR", "mlp", n=4, c=2, N=4 * 600, d=456, lr=0.02, steps=5,
             policy=POLICY_EXACT, cap=1, seed=35, hidden=768, classes=7),
    # five rows per partition: one ragged 16-row head tile, one 64-row weight-gradient K step,
    # and a forward tile that is almost all clamped rows
    Workload("mlp_cr_tiny_partitions", "CR", "mlp", n=4, c=2, N=4 * 5, d=16, lr=0.05, steps=5,
             policy=POLICY_EXACT, cap=1, seed=36, hidden=256, classes=4),
    # m = 385: a second 384-row forward tile holding one row; d_in = 72 pads to two 64-column
    # K steps whose last one skips its upper half (columns 96 .. 127 lie past d_in), and ends
    # in a half-filled 16-feature block of the weight gradient
    Workload("mlp_cr_forward_tile_edge", "CR", "mlp", n=4, c=2, N=4 * 385, d=72, lr=0.05, steps=5,
             policy=POLICY_EXACT, cap=1, seed=38, hidden=256, classes=5),
    # the real-valued code on the MLP
    Workload("mlp_real_code", "CR_REAL", "mlp", n=4, c=2, N=4 * 64, d=64, lr=0.02, steps=5,
             policy=POLICY_EXACT, cap=1, seed=34, hidden=256, classes=10, code_seed=3),
    # the smallest d_in (one 16-byte chunk per row: the forward's one K step is 56 columns of
    # padding, the weight gradient's one feature tile 8 features wide) with the most classes
    Workload("mlp_cr_min_din_max_classes", "CR", "mlp", n=4, c=2, N=4 * 64, d=8, lr=0.05, steps=5,
             policy=POLICY_EXACT, cap=1, seed=37, hidden=256, classes=16),
]

# One class: the softmax is exactly 1, so dZ2, every gradient and every update are exactly zero.
ONE_CLASS = Workload("mlp_cr_one_class", "CR", "mlp", n=4, c=2, N=4 * 64, d=64, lr=0.05, steps=4,
                     policy=POLICY_EXACT, cap=1, seed=37, hidden=256, classes=1)


@pytest.mark.parametrize("w", SMALL, ids=[w.name for w in SMALL])
def test_small_mlp_trajectory_matches_oracle(w):
    _announce("%s N=%d d_in=%d hidden=%d" % (w.name, w.N, w.d, w.hidden))
    _check_trajectory(w)


def test_one_class_mlp_has_exactly_zero_gradients():
    w = ONE_CLASS
    _announce("%s N=%d d_in=%d hidden=%d classes=1" % (w.name, w.N, w.d, w.hidden))
    X, y, beta0 = make_inputs(w, device="cuda")
    masks = gpu_masks(w)
    recs, w_final = gpu_run(w, X, y, beta0, masks)
    for t, g in enumerate(recs):
        assert np.all(g["ghat"] == 0.0), "step %d: nonzero decoded gradient" % t
    assert torch.equal(w_final.cpu(), beta0.cpu())
    ref = oracle_run(w, *_host_inputs(X, y, beta0), oracle_masks(w))
    assert all(np.all(o.ghat == 0.0) for o in ref)


def test_mlp_workload_shape_trajectory_matches_oracle():
    """The 784 -> 1024 -> 10 network, n = 64, c = 4, with 256 rows per partition."""
    w = WORKLOADS["cr_mlp_n64_c4_784x1024x10"].resized(N=64 * 256)
    _announce("%s N=%d" % (w.name, w.N))
    _check_trajectory(w)


def test_mlp_runs_are_bitwise_reproducible():
    w = SMALL[0]
    _announce("mlp reproducibility")
    X, y, beta0 = make_inputs(w, device="cuda")
    masks = gpu_masks(w)
    _, w1 = gpu_run(w, X, y, beta0, masks, keep=())
    _, w2 = gpu_run(w, X, y, beta0, masks, keep=())
    assert torch.equal(w1, w2)


def test_mlp_resume_from_saved_state_is_bitwise_identical():
    w = SMALL[0]
    _announce("mlp resume")
    X, y, beta0 = make_inputs(w, device="cuda")
    masks = gpu_masks(w)
    k = 3
    a, b = gpu_session(w), gpu_session(w)
    try:
        wa = beta0.clone()
        for t in range(k):
            a.step(X, y, wa, masks[t], w.lr)
        state = a.save_state()
        wb = wa.clone()
        for t in range(k, w.steps):
            a.step(X, y, wa, masks[t], w.lr)
        b.load_state(state)
        for t in range(k, w.steps):
            b.step(X, y, wb, masks[t], w.lr)
        assert torch.equal(wa, wb)
    finally:
        a.close()
        b.close()


@pytest.fixture(scope="module")
def full_mlp():
    """Inputs of the full 784 -> 1024 -> 10 workload (N = 1048576), drawn once."""
    w = WORKLOADS["cr_mlp_n64_c4_784x1024x10"]
    _announce("%s full size: generating inputs" % w.name)
    X, y, beta0 = make_inputs(w, device="cuda")
    yield w, X, y, beta0
    del X, y, beta0
    torch.cuda.empty_cache()


def test_full_size_mlp_ring_holds_partition_gradients(full_mlp):
    """Full size (N = 1048576), lr = 0: sampled partitions' ring copies equal the
    oracle's gradient at beta0, computed one partition at a time."""
    w, X, y, beta0 = full_mlp
    _announce("%s full size, lr = 0" % w.name)
    sess = gpu_session(w)
    try:
        wv = beta0.clone()
        for mask in gpu_masks(w, w.c + 1):
            sess.step(X, y, wv, mask, 0.0)
        place = sess.placement()
        beta_h = beta0.cpu().numpy().astype(np.float64)
        shape = (w.d, w.hidden, w.classes)
        for k in (0, w.n // 2, w.n - 1):
            rows = slice(k * w.m, (k + 1) * w.m)
            g = O.partition_gradient(O.MLP, X[rows].float().cpu().numpy().astype(np.float64),
                                     y[rows].cpu().numpy(), beta_h, shape)
            for i, l in [(i, l) for i in range(w.n) for l in range(w.c) if place[i][l] == k]:
                err = normwise_error(sess.ring(i, l).cpu().numpy(), g)
                assert err <= BF16_TOL, "partition %d, worker %d slot %d: %.3g" % (k, i, l, err)
        assert torch.equal(wv, beta0)
    finally:
        sess.close()


def test_full_size_mlp_fresh_slots_match_the_oracle_at_every_iterate(full_mlp):
    """Full size at the workload's learning rate: each step's freshly written
    ring copies of sampled partitions equal the oracle's gradient of that
    partition (all 16,384 rows) at the iterate the step started from (the
    oracle fed the GPU's iterate), within the bf16 bar, for c + 2 steps."""
    w, X, y, beta0 = full_mlp
    _announce("%s full size, teacher-forced slots over %d steps" % (w.name, w.c + 2))
    shape = (w.d, w.hidden, w.classes)
    sampled = (0, w.n // 2, w.n - 1)
    host = {k: (X[k * w.m:(k + 1) * w.m].float().cpu().numpy().astype(np.float64),
                y[k * w.m:(k + 1) * w.m].cpu().numpy()) for k in sampled}
    sess = gpu_session(w)
    try:
        place = sess.placement()
        wv = beta0.clone()
        worst, checked = 0.0, 0
        for t, mask in enumerate(gpu_masks(w, w.c + 2)):
            w_before = wv.cpu().numpy().astype(np.float64)
            sess.step(X, y, wv, mask, w.lr)
            o = (t - 1) % w.c
            for k in sampled:
                holders = ([(i, l) for i in range(w.n) for l in range(w.c) if place[i][l] == k] if t == 0
                           else [(i, o) for i in range(w.n) if place[i][o] == k])
                g = O.partition_gradient(O.MLP, host[k][0], host[k][1], w_before, shape)
                for i, l in holders:
                    err = normwise_error(sess.ring(i, l).cpu().numpy(), g)
                    worst = max(worst, err)
                    checked += 1
                    assert err <= BF16_TOL, "step %d, partition %d, worker %d slot %d: %.3g" % (t, k, i, l, err)
        print("  %d slots checked, worst normwise error %.3g" % (checked, worst), flush=True)
    finally:
        sess.close()


def test_full_size_mlp_trajectory_matches_oracle(full_mlp):
    """All 1,048,576 rows and all 64 partitions: the decoded gradient and the
    weights after each of the workload's first 12 steps (the warm-up and three
    pipeline cycles of c = 4) against the oracle's independent fp64 trajectory,
    within the bf16 bar.  The whole 20-step trajectory runs against the oracle
    at 256 rows per partition above; 12 keeps this test near a minute."""
    w, X, y, beta0 = full_mlp
    w = w.resized(steps=12)
    _announce("%s full size, %d steps against the oracle's trajectory" % (w.name, w.steps))
    masks_gpu, masks_or = gpu_masks(w), oracle_masks(w)
    assert [m.tolist() for m in masks_gpu] == [m.tolist() for m in masks_or]
    recs_gpu, _ = gpu_run(w, X, y, beta0, masks_gpu)
    recs_or = oracle_run(w, *_host_inputs(X, y, beta0), masks_or, progress_every=2)
    worst = 0.0
    for t, (g, o) in enumerate(zip(recs_gpu, recs_or)):
        e_g, e_w = normwise_error(g["ghat"], o.ghat), normwise_error(g["w"], o.beta)
        worst = max(worst, e_g, e_w)
        assert e_g <= BF16_TOL and e_w <= BF16_TOL, "step %d: %.3g %.3g" % (t, e_g, e_w)
    print("  worst normwise error over %d steps: %.3g" % (w.steps, worst), flush=True)


def test_full_size_mlp_runs_are_bitwise_reproducible(full_mlp):
    w, X, y, beta0 = full_mlp
    _announce("%s full size, run twice" % w.name)
    masks = gpu_masks(w, 3)
    r1, w1 = gpu_run(w, X, y, beta0, masks, keep=("ghat",))
    r2, w2 = gpu_run(w, X, y, beta0, masks, keep=("ghat",))
    assert torch.equal(w1, w2)
    for t, (a, b) in enumerate(zip(r1, r2)):
        assert np.array_equal(a["ghat"], b["ghat"]), "step %d" % t


def test_full_size_mlp_decode_and_update_are_consistent(full_mlp):
    w, X, y, beta0 = full_mlp
    _announce("%s full size, %d steps" % (w.name, 3))
    sess = gpu_session(w)
    try:
        wv = beta0.clone()
        for mask in gpu_masks(w, 3):
            w_before = wv.cpu().numpy().astype(np.float64)
            sess.step(X, y, wv, mask, w.lr)
            ghat = sess.decoded().cpu().numpy().astype(np.float64)
            surv, d, scale = sess.decode_coeffs(mask)
            acc = np.zeros_like(ghat)
            for dm, j in zip(d, surv):
                acc += dm * sess.coded(int(j)).cpu().numpy().astype(np.float64)
            assert normwise_error(ghat, scale * acc) <= 1e-5
            assert normwise_error(wv.cpu().numpy().astype(np.float64), w_before - w.lr * ghat) <= 1e-6
    finally:
        sess.close()
