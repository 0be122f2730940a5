"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle.

Every case feeds both sides the same seeded inputs.  Straggler masks come
from each side's own generator and must agree bit for bit; then the decoded
gradient and the weights are compared after every step of independent
trajectories (no re-syncing), normwise within 1e-5.

Sizes: every workload's whole trajectory runs at full size against the
oracle's independent trajectory (the two largest also with fewer rows per
partition, same n, c, d and kernel shape).  At full size, in addition, every
ring copy of sampled partitions written at each of c + 2 steps is compared
with the oracle's gradient at the iterate that step started from (the oracle
fed the GPU's iterate), and properties that hold at any size are checked:
decode and update consistency, and bitwise reproducibility.
"""

import numpy as np
import pytest
import torch

import paper_2607_20739_amd as P
from oracle import pgc_oracle as O
from workloads import WORKLOADS, Workload, make_inputs, POLICY_BERNOULLI, POLICY_EXACT, \
    POLICY_SLOWEST, POLICY_UNIFORM_COUNT

from _parity import FP32_TOL, elementwise_error, gpu_masks, gpu_run, gpu_session, normwise_error, \
    oracle_masks, oracle_run

pytestmark = pytest.mark.gpu


def _announce(what):
    print("\n[gpu case] " + what, flush=True)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    P.lib()  # fails loudly when the library is not built


def _to_host(*tensors):
    return [t.cpu().numpy() for t in tensors]


def _check_trajectory(w, X, y, beta0, steps=None, X_host=None, pipelined=True, progress_every=0):
    masks_gpu = gpu_masks(w, steps)
    masks_or = oracle_masks(w, steps)
    for t, (a, b) in enumerate(zip(masks_gpu, masks_or)):
        assert a.tolist() == b.tolist(), "mask of step %d differs" % t
    recs_gpu, _ = gpu_run(w, X, y, beta0, masks_gpu, pipelined=pipelined)
    Xh = X_host if X_host is not None else X.cpu().numpy()
    yh, bh = _to_host(y, beta0)
    recs_or = oracle_run(w, Xh, yh, bh, masks_or, pipelined=pipelined, progress_every=progress_every)
    worst = worst_elem = 0.0
    for t, (g, o) in enumerate(zip(recs_gpu, recs_or)):
        e_g = normwise_error(g["ghat"], o.ghat)
        e_w = normwise_error(g["w"], o.beta)
        worst = max(worst, e_g, e_w)
        worst_elem = max(worst_elem, elementwise_error(g["ghat"], o.ghat), elementwise_error(g["w"], o.beta))
        assert e_g <= FP32_TOL, "step %d: decoded gradient error %.3g" % (t, e_g)
        assert e_w <= FP32_TOL, "step %d: weight error %.3g" % (t, e_w)
    print("  worst normwise error over %d steps: %.3g (elementwise, floor 1e-3 of the max: %.3g)"
          % (len(recs_gpu), worst, worst_elem), flush=True)
    return recs_or


# --------------------------------------------------------------------------
# Whole trajectories
# --------------------------------------------------------------------------

TRAJECTORIES = [
    ("fr_logistic_n4_c2_d64", {}),
    ("crreal_lsq_n8_c3_d1024", {}),
    ("fr_logistic_n32_c4_d4096", dict(N=32 * 512)),
    ("cr_logistic_n128_c8_d8192", dict(N=128 * 96)),
]


@pytest.mark.parametrize("name,resize", TRAJECTORIES, ids=[t[0] for t in TRAJECTORIES])
def test_workload_trajectory_matches_oracle(name, resize):
    w = WORKLOADS[name]
    if resize:
        w = w.resized(**resize)
    _announce("%s N=%d d=%d steps=%d" % (w.name, w.N, w.d, w.steps))
    X, y, beta0 = make_inputs(w, device="cuda")
    _check_trajectory(w, X, y, beta0)


def test_full_size_fr_d4096_trajectory_matches_oracle():
    """The FR workload with all 1,048,576 rows (16 GiB of features): the GPU's
    decoded gradient and weights after every one of its 50 steps against the
    oracle's independent fp64 trajectory on the same inputs and masks.  FR
    evaluates one partition per group per step, N / c rows, which keeps the
    host's fp64 run to about a minute."""
    w = WORKLOADS["fr_logistic_n32_c4_d4096"]
    _announce("%s full size, %d steps against the oracle's trajectory" % (w.name, w.steps))
    X, y, beta0 = make_inputs(w, device="cuda")
    _check_trajectory(w, X, y, beta0, progress_every=10)


def test_full_size_cr_d8192_trajectory_matches_oracle():
    """The largest workload with all 2,097,152 rows (64 GiB of features): the
    GPU's decoded gradient and weights after every one of its 30 steps against
    the oracle's independent fp64 trajectory.  The host holds the features once,
    widened to fp64 chunk by chunk (128 GiB)."""
    w = WORKLOADS["cr_logistic_n128_c8_d8192"]
    _announce("%s full size, %d steps against the oracle's trajectory" % (w.name, w.steps))
    X, y, beta0 = make_inputs(w, device="cuda")
    masks_gpu, masks_or = gpu_masks(w), oracle_masks(w)
    assert [m.tolist() for m in masks_gpu] == [m.tolist() for m in masks_or]
    recs_gpu, _ = gpu_run(w, X, y, beta0, masks_gpu)
    yh, bh = _to_host(y, beta0)
    Xh = np.empty((w.N, w.d), dtype=np.float64)
    chunk = 1 << 16
    for r in range(0, w.N, chunk):
        Xh[r:r + chunk] = X[r:r + chunk].cpu().numpy()      # fp32 -> fp64 is exact
        if (r + chunk) % (1 << 19) == 0:
            print("  host copy: %d of %d rows" % (r + chunk, w.N), flush=True)
    del X
    torch.cuda.empty_cache()
    recs_or = oracle_run(w, Xh, yh, bh, masks_or, progress_every=5)
    del Xh
    worst = 0.0
    for t, (g, o) in enumerate(zip(recs_gpu, recs_or)):
        e_g, e_w = normwise_error(g["ghat"], o.ghat), normwise_error(g["w"], o.beta)
        worst = max(worst, e_g, e_w)
        assert e_g <= FP32_TOL, "step %d: decoded gradient error %.3g" % (t, e_g)
        assert e_w <= FP32_TOL, "step %d: weight error %.3g" % (t, e_w)
    print("  worst normwise error over %d steps: %.3g" % (w.steps, worst), flush=True)


EDGE = [
    # ragged partitions (m = 1003) and a masked column tail (d = 1000 on float4 lanes)
    Workload("edge_cr_lsq_ragged", "CR", "lsq", n=6, c=4, N=6 * 1003, d=1000, lr=0.05, steps=12,
             policy=POLICY_UNIFORM_COUNT, cap=3, seed=11),
    # d % 4 != 0: scalar lanes
    Workload("edge_fr_logistic_d1001", "FR", "logistic", n=6, c=3, N=6 * 777, d=1001, lr=0.1, steps=10,
             policy=POLICY_UNIFORM_COUNT, cap=2, seed=12),
    Workload("edge_fr_logistic_d3", "FR", "logistic", n=4, c=2, N=4 * 50, d=3, lr=0.5, steps=8,
             policy=POLICY_EXACT, cap=1, seed=13),
    # c = 1 (distributed gradient descent), c = n, n = 1
    Workload("edge_cr_lsq_c1", "CR", "lsq", n=5, c=1, N=5 * 300, d=256, lr=0.1, steps=6,
             policy=POLICY_EXACT, cap=0, seed=14),
    Workload("edge_cr_logistic_c_eq_n", "CR", "logistic", n=4, c=4, N=4 * 333, d=128, lr=0.2, steps=10,
             policy=POLICY_UNIFORM_COUNT, cap=3, seed=15),
    Workload("edge_real_c_eq_n", "CR_REAL", "lsq", n=4, c=4, N=4 * 256, d=64, lr=0.02, steps=9,
             policy=POLICY_UNIFORM_COUNT, cap=3, seed=16, code_seed=16),
    Workload("edge_single_worker", "FR", "lsq", n=1, c=1, N=517, d=40, lr=0.1, steps=4,
             policy=POLICY_EXACT, cap=0, seed=17),
    # the widest rows each lane shape handles
    Workload("edge_cr_logistic_d16384", "CR", "logistic", n=4, c=2, N=4 * 40, d=16384, lr=0.05, steps=5,
             policy=POLICY_EXACT, cap=1, seed=18),
    Workload("edge_fr_lsq_d32768", "FR", "lsq", n=2, c=1, N=2 * 24, d=32768, lr=0.01, steps=3,
             policy=POLICY_EXACT, cap=0, seed=19),
    Workload("edge_fr_logistic_d8191", "FR", "logistic", n=4, c=4, N=4 * 37, d=8191, lr=0.05, steps=6,
             policy=POLICY_UNIFORM_COUNT, cap=3, seed=20),
    # degenerate partitions: one row each, and two rows each with a masked float4 column tail
    Workload("edge_cr_logistic_m1", "CR", "logistic", n=8, c=3, N=8, d=64, lr=0.3, steps=7,
             policy=POLICY_UNIFORM_COUNT, cap=2, seed=23),
    Workload("edge_fr_lsq_m2", "FR", "lsq", n=6, c=2, N=12, d=100, lr=0.05, steps=6,
             policy=POLICY_EXACT, cap=1, seed=24),
    # the largest worker count: 256 decode weights and coded words per step
    Workload("edge_cr_logistic_n256", "CR", "logistic", n=256, c=4, N=256 * 8, d=64, lr=0.2, steps=7,
             policy=POLICY_BERNOULLI, cap=3, p=0.01, seed=25),
    Workload("edge_fr_lsq_n256_c8", "FR", "lsq", n=256, c=8, N=256 * 4, d=32, lr=0.05, steps=10,
             policy=POLICY_UNIFORM_COUNT, cap=7, seed=26),
    # every worker may straggle up to s = 7 in one step
    Workload("edge_cr_logistic_heavy", "CR", "logistic", n=16, c=8, N=16 * 64, d=512, lr=0.1, steps=12,
             policy=POLICY_BERNOULLI, cap=7, p=0.4, seed=21),
]


@pytest.mark.parametrize("w", EDGE, ids=[w.name for w in EDGE])
def test_edge_case_trajectory_matches_oracle(w):
    _announce("%s N=%d d=%d" % (w.name, w.N, w.d))
    X, y, beta0 = make_inputs(w, device="cuda")
    _check_trajectory(w, X, y, beta0)


BASELINES = [
    # gradient coding (every slot evaluated each step) for the three codes
    (Workload("gc_fr_logistic", "FR", "logistic", n=8, c=4, N=8 * 500, d=1024, lr=0.05, steps=8,
              policy=POLICY_UNIFORM_COUNT, cap=3, seed=41), False),
    (Workload("gc_real_lsq", "CR_REAL", "lsq", n=8, c=3, N=8 * 700, d=256, lr=0.02, steps=8,
              policy=POLICY_UNIFORM_COUNT, cap=2, seed=42, code_seed=5), False),
    (Workload("gc_cr_logistic", "CR", "logistic", n=6, c=3, N=6 * 300, d=4096, lr=0.02, steps=6,
              policy=POLICY_UNIFORM_COUNT, cap=2, seed=43), False),
    # ignore-straggler SGD with up to n - 1 stragglers
    (Workload("is_sgd_logistic", "IS_SGD", "logistic", n=12, c=1, N=12 * 200, d=512, lr=0.1, steps=10,
              policy=POLICY_UNIFORM_COUNT, cap=11, seed=44), True),
    (Workload("is_sgd_mlp", "IS_SGD", "mlp", n=4, c=1, N=4 * 64, d=64, lr=0.05, steps=5,
              policy=POLICY_EXACT, cap=2, seed=45, hidden=256, classes=10), True),
    # gradient coding on the MLP: every step takes the warm-up path (all c slots at w)
    (Workload("gc_cr_mlp", "CR", "mlp", n=4, c=2, N=4 * 96, d=64, lr=0.05, steps=5,
              policy=POLICY_EXACT, cap=1, seed=50, hidden=256, classes=10), False),
    # the delay model's stragglers: the s workers with the largest delay draws
    (Workload("delay_cr_logistic_n12_c3", "CR", "logistic", n=12, c=3, N=12 * 256, d=768, lr=0.1, steps=10,
              policy=POLICY_SLOWEST, cap=2, seed=46), True),
    (Workload("delay_fr_lsq_n12_c4", "FR", "lsq", n=12, c=4, N=12 * 300, d=512, lr=0.05, steps=10,
              policy=POLICY_SLOWEST, cap=3, seed=47), True),
    # (naive real-valued CR at c = 6 needs decoding coefficients near 2e5, which
    # multiply fp32 rounding past any fp32 bar; c = 3 peaks near 300)
    (Workload("delay_real_logistic_n12_c3", "CR_REAL", "logistic", n=12, c=3, N=12 * 128, d=256, lr=0.05,
              steps=8, policy=POLICY_SLOWEST, cap=2, seed=48, code_seed=7), True),
    (Workload("delay_gc_real_lsq_n12_c3", "CR_REAL", "lsq", n=12, c=3, N=12 * 200, d=256, lr=0.02, steps=8,
              policy=POLICY_SLOWEST, cap=2, seed=49, code_seed=7), False),
]


@pytest.mark.parametrize("w,pipelined", BASELINES, ids=[b[0].name for b in BASELINES])
def test_baseline_trajectory_matches_oracle(w, pipelined):
    _announce("%s pipelined=%s" % (w.name, pipelined))
    X, y, beta0 = make_inputs(w, device="cuda")
    if w.model == "mlp":
        masks_gpu, masks_or = gpu_masks(w), oracle_masks(w)
        assert [m.tolist() for m in masks_gpu] == [m.tolist() for m in masks_or]
        recs_gpu, _ = gpu_run(w, X, y, beta0, masks_gpu, pipelined=pipelined)
        recs_or = oracle_run(w, X.float().cpu().numpy(), y.cpu().numpy(), beta0.cpu().numpy(), masks_or,
                             pipelined=pipelined)
        for t, (g, o) in enumerate(zip(recs_gpu, recs_or)):
            assert normwise_error(g["ghat"], o.ghat) <= 2e-2, t
            assert normwise_error(g["w"], o.beta) <= 2e-2, t
        return
    _check_trajectory(w, X, y, beta0, pipelined=pipelined)


# Hand-made straggler patterns (each admissible: at most s = c - 1 stragglers,
# and an FR group never loses all of its members).
ADVERSARIAL = [
    # FR: group 0 keeps c - 1 stragglers at every step
    (Workload("adv_fr_group_short", "FR", "logistic", n=6, c=3, N=6 * 300, d=256, lr=0.2, steps=9,
              policy=POLICY_EXACT, cap=0, seed=28),
     lambda t, n: [1 if i in (0, 1) else 0 for i in range(n)]),
    # CR: a contiguous run of s stragglers that moves by one worker per step
    (Workload("adv_cr_moving_run", "CR", "lsq", n=8, c=3, N=8 * 256, d=128, lr=0.05, steps=10,
              policy=POLICY_EXACT, cap=0, seed=29),
     lambda t, n: [1 if (i - t) % n in (0, 1) else 0 for i in range(n)]),
    # the real-valued code with worker 5 straggling at every step
    (Workload("adv_real_persistent", "CR_REAL", "lsq", n=8, c=3, N=8 * 256, d=128, lr=0.02, steps=10,
              policy=POLICY_EXACT, cap=0, seed=30, code_seed=2),
     lambda t, n: [1 if i == 5 else 0 for i in range(n)]),
]


@pytest.mark.parametrize("w,pattern", ADVERSARIAL, ids=[a[0].name for a in ADVERSARIAL])
def test_adversarial_stragglers_match_the_oracle_and_still_store(w, pattern):
    """The trajectory under a hand-made straggler pattern matches the oracle,
    and the workers that straggled at the last step still hold, in every slot,
    the gradient of that slot's partition at the iterate where they last
    evaluated it (stragglers compute and store; only their coded gradients
    are left out)."""
    _announce(w.name)
    masks = [np.array(pattern(t, w.n), np.uint8) for t in range(w.steps)]
    X, y, beta0 = make_inputs(w, device="cuda")
    Xh, yh, bh = _to_host(X, y, beta0)
    recs_or = oracle_run(w, Xh, yh, bh, masks)
    sess = gpu_session(w)
    try:
        wv = beta0.clone()
        iterates = []
        for t, mask in enumerate(masks):
            iterates.append(wv.cpu().numpy().astype(np.float64))
            sess.step(X, y, wv, mask, w.lr)
            assert normwise_error(sess.decoded().cpu().numpy(), recs_or[t].ghat) <= FP32_TOL, t
            assert normwise_error(wv.cpu().numpy(), recs_or[t].beta) <= FP32_TOL, t
        place = sess.placement()
        m = w.m
        for i in np.flatnonzero(masks[-1]):
            for l in range(w.c):
                evaluated = [t for t in range(1, w.steps) if (t - 1) % w.c == l]
                tau = evaluated[-1] if evaluated else 0
                k = place[i][l]
                g = O.partition_gradient(w.model, Xh[k * m:(k + 1) * m].astype(np.float64),
                                         yh[k * m:(k + 1) * m].astype(np.float64), iterates[tau])
                err = normwise_error(sess.ring(int(i), l).cpu().numpy(), g)
                assert err <= FP32_TOL, "worker %d slot %d: %.3g" % (i, l, err)
    finally:
        sess.close()


# lr = 0: every ring copy is g_k(w(0)), so the two exact decoders (FR, and the
# real-valued code of Sec. V-A) must return the full-batch mean gradient
# (1/N) sum_r slope(x_r . w(0), y_r) x_r at every step, under every straggler set
# drawn, and w stays w(0) bit for bit.  The reference is that definition written
# out in fp64, not the oracle's pipeline.
ZERO_LR = [
    Workload("zero_lr_fr_logistic", "FR", "logistic", n=6, c=3, N=6 * 700, d=300, lr=0.0, steps=7,
             policy=POLICY_EXACT, cap=2, seed=43),
    Workload("zero_lr_real_lsq", "CR_REAL", "lsq", n=8, c=3, N=8 * 600, d=256, lr=0.0, steps=7,
             policy=POLICY_UNIFORM_COUNT, cap=2, seed=44, code_seed=2),
]


@pytest.mark.parametrize("w", ZERO_LR, ids=[w.name for w in ZERO_LR])
def test_zero_learning_rate_decodes_the_full_batch_gradient(w):
    _announce("%s N=%d d=%d lr=0" % (w.name, w.N, w.d))
    X, y, beta0 = make_inputs(w, device="cuda")
    recs, w_final = gpu_run(w, X, y, beta0, gpu_masks(w))
    Xh, yh, bh = (t.double().cpu().numpy() for t in (X, y, beta0))
    z = Xh @ bh
    slope = 1.0 / (1.0 + np.exp(-z)) - yh if w.model == "logistic" else z - yh
    full = Xh.T @ slope / w.N
    for t, g in enumerate(recs):
        e = normwise_error(g["ghat"], full)
        assert e <= FP32_TOL, "step %d: error %.3g against the full-batch gradient" % (t, e)
    assert torch.equal(w_final, beta0)


def test_unaligned_features_take_the_scalar_path():
    w = Workload("edge_unaligned", "CR", "lsq", n=4, c=2, N=4 * 200, d=256, lr=0.05, steps=6,
                 policy=POLICY_EXACT, cap=1, seed=22)
    _announce(w.name)
    X, y, beta0 = make_inputs(w, device="cuda")
    buf = torch.empty(w.N * w.d + 1, device="cuda", dtype=torch.float32)
    Xu = buf[1:].view(w.N, w.d)
    Xu.copy_(X)
    assert Xu.data_ptr() % 16 != 0
    _check_trajectory(w, Xu, y, beta0, X_host=X.cpu().numpy())


def test_runs_are_bitwise_reproducible():
    w = WORKLOADS["crreal_lsq_n8_c3_d1024"].resized(N=8 * 4096, steps=7)
    _announce(w.name)
    X, y, beta0 = make_inputs(w, device="cuda")
    masks = gpu_masks(w)
    _, w1 = gpu_run(w, X, y, beta0, masks, keep=())
    _, w2 = gpu_run(w, X, y, beta0, masks, keep=())
    assert torch.equal(w1, w2)


def test_restart_reproduces_the_run():
    """Binding the workspace again starts over at t = 0: the same steps then
    give bitwise the same weights, ring and decoded gradient."""
    w = WORKLOADS["crreal_lsq_n8_c3_d1024"].resized(N=8 * 2048, steps=5)
    _announce("restart")
    X, y, beta0 = make_inputs(w, device="cuda")
    masks = gpu_masks(w)
    sess = gpu_session(w)
    try:
        runs = []
        for _ in range(2):
            wv = beta0.clone()
            for t in range(w.steps):
                sess.step(X, y, wv, masks[t], w.lr)
            runs.append((wv, sess.decoded(), sess.ring(3, 1), sess.t))
            sess.restart()
            assert sess.t == 0
        (w1, g1, r1, t1), (w2, g2, r2, t2) = runs
        assert t1 == t2 == w.steps
        assert torch.equal(w1, w2) and torch.equal(g1, g2) and torch.equal(r1, r2)
    finally:
        sess.close()


RESUME = [
    WORKLOADS["fr_logistic_n4_c2_d64"],
    WORKLOADS["crreal_lsq_n8_c3_d1024"].resized(N=8 * 2048, steps=9),
    Workload("resume_cr_logistic", "CR", "logistic", n=6, c=3, N=6 * 500, d=512, lr=0.1, steps=10,
             policy=POLICY_UNIFORM_COUNT, cap=2, seed=27),
]


@pytest.mark.parametrize("k", [0, 1, 4])
@pytest.mark.parametrize("w", RESUME, ids=[w.name for w in RESUME])
def test_resume_from_saved_state_is_bitwise_identical(w, k):
    """Run T steps straight, or k steps, save, and finish in a new session that
    loads the state: the weights and the last decoded gradient agree bit for
    bit.  Starting a new session without the state (a fresh warm-up at the
    checkpoint's w) lands elsewhere once the ring holds older copies."""
    _announce("%s resume after %d steps" % (w.name, k))
    X, y, beta0 = make_inputs(w, device="cuda")
    masks = gpu_masks(w)
    a, b, fresh = gpu_session(w), gpu_session(w), gpu_session(w)
    try:
        wa = beta0.clone()
        for t in range(k):
            a.step(X, y, wa, masks[t], w.lr)
        state = a.save_state()
        w_saved = wa.clone()
        for t in range(k, w.steps):
            a.step(X, y, wa, masks[t], w.lr)
        b.load_state(state)
        assert b.t == k
        wb = w_saved.clone()
        for t in range(k, w.steps):
            b.step(X, y, wb, masks[t], w.lr)
        assert torch.equal(wa, wb)
        assert torch.equal(a.decoded(), b.decoded())
        if k >= 2:
            wf = w_saved.clone()
            for t in range(k, w.steps):
                fresh.step(X, y, wf, masks[t], w.lr)
            assert not torch.equal(wf, wa)
    finally:
        for sess in (a, b, fresh):
            sess.close()


def test_load_state_rejects_foreign_or_broken_buffers():
    w = WORKLOADS["crreal_lsq_n8_c3_d1024"].resized(N=8 * 512, steps=4)
    other = Workload("same_size_cr", "CR", "lsq", n=8, c=3, N=8 * 512, d=1024, lr=0.01, steps=4,
                     policy=POLICY_EXACT, cap=1, seed=2)
    _announce("state rejection")
    X, y, beta0 = make_inputs(w, device="cuda")
    a, b = gpu_session(w), gpu_session(other)
    try:
        wv = beta0.clone()
        for t, mask in enumerate(gpu_masks(w)):
            a.step(X, y, wv, mask, w.lr)
        state = a.save_state()
        assert P.pgc_state_bytes(b.ctx) == state.numel()   # same size, another scheme
        bad = [(b, state), (a, torch.zeros_like(state)), (a, state[:-256]), (a, state[1:])]
        for sess, buf in bad:
            t_before = sess.t
            with pytest.raises(P.PGCError) as e:
                sess.load_state(buf)
            assert e.value.status == P.PGC_EINVAL
            assert sess.t == t_before
        a.load_state(state)
        assert a.t == w.steps
    finally:
        a.close()
        b.close()


def test_rejected_step_has_no_effect():
    w = WORKLOADS["fr_logistic_n4_c2_d64"]
    _announce("rejected step")
    X, y, beta0 = make_inputs(w, device="cuda")
    sess = gpu_session(w)
    try:
        wv = beta0.clone() + 0.25
        sess.step(X, y, wv, np.zeros(4, np.uint8), w.lr)
        before = wv.clone()
        with pytest.raises(P.PGCError) as e:
            sess.step(X, y, wv, np.array([1, 1, 0, 0], np.uint8), w.lr)   # a whole FR group straggles
        assert e.value.status == P.PGC_ESTRAGGLERS
        for bad_lr in (float("nan"), float("inf"), -float("inf")):
            with pytest.raises(P.PGCError) as e:
                sess.step(X, y, wv, np.zeros(4, np.uint8), bad_lr)
            assert e.value.status == P.PGC_EINVAL
        torch.cuda.synchronize()
        assert sess.t == 1
        assert torch.equal(wv, before)
    finally:
        sess.close()


# --------------------------------------------------------------------------
# Full sizes: sampled partitions and properties that hold at any size
# --------------------------------------------------------------------------

FULL = ["crreal_lsq_n8_c3_d1024", "fr_logistic_n32_c4_d4096", "cr_logistic_n128_c8_d8192"]


@pytest.fixture(scope="module", params=FULL)
def full(request):
    """Inputs of one full-size workload, generated once for every test that uses them."""
    w = WORKLOADS[request.param]
    _announce("%s full size: generating inputs" % w.name)
    X, y, beta0 = make_inputs(w, device="cuda")
    yield w, X, y, beta0
    del X, y, beta0
    torch.cuda.empty_cache()


def _sampled_partitions(w):
    return sorted({0, w.n // 2, w.n - 1})


def _host_partition(w, X, y, k):
    m = w.m
    return (X[k * m:(k + 1) * m].double().cpu().numpy(), y[k * m:(k + 1) * m].double().cpu().numpy())


def _fresh_holders(w, place, t, k):
    """(worker, slot) pairs whose ring copy of partition k was written at step t."""
    if t == 0:
        return [(i, l) for i in range(w.n) for l in range(w.c) if place[i][l] == k]
    o = (t - 1) % w.c
    return [(i, o) for i in range(w.n) if place[i][o] == k]


def test_full_size_ring_holds_partition_gradients(full):
    """With lr = 0 the weights stay at beta0, so every copy the ring ever holds
    is g_k(beta0); sampled partitions are compared with the oracle one by one."""
    w, X, y, beta0 = full
    _announce("%s full size, lr = 0" % w.name)
    sess = gpu_session(w)
    try:
        wv = beta0.clone()
        masks = gpu_masks(w, w.c + 1)
        for t in range(w.c + 1):
            sess.step(X, y, wv, masks[t], 0.0)
        place = sess.placement()
        beta_h = beta0.cpu().numpy().astype(np.float64)
        for k in _sampled_partitions(w):
            Xk, yk = _host_partition(w, X, y, k)
            g = O.partition_gradient(w.model, Xk, yk, beta_h)
            holders = [(i, l) for i in range(w.n) for l in range(w.c) if place[i][l] == k]
            assert len(holders) == w.c
            for i, l in holders:
                err = normwise_error(sess.ring(i, l).cpu().numpy(), g)
                assert err <= FP32_TOL, "partition %d, worker %d slot %d: %.3g" % (k, i, l, err)
        assert torch.equal(wv, beta0)
    finally:
        sess.close()


def test_full_size_fresh_slots_match_the_oracle_at_every_iterate(full):
    """At full size and the workload's learning rate, each step's freshly written
    ring copies of sampled partitions equal the oracle's gradient of that
    partition at the iterate the step started from (Sec. III gradient; the slot
    the schedule of Sec. IV-A / V-B writes at step t), within the fp32 bar.
    The oracle is fed the GPU's iterate (teacher-forced), so every step checks
    the gradient kernel at a nonzero w over all of a partition's rows."""
    w, X, y, beta0 = full
    _announce("%s full size, teacher-forced slots over %d steps" % (w.name, w.c + 2))
    sampled = _sampled_partitions(w)
    host = {k: _host_partition(w, X, y, k) for k in sampled}
    sess = gpu_session(w)
    try:
        place = sess.placement()
        wv = beta0.clone()
        checked = worst = 0.0
        for t, mask in enumerate(gpu_masks(w, w.c + 2)):
            w_before = wv.cpu().numpy().astype(np.float64)
            sess.step(X, y, wv, mask, w.lr)
            for k in sampled:
                holders = _fresh_holders(w, place, t, k)
                if not holders:
                    continue
                g = O.partition_gradient(w.model, host[k][0], host[k][1], w_before)
                for i, l in holders:
                    err = normwise_error(sess.ring(i, l).cpu().numpy(), g)
                    worst = max(worst, err)
                    checked += 1
                    assert err <= FP32_TOL, "step %d, partition %d, worker %d slot %d: %.3g" % (
                        t, k, i, l, err)
            if t >= 1:
                assert np.any(w_before != 0.0), "the iterate must have moved off w(0)"
        # every sampled partition is checked at a pipelined step, not only at t = 0
        for k in sampled:
            assert any(_fresh_holders(w, place, t, k) for t in range(1, w.c + 2))
        print("  %d slots checked, worst normwise error %.3g" % (checked, worst), flush=True)
    finally:
        sess.close()


def test_full_size_decode_and_update_are_consistent(full):
    """At full size and the real learning rate: the decoded gradient is the
    weighted sum of the coded gradients with the library's decode weights, the
    coded gradients are the sums of the ring copies, and w moves by -lr * ghat."""
    w, X, y, beta0 = full
    _announce("%s full size, %d steps" % (w.name, w.c + 2))
    sess = gpu_session(w)
    try:
        wv = beta0.clone()
        B = sess.encoding_matrix()
        place = sess.placement()
        for t, mask in enumerate(gpu_masks(w, w.c + 2)):
            w_before = wv.cpu().numpy().astype(np.float64)
            sess.step(X, y, wv, mask, w.lr)
            ghat = sess.decoded().cpu().numpy().astype(np.float64)
            coded = np.stack([sess.coded(j).cpu().numpy() for j in range(sess.n_coded)]).astype(np.float64)
            surv, d, scale = sess.decode_coeffs(mask)
            idx = surv // w.c if w.scheme == "FR" else surv
            expect = scale * (d[:, None] * coded[idx]).sum(axis=0)
            assert normwise_error(ghat, expect) <= 1e-6
            w_after = wv.cpu().numpy().astype(np.float64)
            assert normwise_error(w_after, w_before - w.lr * ghat) <= 1e-6
            for j in sorted({0, sess.n_coded - 1}):
                worker = j * w.c if w.scheme == "FR" else j
                ring = sum(B[worker, place[worker][l]] * sess.ring(worker, l).cpu().numpy().astype(np.float64)
                           for l in range(w.c))
                assert normwise_error(coded[j], ring) <= 1e-6
    finally:
        sess.close()


def test_full_size_runs_are_bitwise_reproducible(full):
    """Two runs of the same steps at full size (every kernel shape the workloads
    use, including rows that span several waves) give bitwise the same decoded
    gradient at every step and the same final weights."""
    w, X, y, beta0 = full
    _announce("%s full size, run twice" % w.name)
    masks = gpu_masks(w, w.c + 2)
    r1, w1 = gpu_run(w, X, y, beta0, masks, keep=("ghat",))
    r2, w2 = gpu_run(w, X, y, beta0, masks, keep=("ghat",))
    assert torch.equal(w1, w2)
    for t, (a, b) in enumerate(zip(r1, r2)):
        assert np.array_equal(a["ghat"], b["ghat"]), "step %d" % t
