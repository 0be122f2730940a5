"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a worked
example printed in the paper, a closed-form identity (Sec. V-B eq. (1) and
(2), the copy-weight bound), a textbook special case (c = 1 is full-batch
gradient descent; the warm-up step is gradient coding), brute force over
every admissible straggler set, finite differences, or a second bookkeeping
of the same schedule (per-worker rings, as in Sec. VI-A).
"""

import itertools
import math
import os

import numpy as np
import pytest

from oracle import pgc_oracle as O
from oracle import rng as R

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _data(model, N, d, seed, shape=None):
    g = np.random.default_rng(seed)
    if model == O.MLP:
        d_in, h, k = shape
        X = g.random((N, d_in))
        y = g.integers(0, k, N).astype(np.float64)
        beta = g.normal(0.0, 0.3, O.mlp_param_count(shape))
        return X, y, beta
    X = g.normal(size=(N, d))
    w_star = g.normal(size=d) / math.sqrt(d)
    z = X @ w_star
    if model == O.LOGISTIC:
        y = (g.random(N) < O.sigmoid(z)).astype(np.float64)
    else:
        y = z + 0.1 * g.normal(size=N)
    return X, y, 0.1 * g.normal(size=d)


def _full_gradient_linear(model, X, y, beta):
    """Gradient of F(beta) = (1/N) sum_i f(beta; x_i, y_i) over all rows (Sec. III)."""
    z = X @ beta
    r = (1.0 / (1.0 + np.exp(-z)) - y) if model == O.LOGISTIC else (z - y)
    return X.T @ r / X.shape[0]


def _admissible_masks(n, s):
    for k in range(s + 1):
        for strag in itertools.combinations(range(n), k):
            mask = np.zeros(n, dtype=np.uint8)
            mask[list(strag)] = 1
            yield mask


def _code_matrix(n, c, seed=7):
    return O.cyclic_encoding_matrix(n, c, R.null_space_generator(seed, c - 1, n))


# --------------------------------------------------------------------------
# Placement and schedule
# --------------------------------------------------------------------------

def test_fr_placement_matches_the_printed_example():
    rows = {}
    with open(os.path.join(GOLDEN, "fr_placement_n4_c2.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            worker, parts = line.split(":")
            rows[int(worker)] = [int(p) for p in parts.split()]
    assert O.placement(O.FR, 4, 2) == [rows[i] for i in range(4)]


@pytest.mark.parametrize("n,c", [(4, 2), (6, 3), (8, 4), (12, 6), (32, 4), (5, 5), (7, 1)])
def test_fr_groups_hold_disjoint_blocks(n, c):
    P = O.placement(O.FR, n, c)
    groups = {}
    for i, parts in enumerate(P):
        groups.setdefault(tuple(parts), []).append(i)
    assert len(groups) == n // c                          # n/c groups ...
    assert all(len(m) == c for m in groups.values())      # ... of c workers
    assert sorted(k for parts in groups for k in parts) == list(range(n))   # a partition of the data


@pytest.mark.parametrize("scheme", [O.CR, O.CR_REAL])
@pytest.mark.parametrize("n,c", [(4, 2), (5, 2), (7, 3), (8, 3), (12, 6), (6, 6), (9, 1)])
def test_cr_every_partition_has_c_holders(scheme, n, c):
    P = O.placement(scheme, n, c)
    counts = np.zeros(n, dtype=int)
    for parts in P:
        assert len(set(parts)) == c
        for k in parts:
            counts[k] += 1
    assert (counts == c).all()
    # Cyclic: the holders of D_k are c consecutive workers ending at k.
    for k in range(n):
        holders = sorted(i for i in range(n) if k in P[i])
        assert sorted((k - o) % n for o in range(c)) == holders


@pytest.mark.parametrize("scheme,n,c", [(O.FR, 8, 4), (O.CR, 7, 3), (O.CR, 12, 6), (O.FR, 6, 2)])
def test_schedule_rotates_one_partition_per_step(scheme, n, c):
    P = O.placement(scheme, n, c)
    T = 4 * c + 3
    for t in range(1, T):
        ev = [P[i][O.evaluated_slot(t, c)] for i in range(n)]
        if scheme == O.CR:
            assert sorted(ev) == list(range(n))           # a permutation of all partitions
        else:
            for i in range(n):                             # a group evaluates one partition
                assert ev[i] == ev[(i // c) * c]
    for i in range(n):                                     # any c consecutive steps cover all slots
        for t0 in range(1, T - c):
            assert sorted(O.evaluated_slot(t, c) for t in range(t0, t0 + c)) == list(range(c))


@pytest.mark.parametrize("scheme,n,c", [(O.FR, 8, 4), (O.CR, 7, 3), (O.CR, 5, 5)])
def test_copies_are_at_most_c_minus_1_steps_stale(scheme, n, c):
    P = O.placement(scheme, n, c)
    for t in range(0, 5 * c):
        for i in range(n):
            terms = O.coded_terms(scheme, n, c, i, t)
            assert sorted(slot for slot, _, _ in terms) == list(range(c))   # every held partition once
            assert [k for _, k, _ in sorted(terms)] == P[i]
            for slot, k, tau in terms:
                assert tau <= t
                if t >= c:
                    assert t - c + 1 <= tau                 # s(t, i) in [t - c + 1, t] (Sec. IV-B)
                # The copy's step is the latest step <= t that evaluated this slot.
                evals = [u for u in range(1, t + 1) if O.evaluated_slot(u, c) == slot]
                assert tau == (max(evals) if evals else 0)


# --------------------------------------------------------------------------
# The run against a second bookkeeping and against textbook special cases
# --------------------------------------------------------------------------

@pytest.mark.parametrize("scheme,model,n,c", [
    (O.FR, O.LOGISTIC, 6, 3), (O.CR, O.LSQ, 5, 3), (O.CR_REAL, O.LSQ, 6, 3), (O.CR, O.LOGISTIC, 4, 4)])
def test_coded_gradients_equal_per_worker_rings(scheme, model, n, c):
    """Sec. VI-A: each worker keeps the latest gradient of each partition it holds."""
    N, d, T = n * 16, 5, 3 * c + 2
    X, y, beta0 = _data(model, N, d, seed=n * 10 + c)
    B = _code_matrix(n, c) if scheme == O.CR_REAL else None
    masks = [np.zeros(n, dtype=np.uint8) for _ in range(T)]
    recs = O.run(scheme, model, n, c, X, y, beta0, 0.3, masks, B=B)
    P = O.placement(scheme, n, c)
    E = O.encoding_coefficients(scheme, n, c, B)
    m = N // n
    ring = [[None] * c for _ in range(n)]
    beta = beta0
    for t in range(T):
        for i in range(n):
            slots = range(c) if t == 0 else [(t - 1) % c]
            for l in slots:
                k = P[i][l]
                ring[i][l] = O.partition_gradient(model, X[k * m:(k + 1) * m], y[k * m:(k + 1) * m], beta)
        for i in range(n):
            word = sum(E[i][l] * ring[i][l] for l in range(c))
            np.testing.assert_allclose(recs[t].coded[i], word, rtol=1e-13, atol=1e-15)
        beta = recs[t].beta


@pytest.mark.parametrize("model", [O.LOGISTIC, O.LSQ])
@pytest.mark.parametrize("scheme", [O.FR, O.CR, O.CR_REAL])
def test_c1_is_full_batch_gradient_descent(scheme, model):
    """c = 1, s = 0 is DGD (Sec. VI-A): plain gradient descent on F."""
    n, N, d, T, lr = 4, 64, 6, 7, 0.4
    X, y, beta0 = _data(model, N, d, seed=3)
    B = _code_matrix(n, 1) if scheme == O.CR_REAL else None
    recs = O.run(scheme, model, n, 1, X, y, beta0, lr, [np.zeros(n, np.uint8)] * T, B=B)
    beta = beta0.copy()
    for t in range(T):
        g = _full_gradient_linear(model, X, y, beta)
        np.testing.assert_allclose(recs[t].ghat, g, rtol=1e-12, atol=1e-14)
        beta = beta - lr * g
        np.testing.assert_allclose(recs[t].beta, beta, rtol=1e-12, atol=1e-14)


def test_lsq_c1_matches_closed_form_gradient():
    """Least squares: the DGD iterate is beta - eta X^T (X beta - y) / N."""
    n, N, d = 4, 40, 3
    X, y, beta0 = _data(O.LSQ, N, d, seed=11)
    recs = O.run(O.CR, O.LSQ, n, 1, X, y, beta0, 0.2, [np.zeros(n, np.uint8)] * 2)
    expect = beta0 - 0.2 * (X.T @ (X @ beta0 - y)) / N
    np.testing.assert_allclose(recs[0].beta, expect, rtol=1e-13)


@pytest.mark.parametrize("n,c", [(4, 2), (6, 3), (8, 4)])
def test_fr_warmup_is_exact_gradient_coding(n, c):
    """At t = 0 every admissible straggler set decodes to grad F(beta0) (Sec. IV-A)."""
    N, d = n * 8, 4
    X, y, beta0 = _data(O.LOGISTIC, N, d, seed=n)
    g_full = _full_gradient_linear(O.LOGISTIC, X, y, beta0)
    for mask in _admissible_masks(n, c - 1):
        rec = O.run(O.FR, O.LOGISTIC, n, c, X, y, beta0, 0.5, [mask])[0]
        np.testing.assert_allclose(rec.ghat, g_full, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("n,c", [(4, 2), (6, 3), (8, 2)])
def test_fr_decode_picks_one_per_group_and_ignores_which(n, c):
    P = O.placement(O.FR, n, c)
    for mask in _admissible_masks(n, c - 1):
        J = O.survivors(mask)
        d, scale = O.decode_weights(O.FR, n, c, J)
        assert scale == 1.0 / n
        assert set(d.tolist()) <= {0.0, 1.0}
        chosen = [j for dm, j in zip(d, J) if dm == 1.0]
        assert sorted(j // c for j in chosen) == list(range(n // c))     # exactly one per group
        assert all(j == min(i for i in J if i // c == j // c) for j in chosen)
    # The whole trajectory is the same for every admissible mask sequence.
    N, d_, T = n * 6, 3, 3 * c + 1
    X, y, beta0 = _data(O.LOGISTIC, N, d_, seed=5)
    g = np.random.default_rng(1)
    masks_list = list(_admissible_masks(n, c - 1))
    ref = O.run(O.FR, O.LOGISTIC, n, c, X, y, beta0, 0.5, [np.zeros(n, np.uint8)] * T)
    for trial in range(4):
        seq = [masks_list[g.integers(len(masks_list))] for _ in range(T)]
        got = O.run(O.FR, O.LOGISTIC, n, c, X, y, beta0, 0.5, seq)
        for a, b in zip(got, ref):
            assert np.array_equal(a.beta, b.beta)


@pytest.mark.parametrize("n,c", [(4, 2), (5, 2), (7, 3), (8, 3)])
def test_cr_full_sum_identity_eq1(n, c):
    """Sec. V-B eq. (1): sum over all workers of ghat_j = sum_k sum_h g_k^{(s(t,k,h))}."""
    N, d, T = n * 8, 4, 3 * c + 1
    X, y, beta0 = _data(O.LSQ, N, d, seed=n + c)
    masks = [np.zeros(n, np.uint8)] * T
    recs = O.run(O.CR, O.LSQ, n, c, X, y, beta0, 0.2, masks)
    betas = [beta0] + [r.beta for r in recs]
    m = N // n
    for t in range(T):
        total = np.zeros(d)
        for k in range(n):
            for h in range(c):                     # h-th holder: worker (k - h) mod n, slot h
                evals = [u for u in range(1, t + 1) if (u - 1) % c == h]
                tau = max(evals) if evals else 0
                total += O.partition_gradient(O.LSQ, X[k * m:(k + 1) * m], y[k * m:(k + 1) * m], betas[tau])
        np.testing.assert_allclose(recs[t].coded.sum(axis=0), total, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("n,c", [(4, 2), (5, 2), (7, 3), (8, 3), (6, 5)])
def test_cr_decoder_is_unbiased_eq2(n, c):
    """Sec. V-B eq. (2): over all size-(n-s) survivor sets, the mean decode is gbar."""
    s = c - 1
    g = np.random.default_rng(n * c)
    coded = g.normal(size=(n, 6))
    gbar = coded.sum(axis=0) / (n * c)
    acc = np.zeros(6)
    count = 0
    for J in itertools.combinations(range(n), n - s):
        d, scale = O.decode_weights(O.CR, n, c, list(J))
        acc += scale * (d[:, None] * coded[list(J)]).sum(axis=0)
        count += 1
    assert count == math.comb(n, s)
    np.testing.assert_allclose(acc / count, gbar, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("n,c", [(4, 2), (5, 2), (7, 3), (8, 3), (12, 6), (6, 5), (9, 7)])
def test_cr_copy_weight_bound(n, c):
    """Sec. V-B: 0 <= |N_k| / mu < 2, and the bound n/(n-s) or n/(s+1) is attained."""
    s = c - 1
    mu = (n - s) * c / n
    worst = 0.0
    for J in itertools.combinations(range(n), n - s):
        counts = O.copy_counts(O.CR, n, c, J)
        assert counts.sum() == (n - s) * c
        worst = max(worst, counts.max() / mu)
    assert worst < 2.0
    expect = n / (n - s) if s <= (n - 1) / 2 else n / (s + 1)
    assert worst == pytest.approx(expect, rel=1e-15)


@pytest.mark.parametrize("n,c", [(4, 2), (5, 3), (8, 3), (6, 4)])
def test_cr_no_straggler_step_is_the_average(n, c):
    """|J| = n: ghat = (1/(nc)) sum_j ghat_j; with eta = 0 it is grad F(beta0)."""
    N, d = n * 8, 4
    X, y, beta0 = _data(O.LOGISTIC, N, d, seed=2)
    recs = O.run(O.CR, O.LOGISTIC, n, c, X, y, beta0, 0.0, [np.zeros(n, np.uint8)] * (c + 2))
    g_full = _full_gradient_linear(O.LOGISTIC, X, y, beta0)
    for r in recs:
        np.testing.assert_allclose(r.ghat, r.coded.sum(axis=0) / (n * c), rtol=1e-13)
        np.testing.assert_allclose(r.ghat, g_full, rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("n,c", [(4, 2), (5, 2), (6, 3), (8, 3)])
def test_real_code_decodes_exactly_for_every_admissible_set(n, c):
    """Sec. V-A: with current copies any n - s coded gradients recover the partition sum."""
    B = _code_matrix(n, c, seed=n)
    N, d = n * 8, 3
    X, y, beta0 = _data(O.LSQ, N, d, seed=9)
    g_full = _full_gradient_linear(O.LSQ, X, y, beta0)
    for mask in _admissible_masks(n, c - 1):
        recs = O.run(O.CR_REAL, O.LSQ, n, c, X, y, beta0, 0.0, [mask] * 2, B=B)
        for r in recs:
            np.testing.assert_allclose(r.ghat, g_full, rtol=1e-9, atol=1e-12)
            np.testing.assert_allclose(r.alpha.sum(axis=0), np.ones(n), rtol=0, atol=1e-9)


def test_real_code_rows_lie_in_the_null_space():
    n, c = 8, 3
    H = R.null_space_generator(5, c - 1, n)
    B = O.cyclic_encoding_matrix(n, c, H)
    np.testing.assert_allclose(H @ np.ones(n), 0.0, atol=1e-14)
    np.testing.assert_allclose(H @ B.T, 0.0, atol=1e-12)
    for j in range(n):
        support = {(j + l) % n for l in range(c)}
        assert B[j, j] == 1.0
        assert all(B[j, k] == 0.0 for k in range(n) if k not in support)


def test_real_code_minimum_norm_decode_with_extra_survivors():
    """|J| > n - s: the decode weights solve B_J^T d = 1 and lie in range(B_J) (minimum norm)."""
    n, c = 8, 3
    B = _code_matrix(n, c, seed=3)
    for J in ([0, 1, 2, 3, 4, 5, 6, 7], [0, 2, 3, 4, 5, 6, 7]):
        d, scale = O.decode_weights(O.CR_REAL, n, c, J, B)
        A = B[J, :].T
        np.testing.assert_allclose(A @ d, np.ones(n), atol=1e-10)
        # Minimum norm <=> d is orthogonal to the null space of A.
        _, sv, vt = np.linalg.svd(A)
        null = vt[np.sum(sv > 1e-10 * sv[0]):]
        np.testing.assert_allclose(null @ d, 0.0, atol=1e-10)
        assert scale == 1.0 / n


def test_decoder_rejects_too_many_stragglers():
    with pytest.raises(O.StragglerError):
        O.decode_weights(O.CR, 6, 3, [0, 1, 2])
    with pytest.raises(O.StragglerError):
        O.decode_weights(O.FR, 6, 3, [3, 4, 5])
    # With at most s = c - 1 stragglers every FR group keeps a survivor.
    d, _ = O.decode_weights(O.FR, 6, 3, [0, 3, 4, 5])
    assert d.tolist() == [1.0, 1.0, 0.0, 0.0]


# --------------------------------------------------------------------------
# Gradients
# --------------------------------------------------------------------------

@pytest.mark.parametrize("model", [O.LOGISTIC, O.LSQ])
def test_linear_gradients_match_finite_differences(model):
    X, y, beta = _data(model, 50, 7, seed=21)
    g = O.partition_gradient(model, X, y, beta)
    h = 1e-6
    fd = np.array([(O.partition_loss(model, X, y, beta + h * e) - O.partition_loss(model, X, y, beta - h * e)) / (2 * h)
                   for e in np.eye(7)])
    np.testing.assert_allclose(g, fd, rtol=1e-6, atol=1e-9)


def test_mlp_gradient_matches_finite_differences():
    """MLP gradient (R3): W1 and W2 enter as bf16 values, so the check sits on a
    point whose weights are already bf16 and steps one bf16 ulp for weights."""
    shape = (6, 5, 3)
    d_in, hdim, k = shape
    X, y, beta = _data(O.MLP, 20, None, seed=4, shape=shape)
    W1, b1, W2, b2 = O.mlp_unpack(beta, shape)     # views into beta
    W1[:] = O.round_to_bf16(W1)
    W2[:] = O.round_to_bf16(W2)
    assert np.min(np.abs(X @ W1 + b1)) > 1e-3, "the point must stay away from the ReLU kink"
    g = O.partition_gradient(O.MLP, X, y, beta, shape)
    loss = lambda b: O.partition_loss(O.MLP, X, y, b, shape)
    h = 1e-6
    nW1 = d_in * hdim
    for i in list(range(nW1, nW1 + hdim)) + list(range(beta.size - k, beta.size)):   # biases, fp64
        e = np.zeros_like(beta)
        e[i] = h
        assert g[i] == pytest.approx((loss(beta + e) - loss(beta - e)) / (2 * h), rel=1e-6, abs=1e-9)
    for i in [0, 7, nW1 - 1, nW1 + hdim, nW1 + hdim + hdim * k - 1]:                 # weights, bf16 steps
        v = beta[i]
        ulp = 2.0 ** (math.floor(math.log2(abs(v))) - 7)
        up, dn = beta.copy(), beta.copy()
        up[i], dn[i] = v + ulp, v - ulp
        assert O.round_to_bf16(up[i]) == up[i] and O.round_to_bf16(dn[i]) == dn[i]
        assert g[i] == pytest.approx((loss(up) - loss(dn)) / (2 * ulp), rel=2e-3, abs=1e-6)


def test_bf16_rounding_is_round_to_nearest_even():
    vals = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -9, -2.5, 65504.0])
    expect = np.array([1.0, 1.0, 1.0 + 4 * 2.0 ** -8, 1.0, -2.5, 65536.0])
    assert np.array_equal(O.round_to_bf16(vals), expect)


def test_least_squares_loss_decreases_under_pgc():
    """Convergence sanity (Sec. V-C): with a small step the loss falls every step."""
    n, c = 8, 3
    X, y, _ = _data(O.LSQ, n * 64, 16, seed=31)
    beta0 = np.zeros(16)
    masks = [R.straggler_mask(99, t, R.POLICY_UNIFORM_COUNT, n, c - 1) for t in range(40)]
    recs = O.run(O.CR, O.LSQ, n, c, X, y, beta0, 0.05, masks)
    losses = [O.full_loss(O.LSQ, X, y, beta0)] + [O.full_loss(O.LSQ, X, y, r.beta) for r in recs]
    assert all(b <= a + 1e-15 for a, b in zip(losses, losses[1:]))


# --------------------------------------------------------------------------
# Random draws
# --------------------------------------------------------------------------

def test_splitmix64_known_answers():
    with open(os.path.join(GOLDEN, "splitmix64_known_answers.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            seed, index, out = line.split()
            assert R.splitmix64(int(seed), int(index)) == int(out, 0)


def test_mask_policies_draw_the_stated_counts():
    n = 12
    for t in range(300):
        assert R.straggler_mask(5, t, R.POLICY_EXACT, n, 3).sum() == 3
        assert R.straggler_mask(5, t, R.POLICY_UNIFORM_COUNT, n, 2).sum() <= 2
        assert R.straggler_mask(5, t, R.POLICY_BERNOULLI, n, 2, 0.3).sum() <= 2


def test_masks_make_every_worker_equally_likely_to_straggle():
    """Sec. V-B's unbiasedness assumes each worker straggles with equal probability."""
    from scipy.stats import chisquare, binomtest
    n, T = 8, 20000
    for policy, cap, p in [(R.POLICY_EXACT, 1, 0.0), (R.POLICY_UNIFORM_COUNT, 2, 0.0),
                           (R.POLICY_BERNOULLI, 3, 0.1), (R.POLICY_SLOWEST, 2, 0.0)]:
        freq = np.zeros(n)
        counts = np.zeros(cap + 1)
        for t in range(T):
            mask = R.straggler_mask(1234, t, policy, n, cap, p)
            freq += mask
            counts[int(mask.sum())] += 1
        assert chisquare(freq).pvalue > 1e-4
        if policy == R.POLICY_UNIFORM_COUNT:
            assert chisquare(counts).pvalue > 1e-4
        if policy == R.POLICY_BERNOULLI:
            # P(count = 0) = (1 - p)^n for the Bernoulli policy.
            assert binomtest(int(counts[0]), T, (1 - p) ** n).pvalue > 1e-4


def test_delay_step_waits_for_the_fastest():
    """Sec. VI-B: the master continues with the n - s workers that finish first."""
    n = 12
    for s in range(n):
        for t in range(50):
            mask, delays, sec = R.delay_step(77, t, n, s, 1.5, 0.25)
            finish = 0.25 + delays
            assert mask.sum() == s and np.all(delays >= 0.0)
            waited, skipped = finish[mask == 0], finish[mask == 1]
            assert sec == waited.max()
            if s:
                assert skipped.min() >= waited.max()
            # The master proceeds at the first instant when n - s have finished.
            assert (finish <= sec).sum() >= n - s and (finish < sec).sum() < n - s
            # The workers it skips are those of the slowest-draws policy.
            assert np.array_equal(mask, R.straggler_mask(77, t, R.POLICY_SLOWEST, n, s))
    mask, delays, sec = R.delay_step(77, 3, n, 0, 2.0, 1.0)
    assert sec == 1.0 + delays.max() and mask.sum() == 0
    mask, delays, sec = R.delay_step(77, 3, n, 4, 0.0, 1.0)
    assert sec == 1.0 and np.all(delays == 0.0) and mask.sum() == 4


@pytest.mark.parametrize("n,s,mean", [(12, 0, 1.0), (12, 1, 2.0), (12, 3, 1.0), (5, 4, 2.0)])
def test_delay_step_matches_exponential_order_statistics(n, s, mean):
    """The k-th smallest of n i.i.d. exponentials of mean mu has mean
    mu * sum_{j<k} 1/(n - j) and variance mu^2 * sum_{j<k} 1/(n - j)^2
    (Renyi's representation); k = n - s here."""
    T = 6000
    secs = np.array([R.delay_step(2024, t, n, s, mean)[2] for t in range(T)])
    k = n - s
    mu = mean * sum(1.0 / (n - j) for j in range(k))
    sd = mean * math.sqrt(sum(1.0 / (n - j) ** 2 for j in range(k)))
    assert abs(secs.mean() - mu) < 5.0 * sd / math.sqrt(T)
    assert abs(secs.std() - sd) < 0.1 * sd


def test_delays_are_exponential():
    from scipy.stats import kstest
    delays = np.concatenate([R.delay_step(5, t, 16, 0, 2.0)[1] for t in range(2000)])
    assert kstest(delays, "expon", args=(0.0, 2.0)).pvalue > 1e-4


def test_null_space_generator_entries():
    H = R.null_space_generator(17, 3, 9)
    assert H.shape == (3, 9)
    assert np.all(H[:, :-1] >= -1.0) and np.all(H[:, :-1] < 1.0)
    assert np.array_equal(H[:, -1], -np.array([sum(H[a, :-1].tolist()) for a in range(3)]))


# --------------------------------------------------------------------------
# Baselines: gradient coding (no pipelining), DGD and IS-SGD (Sec. III, VI)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("scheme,n,c", [(O.FR, 6, 3), (O.FR, 8, 2), (O.CR_REAL, 6, 3), (O.CR_REAL, 5, 2)])
def test_gradient_coding_coincides_with_dgd(scheme, n, c):
    """Sec. VI-B: GC recovers the same aggregated gradient as DGD, whatever straggles."""
    N, d, T, lr = n * 10, 5, 8, 0.3
    X, y, beta0 = _data(O.LOGISTIC, N, d, seed=40 + n)
    B = _code_matrix(n, c, seed=n) if scheme == O.CR_REAL else None
    masks = [R.straggler_mask(7, t, R.POLICY_UNIFORM_COUNT, n, c - 1) for t in range(T)]
    recs = O.run(scheme, O.LOGISTIC, n, c, X, y, beta0, lr, masks, B=B, pipelined=False)
    beta = beta0.copy()
    for t in range(T):
        beta = beta - lr * _full_gradient_linear(O.LOGISTIC, X, y, beta)
        np.testing.assert_allclose(recs[t].beta, beta, rtol=1e-9, atol=1e-12)


def test_gradient_coding_cr_unit_without_stragglers_is_dgd():
    n, c = 6, 3
    X, y, beta0 = _data(O.LSQ, n * 8, 4, seed=51)
    recs = O.run(O.CR, O.LSQ, n, c, X, y, beta0, 0.2, [np.zeros(n, np.uint8)] * 5, pipelined=False)
    beta = beta0.copy()
    for r in recs:
        beta = beta - 0.2 * _full_gradient_linear(O.LSQ, X, y, beta)
        np.testing.assert_allclose(r.beta, beta, rtol=1e-12, atol=1e-14)


def test_is_sgd_without_stragglers_is_dgd():
    """Sec. VI-A: IS-SGD is DGD when s = 0."""
    n = 5
    X, y, beta0 = _data(O.LOGISTIC, n * 12, 6, seed=52)
    recs = O.run(O.IS_SGD, O.LOGISTIC, n, 1, X, y, beta0, 0.4, [np.zeros(n, np.uint8)] * 6)
    beta = beta0.copy()
    for r in recs:
        beta = beta - 0.4 * _full_gradient_linear(O.LOGISTIC, X, y, beta)
        np.testing.assert_allclose(r.beta, beta, rtol=1e-12, atol=1e-14)


@pytest.mark.parametrize("n,s", [(5, 1), (6, 3), (7, 6)])
def test_is_sgd_is_unbiased_over_straggler_sets(n, s):
    """Averaging the survivors' gradients is unbiased over uniformly chosen straggler sets."""
    X, y, beta0 = _data(O.LSQ, n * 6, 4, seed=53)
    g_full = _full_gradient_linear(O.LSQ, X, y, beta0)
    acc = np.zeros(4)
    count = 0
    for strag in itertools.combinations(range(n), s):
        mask = np.zeros(n, np.uint8)
        mask[list(strag)] = 1
        acc += O.run(O.IS_SGD, O.LSQ, n, 1, X, y, beta0, 0.0, [mask])[0].ghat
        count += 1
    np.testing.assert_allclose(acc / count, g_full, rtol=1e-12, atol=1e-15)


def test_is_sgd_rejects_an_empty_survivor_set_and_c_above_one():
    with pytest.raises(O.StragglerError):
        O.decode_weights(O.IS_SGD, 4, 1, [])
    with pytest.raises(ValueError):
        O.placement(O.IS_SGD, 4, 2)


def test_elementwise_error_with_floor():
    """The reported elementwise metric: relative per entry, with entries below
    1e-3 of the largest judged against that floor instead of themselves."""
    from _parity import elementwise_error
    b = np.array([10.0, 1e-9, -2.0])
    assert elementwise_error(b, b) == 0.0
    assert elementwise_error(b * (1 + 1e-6), b) == pytest.approx(1e-6)
    # An absolute error of 1e-6 on the tiny entry is measured against 1e-3 * 10.
    assert elementwise_error(b + np.array([0.0, 1e-6, 0.0]), b) == pytest.approx(1e-4)


def test_naive_cr_matches_the_printed_n4_c2_example():
    """Sec. V-A's worked example of naive PGC-CR (n = 4, c = 2): D_1 decoded as
    -g_1^(t-1) + 2 g_1^(t), the fresh copy from W_0's second slot, the stale one
    from W_1's first (tests/golden/naive_cr_example_n4_c2.txt).  The example's
    matrix is not printed; in the family of real codes used here (rows in the
    null space of H, whose entries sum to zero), H = [-2, 1, a, 1 - a] with W_3
    straggling yields exactly these coefficients for any a."""
    with open(os.path.join(GOLDEN, "naive_cr_example_n4_c2.txt")) as f:
        lines = [l.split() for l in f if l.strip() and not l.startswith("#")]
    k = int(lines[0][1])
    copies = [tuple(int(v) for v in l[1:]) for l in lines[1:]]
    n, c = 4, 2
    for a in (0.5, 0.3, -1.7):
        H = np.array([[-2.0, 1.0, a, 1.0 - a]])
        B = O.cyclic_encoding_matrix(n, c, H)
        mask = np.array([0, 0, 0, 1], np.uint8)
        J = O.survivors(mask)
        d, scale = O.decode_weights(O.CR_REAL, n, c, J, B)
        alpha = O.decoding_coefficients(O.CR_REAL, n, c, J, d, B)
        P = O.placement(O.CR_REAL, n, c)
        got = {}
        for m, j in enumerate(J):
            for l in range(c):
                if P[j][l] == k:
                    got[(j, l)] = n * scale * alpha[m, k]
        assert sorted(got) == sorted((w, s) for w, s, _, _ in copies)
        for w, s, _, coef in copies:
            assert got[(w, s)] == pytest.approx(coef, abs=1e-12)
        assert sum(got.values()) == pytest.approx(1.0, abs=1e-12)       # the coefficients sum to 1
        # At a step t that evaluates the second slot, W_0's copy of D_1 is fresh
        # and W_1's was evaluated at t - 1 (Sec. IV-A schedule, (t - 1) mod c).
        for t in (2, 4, 6):
            assert O.evaluated_slot(t, c) == 1
            for w, s, offset, _ in copies:
                terms = {slot: (part, tau) for slot, part, tau in O.coded_terms(O.CR_REAL, n, c, w, t)}
                assert terms[s] == (k, t + offset)
