"""Host logic of the comparison studies (no GPU): the decoding coefficients
they report, their accounting of work per step and the simulated clock."""

import itertools
import math

import numpy as np
import pytest

import paper_2607_20739_amd as P
import studies
from oracle import pgc_oracle as O
from oracle import rng as R

NAMES = {"FR": O.FR, "CR": O.CR, "CR_REAL": O.CR_REAL}


@pytest.mark.parametrize("scheme,n,c", [("CR_REAL", 12, 6), ("CR_REAL", 8, 3), ("CR", 12, 6), ("FR", 12, 6)])
def test_study_alpha_matches_the_oracle_decoding_coefficients(scheme, n, c):
    """alpha[m, k] = d_m c_{j_m, l} (Sec. V-A), scaled by n * scale so that an exact
    decoder's coefficients of each partition sum to one."""
    ctx = P.pgc_init(scheme, n, c, 8)
    P.pgc_configure(ctx, "logistic", n * 4, 8, code_seed=12)
    try:
        B = P.pgc_encoding_matrix(ctx, n)
        B_or = O.cyclic_encoding_matrix(n, c, R.null_space_generator(12, c - 1, n)) if scheme == "CR_REAL" else None
        for t in range(30):
            mask = R.straggler_mask(5, t, R.POLICY_SLOWEST, n, c - 1)
            alpha, surv = studies.decoding_alpha(ctx, n, c, mask, B)
            J = O.survivors(mask)
            d_or, scale_or = O.decode_weights(NAMES[scheme], n, c, J, B_or)
            a_or = n * scale_or * O.decoding_coefficients(NAMES[scheme], n, c, J, d_or, B_or)
            held = ~np.isnan(alpha)
            assert surv.tolist() == J
            assert held.sum(axis=1).tolist() == [c] * len(J)
            np.testing.assert_allclose(alpha[held], a_or[held], rtol=1e-9,
                                       atol=1e-9 * np.abs(a_or).max())
            assert np.all(a_or[~held] == 0.0)
            if scheme != "CR":
                np.testing.assert_allclose(np.nansum(alpha, axis=0), 1.0, atol=1e-8 * np.abs(a_or).max())
            else:
                mu = (n - (c - 1)) * c / n
                np.testing.assert_allclose(alpha[held], 1.0 / mu, rtol=1e-15)
    finally:
        P.pgc_destroy(ctx)


def test_naive_cr_coefficients_grow_large_at_n12_c6():
    """Sec. V-A: with n = 12, c = 6 some straggler patterns need decoding
    coefficients in the thousands; PGC-CR's stay below 2 (1 / mu < 2)."""
    n, c = 12, 6
    ctx = P.pgc_init("CR_REAL", n, c, 8)
    P.pgc_configure(ctx, "logistic", n * 4, 8, code_seed=12)
    try:
        B = P.pgc_encoding_matrix(ctx, n)
        worst = 0.0
        for strag in itertools.combinations(range(n), c - 1):
            mask = np.zeros(n, np.uint8)
            mask[list(strag)] = 1
            alpha, _ = studies.decoding_alpha(ctx, n, c, mask, B)
            worst = max(worst, float(np.nanmax(np.abs(alpha))))
        assert worst > 1000.0
    finally:
        P.pgc_destroy(ctx)


def test_work_accounting():
    # PGC evaluates one partition per worker after the warm-up; GC all c.
    assert studies.worker_partitions("PGC-CR", 3, 0) == 4
    assert studies.worker_partitions("PGC-CR", 3, 5) == 1
    assert studies.worker_partitions("GC-CR", 3, 5) == 4
    assert studies.worker_partitions("DGD", 3, 5) == 1
    N = 12 * 64
    assert studies.rows_streamed("PGC-FR", 2, N) == N // 3
    assert studies.rows_streamed("GC-FR", 2, N) == N
    assert studies.rows_streamed("PGC-CR", 2, N) == N
    assert studies.rows_streamed("GC-CR", 2, N) == N
    assert studies.worker_rows("GC-CR", 2, 64) == 3 * 64
    assert studies.worker_rows("PGC-CR", 2, 64) == 64
    assert studies.scheme_setup("DGD", 3) == ("FR", 1, True, 0)
    assert studies.scheme_setup("IS-SGD", 3) == ("IS_SGD", 1, True, 3)


def test_simulated_step_times_follow_the_order_statistics():
    """Mean step time = compute + mu * sum_{j < n - s} 1 / (n - j) for the
    (n - s)-th of n exponential delays; DGD waits for the slowest."""
    n, T, mean = 12, 3000, 1.0
    for name, s in [("DGD", 2), ("PGC-CR", 2), ("GC-FR", 2), ("IS-SGD", 3)]:
        _, _, _, s_tol = studies.scheme_setup(name, s)
        _, secs = studies.delay_masks(n, s_tol, T + 1, 99, mean, 1.0, name, s)
        k = n - s_tol
        compute = studies.worker_partitions(name, s, 1)
        expect = compute + mean * sum(1.0 / (n - j) for j in range(k))
        sd = mean * math.sqrt(sum(1.0 / (n - j) ** 2 for j in range(k)))
        assert abs(np.mean(secs[1:]) - expect) < 5 * sd / math.sqrt(T)
