"""The C-ABI library on the host (no GPU): exports, host tables, error codes.

Host tables are compared with the oracle: placement, schedule, straggler masks
and surviving sets bit for bit; the real-valued code's matrix and decode
weights within 1e-12.  No device work is launched here.
"""

import itertools
import os
import re

import numpy as np
import pytest

import paper_2607_20739_amd as P
from oracle import pgc_oracle as O
from oracle import rng as R

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SCHEME_NAMES = {"FR": O.FR, "CR": O.CR, "CR_REAL": O.CR_REAL, "IS_SGD": O.IS_SGD}


def _declared_symbols():
    with open(os.path.join(ROOT, "include", "pgc.h")) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(pgc_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol():
    declared = _declared_symbols()
    assert len(declared) >= 20
    assert declared == sorted(P.exported_symbols())
    handle = P.lib()
    for name in declared:
        assert hasattr(handle, name), name


def _ctx(scheme, n, c, d=8, model="lsq", N=None, code_seed=0):
    ctx = P.pgc_init(scheme, n, c, d)
    P.pgc_configure(ctx, model, N if N is not None else n * 4, d, code_seed=code_seed)
    return ctx


CASES = [("FR", 4, 2), ("FR", 32, 4), ("FR", 6, 6), ("FR", 5, 1), ("CR", 8, 3), ("CR", 64, 4),
         ("CR", 128, 8), ("CR", 7, 7), ("CR_REAL", 8, 3), ("CR_REAL", 12, 6), ("CR_REAL", 4, 2),
         ("CR_REAL", 5, 1), ("IS_SGD", 12, 1), ("IS_SGD", 1, 1)]


@pytest.mark.parametrize("scheme,n,c", CASES)
def test_placement_and_schedule_match_the_oracle(scheme, n, c):
    ctx = _ctx(scheme, n, c)
    try:
        P_or = O.placement(SCHEME_NAMES[scheme], n, c)
        assert P.pgc_placement(ctx, n, c).tolist() == P_or
        for t in range(1, 3 * c + 2):
            expect = [P_or[i][O.evaluated_slot(t, c)] for i in range(n)]
            assert P.pgc_schedule(ctx, t, n).tolist() == expect
        assert P.pgc_num_coded(ctx) == (n // c if scheme == "FR" else n)
        with pytest.raises(P.PGCError):
            P.pgc_schedule(ctx, 0, n)
    finally:
        P.pgc_destroy(ctx)


def test_splitmix64_matches_the_oracle():
    for seed in [0, 1, 1234567, (5 << 32) | 1, 2 ** 64 - 1]:
        for index in [0, 1, 2, 77, 2 ** 32 + 3, 2 ** 40]:
            assert P.pgc_splitmix64(seed, index) == R.splitmix64(seed, index)


@pytest.mark.parametrize("policy,n,cap,p", [
    (R.POLICY_EXACT, 4, 1, 0.0), (R.POLICY_UNIFORM_COUNT, 8, 2, 0.0), (R.POLICY_BERNOULLI, 32, 3, 0.05),
    (R.POLICY_BERNOULLI, 64, 3, 0.05), (R.POLICY_BERNOULLI, 128, 7, 0.04), (R.POLICY_BERNOULLI, 16, 2, 0.5),
    (R.POLICY_EXACT, 256, 255, 0.0), (R.POLICY_UNIFORM_COUNT, 1, 0, 0.0), (R.POLICY_SLOWEST, 12, 3, 0.0),
    (R.POLICY_SLOWEST, 256, 17, 0.0), (R.POLICY_SLOWEST, 5, 0, 0.0)])
def test_masks_match_the_oracle_bit_for_bit(policy, n, cap, p):
    for seed in [(1 << 32) | 1, (5 << 32) | 1, 99]:
        for t in range(60):
            a = P.pgc_make_mask(seed, t, policy, n, cap, p)
            b = R.straggler_mask(seed, t, policy, n, cap, p)
            assert a.tolist() == b.tolist(), (seed, t)


@pytest.mark.parametrize("n,s,mean,compute", [(12, 1, 1.0, 1.0), (12, 3, 2.0, 4.0), (12, 0, 1.0, 1.0),
                                               (256, 7, 0.5, 0.0), (1, 0, 1.0, 0.0), (8, 7, 0.0, 2.0)])
def test_delay_steps_match_the_oracle(n, s, mean, compute):
    for seed in [(2 << 32) | 1, 31]:
        for t in range(40):
            mask, delays, sec = P.pgc_delay_step(seed, t, n, s, mean, compute)
            m_or, d_or, sec_or = R.delay_step(seed, t, n, s, mean, compute)
            assert mask.tolist() == m_or.tolist()
            np.testing.assert_allclose(delays, d_or, rtol=1e-15, atol=0.0)
            assert sec == pytest.approx(sec_or, rel=1e-15, abs=0.0)
            assert mask.tolist() == P.pgc_make_mask(seed, t, P.PGC_POLICY_SLOWEST, n, s).tolist()


def test_delay_step_rejects_bad_arguments():
    for args in [(1, 0, 4, 4, 1.0, 0.0), (1, 0, 4, -1, 1.0, 0.0), (1, -1, 4, 1, 1.0, 0.0),
                 (1, 0, 4, 1, -1.0, 0.0), (1, 0, 4, 1, float("nan"), 0.0), (1, 0, 4, 1, 1.0, -2.0),
                 (1, 0, 0, 0, 1.0, 0.0), (1, 0, 257, 1, 1.0, 0.0)]:
        with pytest.raises(P.PGCError) as e:
            P.pgc_delay_step(*args)
        assert e.value.status == P.PGC_EINVAL


@pytest.mark.parametrize("n,c,seed", [(4, 2, 1), (8, 3, 2), (12, 6, 3), (5, 1, 4), (16, 5, 9)])
def test_real_code_matrix_matches_the_oracle(n, c, seed):
    ctx = _ctx("CR_REAL", n, c, code_seed=seed)
    try:
        B = P.pgc_encoding_matrix(ctx, n)
        H = R.null_space_generator(seed, c - 1, n)
        B_or = O.cyclic_encoding_matrix(n, c, H)
        np.testing.assert_allclose(B, B_or, rtol=1e-12, atol=1e-12)
        assert np.array_equal(B != 0.0, B_or != 0.0)
    finally:
        P.pgc_destroy(ctx)


@pytest.mark.parametrize("scheme,n,c", [("FR", 6, 3), ("FR", 8, 2), ("CR", 7, 3), ("CR_REAL", 8, 3),
                                        ("CR_REAL", 6, 4), ("CR_REAL", 12, 6)])
def test_decode_coefficients_match_the_oracle_for_every_admissible_mask(scheme, n, c):
    ctx = _ctx(scheme, n, c, code_seed=5)
    try:
        B = P.pgc_encoding_matrix(ctx, n) if scheme == "CR_REAL" else None
        B_or = O.cyclic_encoding_matrix(n, c, R.null_space_generator(5, c - 1, n)) if B is not None else None
        for k in range(c):
            for strag in itertools.combinations(range(n), k):
                mask = np.zeros(n, np.uint8)
                mask[list(strag)] = 1
                surv, d, scale = P.pgc_decode_coeffs(ctx, mask, n)
                J = O.survivors(mask)
                d_or, scale_or = O.decode_weights(SCHEME_NAMES[scheme], n, c, J, B_or)
                assert surv.tolist() == J
                assert scale == pytest.approx(scale_or, rel=1e-15)
                np.testing.assert_allclose(d, d_or, rtol=1e-10, atol=1e-10 * max(1.0, np.abs(d_or).max()))
                if scheme != "CR_REAL":
                    assert d.tolist() == d_or.tolist()
    finally:
        P.pgc_destroy(ctx)


def test_is_sgd_decode_ignores_any_number_of_stragglers():
    n = 6
    ctx = _ctx("IS_SGD", n, 1)
    try:
        for k in range(n):
            for strag in itertools.combinations(range(n), k):
                mask = np.zeros(n, np.uint8)
                mask[list(strag)] = 1
                surv, d, scale = P.pgc_decode_coeffs(ctx, mask, n)
                d_or, scale_or = O.decode_weights(O.IS_SGD, n, 1, O.survivors(mask))
                assert surv.tolist() == O.survivors(mask)
                assert d.tolist() == d_or.tolist() and scale == scale_or
        with pytest.raises(P.PGCError) as e:
            P.pgc_decode_coeffs(ctx, np.ones(n, np.uint8), n)
        assert e.value.status == P.PGC_ESTRAGGLERS
    finally:
        P.pgc_destroy(ctx)
    with pytest.raises(P.PGCError):
        P.pgc_init("IS_SGD", 6, 2, 8)        # IS-SGD holds one partition per worker


def test_binding_constants_match_header():
    """Every numeric #define of include/pgc.h that the binding mirrors has the same value."""
    with open(os.path.join(ROOT, "include", "pgc.h")) as f:
        header = f.read()
    defines = {}
    for name, expr in re.findall(r"^#define (PGC_\w+)\s+(\(?[0-9u <]+\)?)", header, re.M):
        parts = expr.strip("() ").replace("u", "").split("<<")   # "N" or "(Nu << K)"
        defines[name] = int(parts[0]) << (int(parts[1]) if len(parts) > 1 else 0)
    mirrored = [k for k in defines if hasattr(P, k)]
    assert {"PGC_MAX_N", "PGC_NOALLOC_SCRATCH_BYTES", "PGC_MLP_MAX_D_IN"} <= set(mirrored)
    for k in mirrored:
        assert getattr(P, k) == defines[k], k


def _mlp_d(d_in, hidden, classes):
    return d_in * hidden + hidden + hidden * classes + classes


def test_mlp_shape_limits():
    """pgc_configure accepts the MLP shapes include/pgc.h allows and rejects the others."""
    cases = [(64, 256, 10, True), (8, 1024, 16, True), (P.PGC_MLP_MAX_D_IN, 256, 10, True),
             (P.PGC_MLP_MAX_D_IN + 8, 256, 10, False),   # past the forward's 32-bit tile offsets
             (60, 256, 10, False), (0, 256, 10, False),   # d_in % 8, d_in >= 8
             (64, 384, 10, False), (64, 2048, 10, False),  # hidden % 256, hidden <= 1024
             (64, 256, 0, False), (64, 256, 17, False)]    # 1 <= classes <= 16
    for d_in, hidden, classes, ok in cases:
        ctx = P.pgc_init("CR", 4, 2, _mlp_d(d_in, hidden, classes))
        try:
            if ok:
                P.pgc_configure(ctx, "mlp", 4 * 64, d_in, hidden, classes)
                assert P.pgc_workspace_bytes(ctx) > 0
            else:
                with pytest.raises(P.PGCError) as e:
                    P.pgc_configure(ctx, "mlp", 4 * 64, d_in, hidden, classes)
                assert e.value.status == P.PGC_EINVAL, (d_in, hidden, classes)
        finally:
            P.pgc_destroy(ctx)
    ctx = P.pgc_init("CR", 4, 2, _mlp_d(64, 256, 10) + 1)   # d must match the shape
    try:
        with pytest.raises(P.PGCError) as e:
            P.pgc_configure(ctx, "mlp", 4 * 64, 64, 256, 10)
        assert e.value.status == P.PGC_EINVAL
    finally:
        P.pgc_destroy(ctx)


def test_error_codes():
    with pytest.raises(P.PGCError) as e:
        P.pgc_init("FR", 6, 4, 8)                      # c does not divide n
    assert e.value.status == P.PGC_EINVAL
    for args in [("CR", 0, 1, 8), ("CR", 4, 5, 8), ("CR", 300, 2, 8), ("CR", 4, 2, 0), (7, 4, 2, 8)]:
        with pytest.raises(P.PGCError):
            P.pgc_init(*args)
    ctx = P.pgc_init("CR", 8, 3, 16)
    try:
        with pytest.raises(P.PGCError) as e:
            P.pgc_workspace_bytes(ctx)                 # not configured
        assert e.value.status == P.PGC_ESTATE
        for bad in [dict(model="lsq", N=12, d_in=16), dict(model="lsq", N=0, d_in=16),
                    dict(model="lsq", N=16, d_in=15), dict(model=9, N=16, d_in=16)]:
            with pytest.raises(P.PGCError) as e:
                P.pgc_configure(ctx, **bad)
            assert e.value.status == P.PGC_EINVAL
        P.pgc_configure(ctx, "lsq", 64, 16)
        mask = np.zeros(8, np.uint8)
        mask[:3] = 1                                    # three stragglers > s = 2
        with pytest.raises(P.PGCError) as e:
            P.pgc_decode_coeffs(ctx, mask, 8)
        assert e.value.status == P.PGC_ESTRAGGLERS
        with pytest.raises(P.PGCError) as e:
            P.pgc_step(ctx, 1, 1, 1, np.zeros(8, np.uint8), 0.1, 8)   # no workspace bound
        assert e.value.status == P.PGC_ESTATE
        assert P.pgc_get_step(ctx) == 0
        assert "workspace" in P.pgc_last_error(ctx)
    finally:
        P.pgc_destroy(ctx)
    assert P.pgc_strerror(P.PGC_ESTRAGGLERS)


def test_workspace_size_covers_ring_coded_and_partials():
    for scheme, n, c, d, N in [("FR", 4, 2, 64, 4096), ("CR_REAL", 8, 3, 1024, 262144),
                               ("FR", 32, 4, 4096, 1048576), ("CR", 128, 8, 8192, 2097152)]:
        ctx = _ctx(scheme, n, c, d=d, N=N, model="logistic" if scheme != "CR_REAL" else "lsq")
        try:
            planes = 1 if scheme == "FR" else c
            coded = n // c if scheme == "FR" else n
            need = 4 * d * (planes * n + coded + 1)
            assert P.pgc_workspace_bytes(ctx) >= need
            assert P.pgc_workspace_bytes(ctx) % 256 == 0
        finally:
            P.pgc_destroy(ctx)


def test_state_size_is_the_header_and_the_ring():
    """A saved state holds a 256-byte header and every ring slot (c planes for
    CR, one for FR), slots padded to a multiple of 256 floats."""
    for scheme, n, c, d, model in [("FR", 4, 2, 64, "logistic"), ("CR_REAL", 8, 3, 1000, "lsq"),
                                   ("CR", 16, 4, 300, "logistic"), ("IS_SGD", 5, 1, 8, "lsq")]:
        ctx = _ctx(scheme, n, c, d=d, N=n * 8, model=model)
        try:
            planes = 1 if scheme in ("FR", "IS_SGD") else c
            ld = -(-d // 256) * 256
            assert P.pgc_state_bytes(ctx) == 256 + 4 * planes * n * ld
            # Saving and loading need the ring, i.e. a bound workspace.
            for call in (P.pgc_save_state, P.pgc_load_state):
                with pytest.raises(P.PGCError) as e:
                    call(ctx, 1 << 20, 1 << 30)
                assert e.value.status == P.PGC_ESTATE
        finally:
            P.pgc_destroy(ctx)
    ctx = P.pgc_init("CR", 8, 3, 16)
    try:
        with pytest.raises(P.PGCError) as e:
            P.pgc_state_bytes(ctx)                     # not configured
        assert e.value.status == P.PGC_ESTATE
    finally:
        P.pgc_destroy(ctx)


def test_noalloc_step_rejects_on_the_host_before_any_device_work():
    """pgc_step_noalloc's argument checks run before it touches a GPU: an
    unconfigured context, the MLP, a shape whose block partial sums exceed the
    fixed array, and a missing workspace are all rejected on the host."""
    mask = np.zeros(4, np.uint8)
    ctx = P.pgc_init("CR", 4, 2, 64)
    try:
        with pytest.raises(P.PGCError) as e:
            P.pgc_step_noalloc(ctx, 1, 1, 1, mask, 0.1, 4)
        assert e.value.status == P.PGC_ESTATE
        P.pgc_configure(ctx, "lsq", 4 * 4096, 64)
        with pytest.raises(P.PGCError) as e:
            P.pgc_step_noalloc(ctx, 1, 1, 1, mask, 0.1, 4)    # fits, but nothing is bound
        assert e.value.status == P.PGC_ESTATE and "workspace" in P.pgc_last_error(ctx)
    finally:
        P.pgc_destroy(ctx)
    q = 64 * 256 + 256 + 256 * 10 + 10
    ctx = P.pgc_init("CR", 4, 2, q)
    try:
        P.pgc_configure(ctx, "mlp", 4 * 64, 64, 256, 10)
        with pytest.raises(P.PGCError) as e:
            P.pgc_step_noalloc(ctx, 1, 1, 1, mask, 0.1, 4)
        assert e.value.status == P.PGC_EINVAL and "linear" in P.pgc_last_error(ctx)
    finally:
        P.pgc_destroy(ctx)
    # d = 32768 on 512 gradient blocks of 128 KiB of partial sums each: 64 MiB, over the limit.
    ctx = P.pgc_init("CR", 4, 2, 32768)
    try:
        P.pgc_configure(ctx, "lsq", 4 * 2048, 32768)
        with pytest.raises(P.PGCError) as e:
            P.pgc_step_noalloc(ctx, 1, 1, 1, mask, 0.1, 4)
        assert e.value.status == P.PGC_EINVAL and "scratch" in P.pgc_last_error(ctx)
        assert P.pgc_get_step(ctx) == 0
    finally:
        P.pgc_destroy(ctx)


def _random_admissible_case(data):
    from hypothesis import strategies as st
    scheme = data.draw(st.sampled_from(["FR", "CR", "CR_REAL", "IS_SGD"]), label="scheme")
    if scheme == "FR":
        c = data.draw(st.integers(1, 8), label="c")
        n = c * data.draw(st.integers(1, 256 // c), label="groups")
    elif scheme == "CR":
        n = data.draw(st.integers(1, 256), label="n")
        c = data.draw(st.integers(1, min(n, 8)), label="c")
    elif scheme == "CR_REAL":
        n = data.draw(st.integers(2, 16), label="n")
        c = data.draw(st.integers(1, min(n, 4)), label="c")
    else:
        n, c = data.draw(st.integers(1, 256), label="n"), 1
    cap = n - 1 if scheme == "IS_SGD" else c - 1
    k = data.draw(st.integers(0, cap), label="stragglers")
    strag = data.draw(st.lists(st.integers(0, n - 1), min_size=k, max_size=k, unique=True), label="who")
    mask = np.zeros(n, np.uint8)
    mask[strag] = 1
    return scheme, n, c, mask


def test_decode_coefficients_match_the_oracle_on_random_cases():
    """Random schemes, sizes up to n = 256 and admissible straggler sets: the
    library's survivors, decode weights and scale equal the oracle's (bit for
    bit except the real code's least-squares weights)."""
    from hypothesis import given, settings, strategies as st

    @settings(max_examples=300, deadline=None, derandomize=True)
    @given(st.data())
    def check(data):
        scheme, n, c, mask = _random_admissible_case(data)
        ctx = _ctx(scheme, n, c, code_seed=11)
        try:
            B_or = (O.cyclic_encoding_matrix(n, c, R.null_space_generator(11, c - 1, n))
                    if scheme == "CR_REAL" else None)
            surv, d, scale = P.pgc_decode_coeffs(ctx, mask, n)
            J = O.survivors(mask)
            d_or, scale_or = O.decode_weights(SCHEME_NAMES[scheme], n, c, J, B_or)
            assert surv.tolist() == J
            if scheme == "CR_REAL":
                assert scale == pytest.approx(scale_or, rel=1e-15)
                np.testing.assert_allclose(d, d_or, rtol=1e-9, atol=1e-9 * max(1.0, np.abs(d_or).max()))
            else:
                assert scale == scale_or and d.tolist() == d_or.tolist()
        finally:
            P.pgc_destroy(ctx)
    check()
