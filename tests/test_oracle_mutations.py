"""Mutation check of the oracle's pins (CPU).

Each case plants one plausible mistake into the oracle (by replacing one of
its functions for the duration of the case) and runs the pins that should
notice it; at least one of them must fail.  The same pins pass on the
unchanged oracle.  This shows the pins of tests/test_oracle_pins.py pin the
oracle to the paper rather than to itself.  (The ReLU'(0) convention of the
MLP is not covered: it only matters on a set of measure zero.)
"""

import numpy as np
import pytest

from oracle import pgc_oracle as O

import test_oracle_pins as pins

ORIG = {name: getattr(O, name) for name in
        ("coded_terms", "decode_weights", "placement", "encoding_coefficients", "partition_gradient",
         "decode_step")}


def _coded_terms_slot_off_by_one(scheme, n, c, i, t, pipelined=True):
    P = ORIG["placement"](scheme, n, c)
    out = []
    for l in range(c):
        slot = (t - l) % c                                  # planted: (t - 1 - l) mod c
        tau = (t - l if t - l >= 1 else 0) if pipelined else t
        out.append((slot, P[i][slot], tau))
    return out


def _coded_terms_no_staleness(scheme, n, c, i, t, pipelined=True):
    return [(slot, k, t) for slot, k, _ in ORIG["coded_terms"](scheme, n, c, i, t, pipelined)]   # planted


def _decode_weights_wrong_mu(scheme, n, c, J, B=None, tol=1e-9):
    d, scale = ORIG["decode_weights"](scheme, n, c, J, B, tol)
    if scheme == O.CR:
        scale = 1.0 / (n * c)                               # planted: mu = c instead of |J| c / n
    return d, scale


def _decode_weights_last_representative(scheme, n, c, J, B=None, tol=1e-9):
    d, scale = ORIG["decode_weights"](scheme, n, c, J, B, tol)
    if scheme == O.FR:
        J = list(J)
        d = np.zeros(len(J))
        for group in range(n // c):
            members = [m for m, j in enumerate(J) if j // c == group]
            d[members[-1]] = 1.0                            # planted: highest-index survivor
    return d, scale


def _placement_reversed_cycle(scheme, n, c):
    if scheme in (O.CR, O.CR_REAL):
        return [[(i - l) % n for l in range(c)] for i in range(n)]   # planted: (i + l) mod n
    return ORIG["placement"](scheme, n, c)


def _encoding_transposed(scheme, n, c, B=None):
    if scheme == O.CR_REAL:
        return [[float(B[(i + l) % n, i]) for l in range(c)] for i in range(n)]   # planted: B^T
    return ORIG["encoding_coefficients"](scheme, n, c, B)


def _gradient_sum_not_mean(model, Xk, yk, beta, shape=None):
    g = ORIG["partition_gradient"](model, Xk, yk, beta, shape)
    return g * Xk.shape[0] if model in (O.LOGISTIC, O.LSQ) else g   # planted: no 1/m


def _gradient_sign_flipped(model, Xk, yk, beta, shape=None):
    g = ORIG["partition_gradient"](model, Xk, yk, beta, shape)
    return -g if model == O.LOGISTIC else g                 # planted: y - sigmoid(z)


def _gradient_mlp_unscaled(model, Xk, yk, beta, shape=None):
    g = ORIG["partition_gradient"](model, Xk, yk, beta, shape)
    return g * Xk.shape[0] if model == O.MLP else g         # planted: dZ2 not divided by m


def _decode_step_ascent(*args, **kw):
    coded, stale, J, d, scale, ghat = ORIG["decode_step"](*args, **kw)
    return coded, stale, J, d, scale, -ghat                 # planted: beta + eta * ghat


MUTANTS = {
    "slot index": ("coded_terms", _coded_terms_slot_off_by_one, [
        (pins.test_copies_are_at_most_c_minus_1_steps_stale, (O.CR, 7, 3)),
        (pins.test_coded_gradients_equal_per_worker_rings, (O.CR, O.LSQ, 5, 3)),
        (pins.test_naive_cr_matches_the_printed_n4_c2_example, ())]),
    "staleness": ("coded_terms", _coded_terms_no_staleness, [
        (pins.test_copies_are_at_most_c_minus_1_steps_stale, (O.FR, 8, 4)),
        (pins.test_cr_full_sum_identity_eq1, (5, 2))]),
    "mu": ("decode_weights", _decode_weights_wrong_mu, [
        (pins.test_cr_decoder_is_unbiased_eq2, (5, 2)),
        (pins.test_cr_decoder_is_unbiased_eq2, (7, 3))]),
    "FR representative": ("decode_weights", _decode_weights_last_representative, [
        (pins.test_fr_decode_picks_one_per_group_and_ignores_which, (6, 3)),
        (pins.test_decoder_rejects_too_many_stragglers, ())]),
    "placement": ("placement", _placement_reversed_cycle, [
        (pins.test_cr_every_partition_has_c_holders, (O.CR, 7, 3)),
        (pins.test_naive_cr_matches_the_printed_n4_c2_example, ())]),
    "transposed B": ("encoding_coefficients", _encoding_transposed, [
        (pins.test_real_code_decodes_exactly_for_every_admissible_set, (5, 2)),
        (pins.test_real_code_decodes_exactly_for_every_admissible_set, (8, 3)),
        (pins.test_naive_cr_matches_the_printed_n4_c2_example, ())]),
    "1/m": ("partition_gradient", _gradient_sum_not_mean, [
        (pins.test_linear_gradients_match_finite_differences, (O.LSQ,)),
        (pins.test_c1_is_full_batch_gradient_descent, (O.CR, O.LSQ))]),
    "sign": ("partition_gradient", _gradient_sign_flipped, [
        (pins.test_linear_gradients_match_finite_differences, (O.LOGISTIC,)),
        (pins.test_fr_warmup_is_exact_gradient_coding, (4, 2))]),
    "MLP scale": ("partition_gradient", _gradient_mlp_unscaled, [
        (pins.test_mlp_gradient_matches_finite_differences, ())]),
    "update direction": ("decode_step", _decode_step_ascent, [
        (pins.test_c1_is_full_batch_gradient_descent, (O.FR, O.LOGISTIC)),
        (pins.test_lsq_c1_matches_closed_form_gradient, ())]),
}


def _failures(cases):
    failed = []
    for pin, args in cases:
        try:
            pin(*args)
        except Exception as e:   # an assertion, or an error the mistake provokes
            failed.append((pin.__name__, type(e).__name__))
    return failed


@pytest.mark.parametrize("name", list(MUTANTS))
def test_the_pins_catch_a_planted_mistake(name, monkeypatch):
    attr, mutant, cases = MUTANTS[name]
    assert _failures(cases) == [], "the pins must pass on the unchanged oracle"
    monkeypatch.setattr(O, attr, mutant)
    failed = _failures(cases)
    assert failed, "no pin noticed the planted mistake %r" % name
    # Every pin listed for a mistake notices it.
    assert len(failed) == len(cases), failed
