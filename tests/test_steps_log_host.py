"""Host checks of the per-step error tooling: the oracle's teacher-forced decode
and tests/steps_log_errors.py on a log written from known vectors.  No GPU."""

import json
import os
import sys

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

from oracle import pgc_oracle as O  # noqa: E402
from oracle import rng as R  # noqa: E402
from workloads import Workload, make_inputs, POLICY_UNIFORM_COUNT  # noqa: E402

import steps_log_errors  # noqa: E402


def _case(scheme, n, c, model="lsq", d=12, m=20, seed=3):
    rng = np.random.default_rng(seed)
    X = rng.normal(size=(n * m, d))
    y = rng.normal(size=n * m) if model == "lsq" else (rng.random(n * m) < 0.5).astype(np.float64)
    B = O.cyclic_encoding_matrix(n, c, R.null_space_generator(seed, c - 1, n)) if scheme == O.CR_REAL else None
    masks = [R.straggler_mask(seed, t, POLICY_UNIFORM_COUNT, n, c - 1) for t in range(3 * c + 2)]
    return X, y, B, masks


@pytest.mark.parametrize("scheme,n,c", [(O.FR, 6, 3), (O.CR, 7, 3), (O.CR_REAL, 8, 3), (O.CR, 5, 1)])
@pytest.mark.parametrize("pipelined", [True, False])
def test_teacher_forced_decode_at_the_oracles_own_iterates_is_its_decode(scheme, n, c, pipelined):
    """Fed the oracle's own trajectory, the teacher-forced decode of every step
    is the decoded gradient run() used, bit for bit."""
    X, y, B, masks = _case(scheme, n, c)
    beta0 = np.zeros(X.shape[1])
    recs = O.run(scheme, "lsq", n, c, X, y, beta0, 0.05, masks, B=B, pipelined=pipelined)
    iterates = {0: beta0}
    for t, r in enumerate(recs):
        tf = O.teacher_forced_ghat(scheme, "lsq", n, c, X, y, iterates, t, masks[t], B=B, pipelined=pipelined)
        assert np.array_equal(tf, r.ghat), t
        iterates[t + 1] = r.beta


def test_teacher_forced_decode_uses_the_given_iterates():
    """Perturbing the iterate of one step changes exactly the decodes whose
    copies were evaluated there: steps t .. t + c - 1 for PGC-CR."""
    n, c = 6, 3
    X, y, B, masks = _case(O.CR, n, c, model="logistic")
    beta0 = np.zeros(X.shape[1])
    recs = O.run(O.CR, "logistic", n, c, X, y, beta0, 0.3, masks)
    iterates = {0: beta0}
    for t, r in enumerate(recs):
        iterates[t + 1] = r.beta
    bumped = dict(iterates)
    bumped[4] = iterates[4] + 0.01
    for t in range(len(recs)):
        same = np.array_equal(O.teacher_forced_ghat(O.CR, "logistic", n, c, X, y, bumped, t, masks[t]), recs[t].ghat)
        assert same == (not 4 <= t < 4 + c), t


def test_steps_log_errors_reports_the_rounding_of_known_vectors(tmp_path):
    """A log whose vectors are the oracle's own, rounded to fp32, shows errors
    at the level of fp32 rounding; a planted error in one step shows there."""
    w = Workload("log_check", "CR", "logistic", n=4, c=2, N=4 * 64, d=16, lr=0.2, steps=6,
                 policy=POLICY_UNIFORM_COUNT, cap=1, seed=7)
    X, y, beta0 = make_inputs(w)
    masks = [R.straggler_mask(w.mask_seed, t, w.policy, w.n, w.cap, w.p) for t in range(w.steps)]
    ref = O.run(O.CR, w.model, w.n, w.c, X.numpy(), y.numpy(), beta0.numpy(), w.lr, masks)
    ghat = np.stack([r.ghat for r in ref]).astype(np.float32)
    wv = np.stack([r.beta for r in ref]).astype(np.float32)
    ghat[3, 5] *= 1.01
    log = tmp_path / "steps.jsonl"
    with open(log, "w") as f:
        for t, m in enumerate(masks):
            f.write(json.dumps({"t": t, "stragglers": [int(i) for i in np.flatnonzero(m)]}) + "\n")
    np.savez(str(log) + ".npz", ghat=ghat, w=wv, workload=w.name, lr=w.lr, seed=w.seed)
    recs = steps_log_errors.annotate(str(log), w, X.numpy(), y.numpy(), beta0.numpy(), teacher_forced=True)
    for t, r in enumerate(recs):
        assert r["err_w"] < 1e-6
        if t == 3:
            assert r["err_ghat"] > 1e-3 and r["tf_err_ghat"] > 1e-3
        else:
            assert r["err_ghat"] < 1e-6 and r["tf_err_ghat"] < 1e-6
    with open(log) as f:
        assert [json.loads(line)["t"] for line in f] == list(range(w.steps))
