"""The step on a side stream and under HIP graph capture (GPU).

A session launches on whatever stream it is given, so a step can be recorded
into a HIP graph and replayed.  The schedule of Sec. IV-A / V-B repeats with
period c (slot (t-1) mod c at step t >= 1), so a graph holding c consecutive
steps t = 1..c replays exactly the next c steps of an eager run whose masks
repeat with the same period.  Every replay is compared bit for bit with that
eager run, with eager work and synchronisations between the replays.
"""

import numpy as np
import pytest
import torch

import paper_2607_20739_amd as P
from workloads import Workload, make_inputs, POLICY_EXACT

pytestmark = pytest.mark.gpu


def _announce(what):
    print("\n[gpu case] " + what, flush=True)


def _periodic_masks(w, periods):
    # Step 0 is the warm-up; steps 1.. repeat the masks of steps 1..c.
    base = [P.pgc_make_mask(w.mask_seed, t, w.policy, w.n, w.cap, w.p) for t in range(w.c + 1)]
    return [base[0]] + [base[1 + (t % w.c)] for t in range(w.c * periods)]


def _session(w):
    return P.PGCSession(w.scheme, w.n, w.c, w.model, w.N, w.d, hidden=w.hidden, classes=w.classes,
                        code_seed=w.code_seed)


CASES = [
    Workload("graph_crreal_lsq", "CR_REAL", "lsq", n=8, c=3, N=8 * 512, d=256, lr=0.02, steps=1,
             policy=POLICY_EXACT, cap=2, seed=61, code_seed=3),
    Workload("graph_fr_logistic", "FR", "logistic", n=8, c=4, N=8 * 300, d=1024, lr=0.05, steps=1,
             policy=POLICY_EXACT, cap=3, seed=62),
    Workload("graph_cr_mlp", "CR", "mlp", n=4, c=2, N=4 * 64, d=64, lr=0.05, steps=1,
             policy=POLICY_EXACT, cap=1, seed=63, hidden=256, classes=10),
]


@pytest.mark.parametrize("w", CASES, ids=[w.name for w in CASES])
def test_graph_replays_match_eager_steps(w):
    _announce(w.name)
    periods = 4
    X, y, beta0 = make_inputs(w, device="cuda")
    masks = _periodic_masks(w, periods)

    eager = _session(w)
    we = beta0.clone()
    traj = []
    for t, m in enumerate(masks):
        eager.step(X, y, we, m, w.lr)
        traj.append(we.clone())
    torch.cuda.synchronize()
    eager.close()

    sess = _session(w)
    wg = beta0.clone()
    sess.step(X, y, wg, masks[0], w.lr)            # warm-up t = 0, eager
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        sess.set_stream(torch.cuda.current_stream())
        for t in range(1, w.c + 1):               # records steps t = 1..c
            sess.step(X, y, wg, masks[t], w.lr)
    sess.set_stream(torch.cuda.current_stream())
    torch.cuda.synchronize()
    # Capture does not run the steps: wg still holds w after the warm-up.
    assert torch.equal(wg, traj[0])
    try:
        for r in range(periods):
            graph.replay()
            scratch = torch.randn(1 << 16, device="cuda")   # eager work between replays
            scratch.mul_(2.0).sum().item()
            torch.cuda.synchronize()
            expect = traj[(r + 1) * w.c]
            assert torch.equal(wg, expect), "replay %d differs from eager step %d" % (r, (r + 1) * w.c)
    finally:
        del graph
        sess.close()


def test_side_stream_matches_default_stream():
    w = CASES[0]
    _announce("side stream " + w.name)
    X, y, beta0 = make_inputs(w, device="cuda")
    masks = _periodic_masks(w, 2)
    a = _session(w)
    wa = beta0.clone()
    for m in masks:
        a.step(X, y, wa, m, w.lr)
    torch.cuda.synchronize()
    a.close()
    side = torch.cuda.Stream()                     # default priority
    side.wait_stream(torch.cuda.current_stream())
    b = _session(w)
    b.set_stream(side)
    wb = beta0.clone()
    with torch.cuda.stream(side):
        for m in masks:
            b.step(X, y, wb, m, w.lr)
    side.synchronize()
    torch.cuda.current_stream().wait_stream(side)
    b.close()
    assert torch.equal(wa, wb)


def test_switching_streams_mid_run_keeps_the_step_order():
    """Steps queued on one stream, then more steps after pgc_set_stream moves the
    session to another stream with no wait by the caller: the library orders
    the two streams itself, so the weights equal a single-stream run's bit for
    bit."""
    from workloads import WORKLOADS
    w = WORKLOADS["crreal_lsq_n8_c3_d1024"].resized(N=8 * 8192, steps=30)
    _announce("stream switch " + w.name)
    X, y, beta0 = make_inputs(w, device="cuda")
    masks = [P.pgc_make_mask(w.mask_seed, t, w.policy, w.n, w.cap, w.p) for t in range(w.steps)]
    ref = _session(w)
    wr = beta0.clone()
    for m in masks:
        ref.step(X, y, wr, m, w.lr)
    torch.cuda.synchronize()
    ref.close()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()     # default priority
    s1.wait_stream(torch.cuda.current_stream())
    sess = _session(w)
    ws = beta0.clone()
    try:
        sess.set_stream(s1)
        for m in masks[:20]:            # ~20 queued steps, nothing waited for
            sess.step(X, y, ws, m, w.lr)
        sess.set_stream(s2)
        for m in masks[20:]:
            sess.step(X, y, ws, m, w.lr)
        s2.synchronize()
        torch.cuda.current_stream().wait_stream(s2)
        assert torch.equal(ws, wr)
    finally:
        sess.close()
