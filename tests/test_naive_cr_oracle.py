"""The naive PGC-CR instability (Sec. V-A, Fig. 6) in the fp64 oracle, on the
data and straggler sets of the GPU study (n = 12, c = 6, the 5 slowest of 12
exponential delays dropped each step).  The naive code's loss leaves the basin
in fp64 as well, while PGC-FR and PGC-CR converge: the divergence comes from
stale copies weighted by large decoding coefficients, not from fp32 rounding.
CPU only (40 steps, 1,024 rows per partition)."""

import math
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

import naive_cr_oracle as NC  # noqa: E402


def test_naive_cr_diverges_in_fp64_while_pgc_fr_and_cr_converge():
    w, X, y, beta0 = NC.study_inputs(rows_per_partition=1024, d=256, lr=0.5, steps=40)
    masks = NC.study_masks(40)
    assert all(int(m.sum()) == 5 for m in masks)
    res = {name: NC.run_scheme(name, w, X, y, beta0, masks) for name in NC.SCHEMES}
    start = res["PGC-FR"][0][0]
    assert abs(start - math.log(2.0)) < 1e-12     # w(0) = 0: loss log 2
    for name in ("PGC-FR", "PGC-CR"):
        losses, amax, amin = res[name]
        assert max(losses) == losses[0] and losses[-1] < 0.95 * start, name
        assert max(amax) <= 1.0 + 1e-12 and min(amin) >= 0.0, name   # weights in [0, 1]
    losses, amax, amin = res["naive PGC-CR"]
    finite = [v for v in losses if math.isfinite(v)]
    assert max(finite) > 10.0 * start
    assert max(amax) > 1e3 and min(amin) < -1e3    # the large real coefficients of Sec. V-A
