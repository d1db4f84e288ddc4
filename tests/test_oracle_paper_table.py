"""Oracle pinned to numbers the paper prints.

* Eq. (6) with the per-operator w_i and S_i of Appendix A (tab:app-ops)
  reproduces the printed S_agg of section 4.2 (tab:main-xpu-a) for both
  leading candidates, within the rounding of the printed inputs.
* The printed top-5 / top-10 cumulative shares follow from the printed w_i.
* Statistical check: a trace whose operators are drawn with probability w_i
  (key independent of duration, app and phase) recovers w_i through
  Eq. (2)-(3) within sampling error.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import oracle as O

TABLE = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "app_ops_table.json")))
ROWS = TABLE["rows"]


def _trace_with_weights():
    """One app, one phase, one invocation per operator with duration w_i in
    units of 0.1 percent, so that Eq. (3) gives exactly the printed w_i."""
    dur = [int(round(r[1] * 10)) for r in ROWS]
    assert sum(dur) == 1000
    key = [(i + 1) << 16 for i in range(len(ROWS))]
    return key, [0] * len(ROWS), [0] * len(ROWS), dur


@pytest.mark.parametrize("col,name", [(3, "S_opus"), (4, "S_gpt")])
def test_s_agg_matches_printed(col, name):
    key, app, ph, dur = _trace_with_weights()
    # printed 0.00 means a value in (0, 0.005): take the midpoint; '--' = not correct
    S = [math.nan if r[col] is None else (0.0025 if r[col] == 0 else r[col]) for r in ROWS]
    res = O.run(key, app, ph, dur, [65536], 1, score_key=key, s=S)
    w = res["score_op_weight"]
    assert np.allclose(w, [r[1] / 100 for r in ROWS], rtol=1e-14, atol=0)
    # rounding bound: each w_i is +-0.0005, each S_i +-0.005, S_agg printed +-0.0005
    Ss = np.array([0 if math.isnan(x) else x for x in S])
    bound = 0.0005 * Ss.sum() + 0.005 * w.sum() + 0.0005
    assert abs(res["s_agg"] - TABLE["s_agg_printed"][name]) <= bound, (res["s_agg"], bound)


def test_top_k_shares_match_printed():
    key, app, ph, dur = _trace_with_weights()
    res = O.run(key, app, ph, dur, [65536], 1)
    w = np.sort(res["op_w"])[::-1]
    assert abs(w[:5].sum() - TABLE["top5_share_printed"]) <= 5 * 0.0005 + 0.0005
    assert abs(w[:10].sum() - TABLE["top10_share_printed"]) <= 10 * 0.0005 + 0.0005
    assert sum(r[2] for r in ROWS) == TABLE["num_shapes_printed"]


def test_statistical_recovery_of_printed_weights():
    rng = np.random.default_rng(5)
    n = 1 << 20
    w = np.array([r[1] for r in ROWS]) / 100.0
    w = w / w.sum()
    op = rng.choice(len(ROWS), size=n, p=w)
    shapes = np.array([r[2] for r in ROWS])
    shape = (rng.random(n) * shapes[op]).astype(np.uint32)
    key = ((op + 1).astype(np.uint32) << np.uint32(16)) | shape
    app = rng.integers(0, 20, n).astype(np.uint32)
    ph = rng.integers(0, 2, n).astype(np.uint8)
    dur = np.rint(np.exp(np.log(3e4) + 1.0 * rng.standard_normal(n))).astype(np.int64)
    c = np.rint(65536 * (1 + 999 * rng.random(20))).astype(np.uint32)
    res = O.run(key, app, ph, dur, c, 2)
    assert np.abs(res["op_w"] - w).max() < 0.005
