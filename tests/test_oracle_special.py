"""Oracle special cases that reduce to textbook results, and its status codes."""
import math

import numpy as np
import pandas as pd
import pytest

from oracle import oracle as O


def test_single_app_is_plain_time_share():
    """One application (p = 1): the per-phase weight is the key's share of the
    phase's device time -- a plain group-by sum (pandas)."""
    rng = np.random.default_rng(11)
    n = 50000
    key = (rng.integers(0, 20, n).astype(np.uint32) << np.uint32(16)) | rng.integers(0, 5, n).astype(np.uint32)
    ph = rng.integers(0, 3, n).astype(np.uint8)
    dur = rng.integers(0, 10 ** 7, n).astype(np.int64)
    r = O.run(key, np.zeros(n, np.uint32), ph, dur, [12345], 3)
    df = pd.DataFrame(dict(key=key, ph=ph, d=dur))
    g = df.groupby(["key", "ph"])["d"].sum()
    tot = df.groupby("ph")["d"].sum()
    share = np.array([g[(k, p)] / tot[p] for k, p in zip(r["key"], r["phase"])])
    assert np.allclose(r["weight"], share, rtol=1e-13, atol=0)


def test_equal_apps_equal_totals_is_plain_share():
    """Equal p_a and equal D_a^phi: the weighting reduces to the pooled share."""
    key = [1 << 16, 2 << 16, 1 << 16, 2 << 16]
    app = [0, 0, 1, 1]
    dur = [300, 700, 100, 900]
    r = O.run(key, app, [0, 0, 0, 0], dur, [7, 7], 1)
    assert np.allclose(r["weight"], [0.2, 0.8], rtol=1e-15)


def test_one_phase_reduces_to_per_phase_weight():
    rng = np.random.default_rng(3)
    n = 3000
    key = (rng.integers(1, 6, n).astype(np.uint32) << np.uint32(16)) | rng.integers(0, 4, n).astype(np.uint32)
    app = rng.integers(0, 9, n).astype(np.uint32)
    dur = rng.integers(1, 10 ** 6, n).astype(np.int64)
    c = rng.integers(1, 1000, 9).astype(np.uint32)
    r = O.run(key, app, np.zeros(n, np.uint8), dur, c, 1)
    per_op = pd.Series(r["weight"]).groupby(r["key"] >> 16).sum()
    assert np.allclose(r["op_w"], per_op.values, rtol=1e-14)


def test_single_key_per_phase_gets_weight_one():
    key = [5 << 16, 5 << 16, 9 << 16 | 2]
    r = O.run(key, [0, 1, 1], [0, 0, 1], [10, 20, 30], [1, 2], 2)
    assert list(r["weight"]) == [1.0, 1.0]


def test_operator_in_one_phase_takes_that_phase_share():
    # op 1 only in phase 0 (share 1/2 there), op 2 in both (1/2 and 1)
    key = [1 << 16, 2 << 16, 2 << 16]
    r = O.run(key, [0, 0, 0], [0, 0, 1], [50, 50, 80], [1], 2)
    # U_1 = L * 1/2, U_2 = L/2 * (1/2 + 1) -> w = (1/2)/(1/2 + 3/4) = 0.4
    assert np.allclose(r["op_w"], [0.4, 0.6], rtol=1e-15)


def test_all_equal_scores_give_that_score():
    rng = np.random.default_rng(8)
    n = 2000
    key = (rng.integers(0, 7, n).astype(np.uint32) << np.uint32(16)) | rng.integers(0, 3, n).astype(np.uint32)
    app = rng.integers(0, 4, n).astype(np.uint32)
    ph = rng.integers(0, 2, n).astype(np.uint8)
    dur = rng.integers(1, 10 ** 6, n).astype(np.int64)
    keys = np.unique(key)
    for s in (1.0, 0.37):
        r = O.run(key, app, ph, dur, [3, 5, 7, 11], 2, score_key=keys, s=np.full(keys.size, s))
        assert abs(r["s_agg"] - s) <= 4 * 2.0 ** -53


def test_median_odd_even_and_zero_for_no_correct_shape():
    key = [1 << 16 | 0, 1 << 16 | 1, 1 << 16 | 2, 2 << 16, 3 << 16]
    r = O.run(key, [0] * 5, [0] * 5, [10, 10, 10, 35, 35], [1], 1,
              score_key=[1 << 16 | 0, 1 << 16 | 1, 1 << 16 | 2, 2 << 16, 3 << 16, 3 << 16 | 9],
              s=[0.9, 0.1, 0.5, math.nan, 0.2, 0.4])
    assert list(r["score_op"]) == [1, 2, 3]
    assert list(r["score_op_S"]) == [0.5, 0.0, 0.30000000000000004]
    # a shape named in the score but absent from the trace still counts for the median
    w = r["score_op_weight"]
    assert np.allclose(w, [0.3, 0.35, 0.35], rtol=1e-15)
    assert abs(r["s_agg"] - (0.3 * 0.5 + 0.35 * 0.30000000000000004)) < 1e-16


def test_retention_renormalises_over_scored_operators():
    key = [1 << 16, 2 << 16, 3 << 16]
    r = O.run(key, [0] * 3, [0] * 3, [20, 30, 50], [1], 1, score_key=[1 << 16, 3 << 16], s=[1.0, 0.5])
    assert np.allclose(r["score_op_weight"], [20 / 70, 50 / 70], rtol=1e-15)
    # a retained operator absent from the trace gets weight 0
    r = O.run(key, [0] * 3, [0] * 3, [20, 30, 50], [1], 1, score_key=[1 << 16, 9 << 16], s=[1.0, 0.5])
    assert list(r["score_op"]) == [1, 9] and r["score_op_weight"][1] == 0.0


ok_ev = dict(key=[1 << 16], app=[0], phase=[0], dur_ns=[5])


@pytest.mark.parametrize("P,c,ev,status", [
    (0, [1], ok_ev, O.E_INVALID_ARG),
    (9, [1], ok_ev, O.E_INVALID_ARG),
    (2, [], ok_ev, O.E_INVALID_ARG),
    (2, [0, 0], ok_ev, O.E_INVALID_ARG),
    (2, [1], dict(key=[1], app=[1], phase=[0], dur_ns=[5]), O.E_OUT_OF_RANGE),
    (2, [1], dict(key=[1], app=[0], phase=[2], dur_ns=[5]), O.E_OUT_OF_RANGE),
    (2, [1], dict(key=[1], app=[0], phase=[0], dur_ns=[-1]), O.E_OUT_OF_RANGE),
])
def test_status_codes_events(P, c, ev, status):
    assert O.status_of(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P) == status


@pytest.mark.parametrize("sk,s,status", [
    ([1 << 16], [1.5], O.E_OUT_OF_RANGE),
    ([1 << 16], [0.0], O.E_OUT_OF_RANGE),
    ([1 << 16], [-0.5], O.E_OUT_OF_RANGE),
    ([1 << 16], [math.inf], O.E_OUT_OF_RANGE),
    ([1 << 16, 1 << 16], [0.5, 0.5], O.E_INVALID_ARG),
    ([7 << 16], [0.5], O.E_INVALID_ARG),      # retained operator has no time at all
    ([], [], O.E_INVALID_ARG),
    ([1 << 16], [math.nan], O.OK),
    ([1 << 16], [1.0], O.OK),
])
def test_status_codes_score(sk, s, status):
    assert O.status_of([1 << 16], [0], [0], [5], [1], 1, score_key=sk, s=s) == status
