"""Oracle pinned to the hand-worked trace (exact rationals from Eq. (2)-(6))."""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import brute_force as bf
from oracle import oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden", "tiny_trace.json")


@pytest.fixture(scope="module")
def case():
    g = json.load(open(GOLD))
    K = g["keys"]
    ev = g["events"]
    key = [K[e[0]] for e in ev]
    app = [e[1] for e in ev]
    ph = [e[2] for e in ev]
    dur = [e[3] for e in ev]
    sk = [K[k] for k in g["score"]["score_keys"]]
    s = [math.nan if x is None else x for x in g["score"]["S"]]
    r = O.run(key, app, ph, dur, g["app_weight_q16"], g["num_phases"], score_key=sk, s=s)
    return g, (key, app, ph, dur), r


def close(x, q, ulps=2):
    q = float(Fraction(q))
    return abs(x - q) <= ulps * math.ulp(max(abs(q), 1e-300))


def test_app_totals(case):
    g, _, r = case
    T = O.u128_to_int(r["app_total"])
    assert T == g["app_totals"]["index_a_times_P_plus_phase"]
    assert list(r["app_count"]) == g["app_totals"]["counts"]


def test_group_order_counts_and_weights(case):
    g, _, r = case
    K = g["keys"]
    rows = g["group_weights"]["rows"]
    assert list(r["key"]) == [K[row[0]] for row in rows]
    assert list(r["phase"]) == [row[1] for row in rows]
    assert list(r["count"]) == [row[4] for row in rows]
    for w, row in zip(r["weight"], rows):
        assert close(w, row[2]), (w, row)
    # each phase sums to one
    for ph in range(g["num_phases"]):
        assert abs(r["weight"][r["phase"] == ph].sum() - 1.0) < 1e-15


def test_op_and_key_weights(case):
    g, _, r = case
    assert list(r["op"]) == [row[0] for row in g["op_weights"]["rows"]]
    for w, row in zip(r["op_w"], g["op_weights"]["rows"]):
        assert close(w, row[1])
    K = g["keys"]
    assert list(r["ukey"]) == [K[row[0]] for row in g["key_weights"]["rows"]]
    for w, row in zip(r["omega"], g["key_weights"]["rows"]):
        assert close(w, row[1])


def test_score(case):
    g, _, r = case
    assert close(r["s_agg"], g["score"]["s_agg"], ulps=4)
    for S, row in zip(r["score_op_S"], g["score"]["op_S"]):
        assert close(S, row[1])
    assert list(r["score_op"]) == [row[0] for row in g["score"]["op_S"]]


def test_fixed_point_matches_rational_definition(case):
    g, (key, app, ph, dur), r = case
    fx = bf.fixed_point(key, app, ph, dur, g["app_weight_q16"], g["num_phases"])
    P = g["num_phases"]
    C = sum(g["app_weight_q16"])
    for (a, p), (m, rho) in fx["scale"].items():
        i = a * P + p
        assert int(r["mant"][i]) == m and int(r["rho"][i]) == rho
        # bracket: m 2^(rho-55) <= r < (m+1) 2^(rho-55), 2^55 <= m < 2^56
        rr = Fraction(g["app_weight_q16"][a] * 2 ** 96, C * fx["T"][(a, p)])
        assert 2 ** 55 <= m < 2 ** 56
        assert Fraction(m) * Fraction(2) ** (rho - 55) <= rr < Fraction(m + 1) * Fraction(2) ** (rho - 55)
    W = O.u128_to_int(r["wsum"])
    assert W == [fx["W"][(int(k), int(p))] for k, p in zip(r["key"], r["phase"])]
    # Q96 sums sit just below 2^96 times the exact shares
    rows = g["group_weights"]["rows"]
    for w, row in zip(W, rows):
        exact = Fraction(row[2]) * 2 ** 96
        assert 0 <= exact - w <= exact * Fraction(1, 2 ** 55) + row[4]
