"""Oracle vs exact-rational brute force on random traces of <= 100 events.

Bit-exact on every integer (T, n, m, rho, W, raw D, S, U) against the Q96
definition evaluated with Fractions; within the fixed-point fidelity bound
against the real-valued Eq. (2)-(3) evaluated in the paper's own nesting.
Edge cases: zero durations, apps absent from a phase, apps whose durations in
a phase are all zero, c_a = 0, single-phase keys, duplicate events, one app,
one key, durations near 2^62, up to 8 phases.
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import brute_force as bf
from oracle import oracle as O


def random_trace(seed):
    rng = np.random.default_rng(seed)
    kind = seed % 8
    P = int(rng.integers(1, 9))
    A = int(rng.integers(1, 7))
    n = int(rng.integers(0, 101))
    nops, nsh = int(rng.integers(1, 5)), int(rng.integers(1, 5))
    key = ((rng.integers(0, nops, n) + 1) << 16 | rng.integers(0, nsh, n)).astype(np.uint32)
    app = rng.integers(0, A, n).astype(np.uint32)
    ph = rng.integers(0, P, n).astype(np.uint8)
    mag = rng.choice([0, 1, 1000, 10 ** 6, 10 ** 12, 2 ** 62], size=n)
    dur = (rng.random(n) * mag).astype(np.int64)
    c = rng.integers(0, 2 ** 32, A, dtype=np.uint64).astype(np.uint32)
    if kind == 1:      # zero durations everywhere in one app
        dur[app == 0] = 0
    elif kind == 2:    # c_a = 0 for some apps
        c[: A // 2] = 0
    elif kind == 3:    # duplicate every event
        key, app, ph, dur = [np.concatenate([x, x]) for x in (key, app, ph, dur)]
    elif kind == 4:    # single app
        A = 1
        app[:] = 0
        c = c[:1]
    elif kind == 5:    # single key
        key[:] = 7 << 16 | 3
    elif kind == 6:    # keys confined to one phase each
        ph = (key & 0xFFFF) % P
        ph = ph.astype(np.uint8)
    elif kind == 7:    # app absent from a phase
        if P > 1:
            ph[app == 0] = 0
    if int(c.astype(np.uint64).sum()) == 0:
        c[0] = 1
    return key, app, ph, dur, c, P


def real_bound(n_events, share):
    """Relative error allowed between oracle output and the real-valued share:
    scale truncation (< 2^-55 per factor) plus per-invocation floors (< 1/2^96
    each, relative to the share), doubled for the normalisation, plus fp64."""
    if share == 0:
        return 0.0
    return 4.0 * (2.0 ** -55 + n_events / (2.0 ** 96 * float(share))) + 8 * 2.0 ** -53


@pytest.mark.parametrize("seed", range(240))
def test_bruteforce(seed):
    key, app, ph, dur, c, P = random_trace(seed)
    r = O.run(key, app, ph, dur, c, P)
    fx = bf.fixed_point(key, app, ph, dur, c, P)
    A = len(c)
    # pass A and scale, bit-exact
    T = O.u128_to_int(r["app_total"])
    for a in range(A):
        for p in range(P):
            i = a * P + p
            assert T[i] == fx["T"].get((a, p), 0)
            assert int(r["app_count"][i]) == fx["n_app"].get((a, p), 0)
            m, rho = fx["scale"].get((a, p), (0, 0))
            assert int(r["mant"][i]) == m and int(r["rho"][i]) == rho
    # pass B, bit-exact; groups ascending by (key, phase)
    groups = sorted(fx["W"])
    assert r["num_groups"] == len(groups)
    assert [(int(k), int(p)) for k, p in zip(r["key"], r["phase"])] == groups
    assert O.u128_to_int(r["wsum"]) == [fx["W"][g] for g in groups]
    assert O.u128_to_int(r["raw_ns"]) == [fx["raw"][g] for g in groups]
    assert [int(x) for x in r["count"]] == [fx["n"][g] for g in groups]
    assert O.u128_to_int(r["phase_total"]) == [fx["S"].get(p, 0) for p in range(P)]
    # weights: RN(W)/RN(S) within an ulp or two of the exact ratio
    for w, g in zip(r["weight"], groups):
        S = fx["S"][g[1]]
        q = Fraction(fx["W"][g], S) if S else Fraction(0)
        assert abs(Fraction(w) - q) <= 2 * math.ulp(float(q) if q else 0.0) + Fraction(0)
    # Eq. (3) units: U bit-exact
    assert O.u128_to_int(r["op_U"]) == [fx["U"]["op"][u] for u in sorted(fx["U"]["op"])]
    assert O.u128_to_int(r["key_U"]) == [fx["U"]["key"][u] for u in sorted(fx["U"]["key"])]
    # fidelity to the real-valued Eq. (2)-(3)
    rv = bf.real_valued(key, app, ph, dur, c, P)
    n = len(key)
    for w, u in zip(r["op_w"], r["op"]):
        exact = rv["op"][int(u)]
        assert abs(Fraction(w) - exact) <= Fraction(real_bound(n, exact)) * exact + Fraction(0), (u, w, exact)
    for w, u in zip(r["omega"], r["ukey"]):
        exact = rv["key"][int(u)]
        assert abs(Fraction(w) - exact) <= Fraction(real_bound(n, exact)) * exact, (u, w, exact)
    for w, g in zip(r["weight"], groups):
        exact = rv["group"][g]
        if exact == 0:
            assert w == 0.0
        else:
            assert abs(Fraction(w) - exact) <= Fraction(real_bound(n, exact)) * exact, (g, w, exact)


def test_empty_trace():
    r = O.run([], [], [], [], [5], 3)
    assert r["num_groups"] == 0
    assert O.u128_to_int(r["phase_total"]) == [0, 0, 0]
