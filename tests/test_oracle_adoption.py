"""Pins of the oracle's target-DSL device-time share (§4.1, Metrics: the mean
across operators of each operator's mean per-shape share of device time spent
inside the target DSL, taken over the operators where it is defined).

Pinned by a hand-worked profile, closed forms (all or nothing inside the DSL),
brute force with Python integers and Fractions (float(int) and int / int are
correctly rounded in Python), tie and cancellation cases of the exact mean, and
invariances (event order, scaling every duration by two)."""
import math
import random
from fractions import Fraction

import numpy as np
import pytest

from oracle import oracle as O


def K(op, shape):
    return (op << 16) | shape


def test_hand_worked_profile():
    # op 1: shape 0 has 10 of 20 ns inside the DSL (1/2), shape 1 has 1 of 4
    #       (1/4), shape 2 only zero-length invocations (does not run);
    # op 2: one shape, all inside the DSL (1);
    # op 3: only zero-length invocations: excluded, not scored 0.
    ev = [(K(1, 0), 1, 10), (K(1, 0), 0, 10), (K(1, 1), 1, 1), (K(1, 1), 0, 3),
          (K(1, 2), 1, 0), (K(2, 0), 1, 6), (K(2, 0), 1, 9), (K(3, 7), 0, 0)]
    key, flag, dur = (np.array(c) for c in zip(*ev))
    r = O.target_share(key, flag, dur)
    assert r["key"].tolist() == [K(1, 0), K(1, 1), K(1, 2), K(2, 0), K(3, 7)]
    assert r["count"].tolist() == [2, 2, 1, 2, 1]
    assert [int(x) for x in r["dsl_ns"][:, 0]] == [10, 1, 0, 15, 0]
    assert [int(x) for x in r["total_ns"][:, 0]] == [20, 4, 0, 15, 0]
    assert r["share"][:2].tolist() == [0.5, 0.25] and r["share"][3] == 1.0
    assert math.isnan(r["share"][2]) and math.isnan(r["share"][4])
    assert r["op"].tolist() == [1, 2, 3]
    assert r["op_shapes"].tolist() == [2, 1, 0]
    assert r["op_share"][0] == 3 / 8 and r["op_share"][1] == 1.0 and math.isnan(r["op_share"][2])
    assert r["defined_ops"] == 2
    assert r["adoption"] == 11 / 16


@pytest.mark.parametrize("flag", [0, 1])
def test_all_or_nothing_inside_the_dsl(flag):
    rng = np.random.default_rng(3)
    n = 5000
    key = (rng.integers(0, 40, n) << 16 | rng.integers(0, 30, n)).astype(np.uint32)
    dur = rng.integers(1, 1 << 40, n)
    r = O.target_share(key, np.full(n, flag, np.uint8), dur)
    assert np.all(r["share"] == float(flag))
    assert np.all(r["op_share"] == float(flag))
    assert r["adoption"] == float(flag)
    assert r["defined_ops"] == len(np.unique(key >> 16))


def _brute(key, flag, dur):
    keys = {}
    for k, f, d in zip(key.tolist(), flag.tolist(), dur.tolist()):
        e = keys.setdefault(k, [0, 0, 0])
        e[0] += 1
        e[1] += d if f else 0
        e[2] += d
    share = {k: (float(v[1]) / float(v[2]) if v[2] else math.nan) for k, v in keys.items()}
    ops = {}
    for k in sorted(keys):
        ops.setdefault(k >> 16, [])
        if keys[k][2]:
            ops[k >> 16].append(share[k])
    means = {i: (float(sum(Fraction(x) for x in v) / len(v)) if v else math.nan) for i, v in ops.items()}
    defined = [m for m in means.values() if not math.isnan(m)]
    adoption = float(sum(Fraction(x) for x in defined) / len(defined)) if defined else math.nan
    return keys, share, means, adoption, len(defined)


@pytest.mark.parametrize("seed", range(12))
def test_brute_force_with_fractions(seed):
    rng = random.Random(seed)
    n = rng.randint(1, 300)
    nops = rng.randint(1, 6)
    big = seed % 3 == 0  # durations near 2^62: RN of the sums matters
    key = np.array([K(rng.randrange(nops), rng.randrange(5)) for _ in range(n)], np.uint32)
    flag = np.array([rng.random() < 0.6 for _ in range(n)], np.uint8)
    dur = np.array([rng.choice([0, rng.randrange(1 << 62) if big else rng.randrange(10 ** 6)]) for _ in range(n)],
                   np.int64)
    keys, share, means, adoption, nd = _brute(key, flag, dur)
    r = O.target_share(key, flag, dur)
    assert r["key"].tolist() == sorted(keys)
    for i, k in enumerate(sorted(keys)):
        assert int(r["count"][i]) == keys[k][0]
        assert O.u128_to_int(r["dsl_ns"][i:i + 1])[0] == keys[k][1]
        assert O.u128_to_int(r["total_ns"][i:i + 1])[0] == keys[k][2]
        s = r["share"][i]
        assert (math.isnan(s) and math.isnan(share[k])) or s == share[k]
    assert r["op"].tolist() == sorted(means)
    for i, op in enumerate(sorted(means)):
        m = r["op_share"][i]
        assert (math.isnan(m) and math.isnan(means[op])) or m == means[op]
    assert r["defined_ops"] == nd
    assert (math.isnan(r["adoption"]) and math.isnan(adoption)) or r["adoption"] == adoption


def test_exact_mean_is_the_rounded_exact_mean():
    # 1 + 2^-53 + 2^-53 summed left to right in fp64 is 1 (each addition ties to
    # even); the exact sum 1 + 2^-52 over 3 rounds to a different double
    x = [1.0, 2.0 ** -53, 2.0 ** -53]
    naive = ((x[0] + x[1]) + x[2]) / 3
    exact = float((Fraction(1) + 2 * Fraction(2.0 ** -53)) / 3)
    assert naive != exact
    assert O.exact_mean(x) == exact
    # a tie: (1 + (1 + 2^-52)) / 2 = 1 + 2^-53 lies halfway; ties go to the even 1.0
    assert O.exact_mean([1.0, 1.0 + 2.0 ** -52]) == 1.0
    # the next tie goes up to the even neighbour
    a = 1.0 + 2.0 ** -52
    assert O.exact_mean([a, a + 2.0 ** -52]) == a + 2.0 ** -52
    assert O.exact_mean([0.0, 0.0]) == 0.0
    assert O.exact_mean([0.75]) == 0.75
    assert math.isnan(O.exact_mean([]))
    rng = random.Random(11)
    for _ in range(300):
        m = rng.randint(1, 50)
        v = [rng.random() * 2.0 ** rng.randint(-100, 3) for _ in range(m)]
        assert O.exact_mean(v) == float(sum(Fraction(t) for t in v) / m)


def test_invariant_under_event_order_and_doubling():
    rng = np.random.default_rng(5)
    n = 4000
    key = (rng.integers(0, 20, n) << 16 | rng.integers(0, 50, n)).astype(np.uint32)
    flag = (rng.random(n) < 0.3).astype(np.uint8)
    dur = rng.integers(0, 1 << 50, n)
    a = O.target_share(key, flag, dur)
    p = rng.permutation(n)
    b = O.target_share(key[p], flag[p], dur[p])
    c = O.target_share(key, flag, dur * 2)  # RN(2x) = 2 RN(x): every share the same
    for r in (b, c):
        assert np.array_equal(a["key"], r["key"])
        assert np.array_equal(a["share"], r["share"], equal_nan=True)
        assert np.array_equal(a["op_share"], r["op_share"], equal_nan=True)
        assert a["adoption"] == r["adoption"]


def test_errors_and_empty_profile():
    with pytest.raises(O.OracleError) as e:
        O.target_share([1], [2], [5])
    assert e.value.status == O.E_OUT_OF_RANGE
    with pytest.raises(O.OracleError) as e:
        O.target_share([1, 2], [0, 1], [5, -1])
    assert e.value.status == O.E_OUT_OF_RANGE
    r = O.target_share(np.zeros(0, np.uint32), np.zeros(0, np.uint8), np.zeros(0, np.int64))
    assert r["key"].size == 0 and r["op"].size == 0
    assert r["defined_ops"] == 0 and math.isnan(r["adoption"])
