"""Pins of the oracle's observed runtime per unit (§3.1, "Baselines and
weights": the production runtime recorded for every retained (operator,
shape) unit as its deployment baseline).

Nearest-rank quantiles: rank ceil(q n) of the ascending durations.  Pinned by
a hand-worked unit, Python integer brute force, numpy's inverted-CDF
percentile (the same definition, computed by a library), closed forms (q = 1
is the maximum, a tiny q the minimum) and invariances (event order; merging
phases equals the statistics of the union)."""
import random

import numpy as np
import pytest

from oracle import oracle as O


def test_hand_worked_unit():
    r = O.unit_stats([9, 9, 9, 9], [0, 0, 0, 0], [40, 10, 30, 20], 1, q_1e5=(25000, 50000, 75000, 99000, 100000))
    assert r["key"].tolist() == [9] and r["count"].tolist() == [4]
    assert int(r["total_ns"][0, 0]) == 100 and r["mean_ns"][0] == 25.0
    assert r["min_ns"][0] == 10 and r["max_ns"][0] == 40
    # ranks ceil(0.25*4)=1, ceil(0.5*4)=2, ceil(0.75*4)=3, ceil(0.99*4)=4, 4
    assert r["quantile_ns"][0].tolist() == [10, 20, 30, 40, 40]


def _brute(key, phase, dur, q, by_phase):
    units = {}
    for k, p, d in zip(key.tolist(), phase.tolist(), dur.tolist()):
        units.setdefault((k, p if by_phase else 0), []).append(d)
    out = []
    for u in sorted(units):
        v = sorted(units[u])
        n = len(v)
        qs = [v[-(-qq * n // 100000) - 1] for qq in q]  # rank ceil(q n), exact in integers
        out.append((u, n, sum(v), float(sum(v)) / float(n), v[0], v[-1], qs))
    return out


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("by_phase", [True, False])
def test_brute_force(seed, by_phase):
    rng = random.Random(seed)
    n = rng.randint(1, 400)
    P = rng.randint(1, 4)
    key = np.array([(rng.randrange(3) << 16) | rng.randrange(4) for _ in range(n)], np.uint32)
    phase = np.array([rng.randrange(P) for _ in range(n)], np.uint8)
    big = seed % 2 == 0
    dur = np.array([rng.randrange(1 << 62) if big else rng.randrange(1000) for _ in range(n)], np.int64)
    q = [rng.randint(1, 100000) for _ in range(rng.randint(0, 8))]
    r = O.unit_stats(key, phase, dur, P, q_1e5=q, by_phase=by_phase)
    b = _brute(key, phase, dur, q, by_phase)
    assert len(b) == r["key"].size
    for i, (u, cnt, tot, mean, mn, mx, qs) in enumerate(b):
        assert (int(r["key"][i]), int(r["phase"][i])) == u
        assert int(r["count"][i]) == cnt
        assert O.u128_to_int(r["total_ns"][i:i + 1])[0] == tot
        assert r["mean_ns"][i] == mean
        assert int(r["min_ns"][i]) == mn and int(r["max_ns"][i]) == mx
        assert r["quantile_ns"][i].tolist() == qs


def test_against_numpy_inverted_cdf():
    rng = np.random.default_rng(4)
    n = 20000
    key = rng.integers(0, 12, n).astype(np.uint32)
    dur = np.rint(np.exp(10 + 2 * rng.standard_normal(n))).astype(np.int64)
    q = [1000, 10000, 50000, 90000, 99000, 99900]
    r = O.unit_stats(key, np.zeros(n, np.uint8), dur, 1, q_1e5=q)
    for i, k in enumerate(r["key"]):
        v = dur[key == k]
        ref = [int(np.percentile(v, qq / 1000.0, method="inverted_cdf")) for qq in q]
        assert r["quantile_ns"][i].tolist() == ref
        assert r["min_ns"][i] == v.min() and r["max_ns"][i] == v.max()


def test_closed_forms_and_invariances():
    rng = np.random.default_rng(8)
    n = 5000
    key = (rng.integers(0, 5, n) << 16 | rng.integers(0, 7, n)).astype(np.uint32)
    phase = rng.integers(0, 3, n).astype(np.uint8)
    dur = rng.integers(0, 1 << 40, n)
    q = (1, 50000, 100000)
    a = O.unit_stats(key, phase, dur, 3, q_1e5=q)
    assert np.array_equal(a["quantile_ns"][:, 0], a["min_ns"])  # a unit has < 1e5 invocations
    assert np.array_equal(a["quantile_ns"][:, 2], a["max_ns"])
    p = rng.permutation(n)
    b = O.unit_stats(key[p], phase[p], dur[p], 3, q_1e5=q)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    # merging the phases of a key gives the statistics of the union
    m = O.unit_stats(key, phase, dur, 3, q_1e5=q, by_phase=False)
    z = O.unit_stats(key, np.zeros(n, np.uint8), dur, 1, q_1e5=q)
    for k in m:
        assert np.array_equal(m[k], z[k]), k
    per_key = {}
    for kk, c in zip(a["key"].tolist(), a["count"].tolist()):
        per_key[kk] = per_key.get(kk, 0) + c
    assert [per_key[k] for k in m["key"].tolist()] == m["count"].tolist()


def test_errors():
    for q in ((0,), (100001,), tuple(range(1, 10))):
        with pytest.raises(O.OracleError) as e:
            O.unit_stats([1], [0], [5], 1, q_1e5=q)
        assert e.value.status == O.E_INVALID_ARG
    with pytest.raises(O.OracleError) as e:
        O.unit_stats([1, 2], [0, 2], [5, 6], 2)
    assert e.value.status == O.E_OUT_OF_RANGE
    with pytest.raises(O.OracleError) as e:
        O.unit_stats([1, 2], [0, 1], [5, -6], 2)
    assert e.value.status == O.E_OUT_OF_RANGE
    r = O.unit_stats(np.zeros(0, np.uint32), np.zeros(0, np.uint8), np.zeros(0, np.int64), 2)
    assert r["key"].size == 0
