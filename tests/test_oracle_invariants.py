"""Oracle invariants on larger random traces (10^3 .. 10^5 events).

* per-phase sums: sum_k W[k,ph] == S[ph] exactly; fp64 weights sum to 1
* permutation of events changes nothing (bit-exact)
* duplicating every event doubles counts, T and raw D exactly; each doubled
  group's Q96 sum W' lies in [W - n, W] (the floor of half a product loses at
  most one unit per invocation), so the weights agree within that bound
* sum over (a, ph) of T equals the sum of all durations (separate loop)
* sum_k n[k,ph] == sum_a n[a,ph];  sum_k D[k,ph] == sum_a T[a,ph]
"""
import numpy as np
import pytest

from oracle import oracle as O


def trace(seed, n):
    rng = np.random.default_rng(1000 + seed)
    P = int(rng.integers(1, 9))
    A = int(rng.integers(1, 200))
    key = ((rng.zipf(1.3, n) % 50).astype(np.uint32) << np.uint32(16)) | rng.integers(0, 8, n).astype(np.uint32)
    app = rng.integers(0, A, n).astype(np.uint32)
    ph = rng.integers(0, P, n).astype(np.uint8)
    dur = np.rint(np.exp(np.log(2e4) + 2.0 * rng.standard_normal(n))).astype(np.int64)
    dur[rng.random(n) < 0.01] = 0
    c = rng.integers(1, 2 ** 26, A).astype(np.uint32)
    return key, app, ph, dur, c, P


CASES = [(0, 1000), (1, 20000), (2, 100000), (3, 5000)]


@pytest.mark.parametrize("seed,n", CASES)
def test_sums(seed, n):
    key, app, ph, dur, c, P = trace(seed, n)
    r = O.run(key, app, ph, dur, c, P)
    W = O.u128_to_int(r["wsum"])
    S = O.u128_to_int(r["phase_total"])
    T = O.u128_to_int(r["app_total"])
    raw = O.u128_to_int(r["raw_ns"])
    total = 0
    for d in dur.tolist():
        total += d
    assert sum(T) == total
    for p in range(P):
        sel = r["phase"] == p
        assert sum(w for w, s in zip(W, sel) if s) == S[p]
        assert S[p] <= 2 ** 96
        if S[p]:
            assert abs(r["weight"][sel].sum() - 1.0) <= sel.sum() * 2.0 ** -52
        assert int(r["count"][sel].sum()) == int(r["app_count"].reshape(-1, P)[:, p].sum())
        assert sum(x for x, s in zip(raw, sel) if s) == sum(T[a * P + p] for a in range(len(c)))


@pytest.mark.parametrize("seed,n", CASES)
def test_permutation_invariance(seed, n):
    key, app, ph, dur, c, P = trace(seed, n)
    r1 = O.run(key, app, ph, dur, c, P)
    perm = np.random.default_rng(seed).permutation(n)
    r2 = O.run(key[perm], app[perm], ph[perm], dur[perm], c, P)
    for k in ("key", "phase", "count", "wsum", "raw_ns", "weight", "phase_total", "app_total",
              "mant", "rho", "op", "op_U", "op_w", "ukey", "key_U", "omega"):
        assert np.array_equal(r1[k], r2[k]), k


@pytest.mark.parametrize("seed,n", CASES)
def test_duplication_invariance(seed, n):
    key, app, ph, dur, c, P = trace(seed, n)
    r1 = O.run(key, app, ph, dur, c, P)
    d2 = [np.concatenate([x, x]) for x in (key, app, ph, dur)]
    r2 = O.run(*d2, c, P)
    assert np.array_equal(r1["key"], r2["key"]) and np.array_equal(r1["phase"], r2["phase"])
    assert np.array_equal(2 * r1["count"], r2["count"])
    assert [2 * x for x in O.u128_to_int(r1["app_total"])] == O.u128_to_int(r2["app_total"])
    assert [2 * x for x in O.u128_to_int(r1["raw_ns"])] == O.u128_to_int(r2["raw_ns"])
    W1, W2 = O.u128_to_int(r1["wsum"]), O.u128_to_int(r2["wsum"])
    for w1, w2, cnt in zip(W1, W2, r1["count"]):
        assert w1 - int(cnt) <= w2 <= w1
    nz = r1["weight"] > 0
    rel = np.abs(r2["weight"][nz] - r1["weight"][nz]) / r1["weight"][nz]
    bound = 2 * (2 * r1["count"][nz].astype(np.float64) /
                 np.array([float(w) for w, z in zip(W1, nz) if z]) + 2.0 ** -52)
    assert np.all(rel <= bound)
