"""HIP path vs the CPU oracle, through the C ABI, on the same seeded inputs.

Integers (keys, counts, T, m, rho, W, raw time, S, U) must match bit for bit;
fp64 outputs (weights, S_agg) within 1e-12 relative, zeros exactly zero.
Every engine is forced in turn."""
import json
import math
import os

import numpy as np
import pytest

import gpu_helpers as H
from oracle import oracle as O
from paper_2607_14541_amd import synth
from test_oracle_bruteforce import random_trace

pytestmark = pytest.mark.gpu
ENGINES = ["lds_hash", "global_hash", "radix_sort"]


@pytest.mark.parametrize("path", ENGINES)
def test_golden_trace(path):
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "tiny_trace.json")))
    K = g["keys"]
    ev = g["events"]
    key, app, ph, dur = ([K[e[0]] for e in ev], [e[1] for e in ev], [e[2] for e in ev], [e[3] for e in ev])
    sk = [K[k] for k in g["score"]["score_keys"]]
    s = [math.nan if x is None else x for x in g["score"]["S"]]
    H.say("golden", path)
    gr = H.run_gpu(key, app, ph, dur, g["app_weight_q16"], 2, path=path, score_key=sk, s=s)
    o = O.run(key, app, ph, dur, g["app_weight_q16"], 2, score_key=sk, s=s)
    H.compare(gr, o, score=True)
    assert abs(gr["s_agg"] - 363 / 1280) < 1e-15


@pytest.mark.parametrize("path", ENGINES)
@pytest.mark.parametrize("seed", range(0, 48))
def test_random_small(path, seed):
    key, app, ph, dur, c, P = random_trace(seed)
    if key.size == 0:
        pytest.skip("empty trace covered separately")
    H.say("random", seed, path, key.size)
    H.compare(H.run_gpu(key, app, ph, dur, c, P, path=path), O.run(key, app, ph, dur, c, P))


@pytest.mark.parametrize("path", ENGINES)
@pytest.mark.parametrize("n", [1, 3, 5, 64, 4095, 4097, 100003])
def test_ragged_sizes(path, n):
    rng = np.random.default_rng(n)
    P, A = 3, 17
    key = ((rng.integers(0, 40, n) << 16) | rng.integers(0, 9, n)).astype(np.uint32)
    app = rng.integers(0, A, n).astype(np.uint32)
    ph = rng.integers(0, P, n).astype(np.uint8)
    dur = rng.integers(0, 10 ** 9, n).astype(np.int64)
    c = rng.integers(1, 2 ** 24, A).astype(np.uint32)
    H.say("ragged", n, path)
    H.compare(H.run_gpu(key, app, ph, dur, c, P, path=path), O.run(key, app, ph, dur, c, P))


@pytest.mark.parametrize("path", ENGINES)
def test_empty_trace(path):
    H.say("empty", path)
    g = H.run_gpu(np.zeros(0, np.uint32), np.zeros(0, np.uint32), np.zeros(0, np.uint8),
                  np.zeros(0, np.int64), [5, 6], 3, path=path)
    assert g["num_groups"] == 0 and not g["phase_total"].any()


def _config_case(ci, n):
    cfg = synth.CONFIGS[ci]
    ev = synth.events(cfg, n=n)
    c = synth.app_weights(cfg)
    return cfg, ev, c


@pytest.mark.parametrize("path,count", [("lds_hash", True), ("global_hash", True), ("radix_sort", True),
                                        ("lds_hash", False), ("radix_sort", False)])
@pytest.mark.parametrize("ci,n", [(0, 1 << 20), (1, 1 << 21), (2, 1 << 20), (3, 1 << 21), (4, 1 << 21)])
def test_config_prefix(path, count, ci, n):
    """Prefixes of every workload; pass A with and without the per-(app,
    phase) invocation counts (the counting variants take more LDS per pair, so
    the 256M- and 1B-event workloads' pair tables split differently)."""
    cfg, ev, c = _config_case(ci, n)
    keys = synth.key_space(cfg)
    if keys.size > 1 << 18:
        keys = keys[:: keys.size // (1 << 18)]
    s = synth.scores(cfg, keys, nan_frac=0.1)
    H.say("config", ci, "n", n, path)
    g = H.run_gpu(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, cfg["num_phases"], path=path,
                  score_key=keys, s=s, max_groups=2 * n, max_keys=n, app_count=count)
    o = O.run(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, cfg["num_phases"], score_key=keys, s=s,
              threads=8)
    H.compare(g, o, score=True)


def test_lds_engine_spill_overflow_falls_back_to_partitioning():
    """1M distinct keys forced through the LDS engine: nearly every event
    spills; with 8M events the per-workgroup spill regions overflow and the
    whole pass is redone by the partition engine."""
    cfg, ev, c = _config_case(2, 1 << 23)
    H.say("spill overflow")
    g = H.run_gpu(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, 4, path="lds_hash", raw=False,
                  max_groups=1 << 23, max_keys=1 << 21)
    assert g["path"] == "lds_hash+radix_all"
    o = O.run(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, 4)
    H.compare(g, o, raw=False)


def test_repeat_runs_are_bit_identical():
    cfg, ev, c = _config_case(1, 1 << 20)
    H.say("determinism")
    a = H.run_gpu(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, 2)
    b = H.run_gpu(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, 2)
    for k in ("key", "count", "wsum", "weight", "op_U", "omega"):
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("path", ENGINES)
@pytest.mark.parametrize("G", [1023, 1024, 1025, 8191, 8192, 8193, 20000])
def test_group_count_boundaries(path, G):
    """Exactly G (key, phase) groups around the one-workgroup unit kernel's
    limit and the 1024-group tiles; operators of 7 shapes, so that operator
    runs and key runs cross thread and tile boundaries."""
    rng = np.random.default_rng(G)
    P = 2
    nk = (G + 1) // 2
    keys = np.array([((k // 7) << 16) | (k % 7) for k in range(nk)], np.uint32)
    gk = np.repeat(keys, 2)[:G]
    gp = np.tile(np.array([0, 1], np.uint8), nk)[:G]
    reps = rng.integers(1, 4, G)
    key = np.repeat(gk, reps)
    ph = np.repeat(gp, reps)
    order = rng.permutation(key.size)
    key, ph = key[order], ph[order]
    A = 5
    app = rng.integers(0, A, key.size).astype(np.uint32)
    dur = rng.integers(1, 10 ** 7, key.size).astype(np.int64)
    c = rng.integers(1, 2 ** 20, A).astype(np.uint32)
    H.say("groups", G, path)
    g = H.run_gpu(key, app, ph, dur, c, P, path=path, max_groups=G, max_keys=nk)
    assert g["num_groups"] == G
    H.compare(g, O.run(key, app, ph, dur, c, P))


@pytest.mark.parametrize("count", [False, True])
@pytest.mark.parametrize("seed", [0, 1])
def test_range_split_pass_a_wraps_and_high_words(seed, count):
    """100000 apps x 3 phases: pass A runs in ranges of the (app, phase)
    table with 32-bit LDS counters.  A third of the events land on one
    (app, phase) with durations near 2^31 (the 32-bit counter wraps every
    few events) and a tenth carry durations up to 2^40 (high words), spread
    over every range; the tail of the trace is ragged (n not a multiple of 4)."""
    rng = np.random.default_rng(100 + seed)
    n, A, P = (1 << 20) + 3, 100000, 3
    key = rng.integers(0, 4096, n).astype(np.uint32)
    app = rng.integers(0, A, n).astype(np.uint32)
    ph = rng.integers(0, P, n).astype(np.uint8)
    dur = rng.lognormal(math.log(3e4), 2.0, n).astype(np.int64)
    hot = rng.random(n) < 1 / 3
    app[hot], ph[hot] = 77777, 1
    dur[hot] = rng.integers(1 << 30, 1 << 31, int(hot.sum()))
    big = rng.random(n) < 0.1
    dur[big] = rng.integers(1 << 32, 1 << 40, int(big.sum()))
    c = rng.integers(1, 1000, A).astype(np.uint32)
    H.say("range-split pass A, wraps and high words, seed", seed, "counts", count)
    g = H.run_gpu(key, app, ph, dur, c, P, max_groups=2 * n, max_keys=n, app_count=count)
    o = O.run(key, app, ph, dur, c, P)
    H.compare(g, o)


def _u(pairs):
    return [int(lo) | (int(hi) << 64) for lo, hi in np.asarray(pairs, np.uint64).reshape(-1, 2)]


@pytest.mark.parametrize("ci,n", [(1, 1 << 20), (3, 1 << 20), (4, 1 << 20)])
def test_weights_are_correctly_rounded_ratios(ci, n):
    """Every fp64 weight the kernels produce is RN(numerator) / RN(denominator)
    of the exact integers they also return (group W over the phase total S,
    U_i over sum U, U_k over sum U_k): Python's int -> float conversion rounds
    to nearest even, so this pins the device's 128-bit -> fp64 conversion and
    its division bit for bit, not only within the parity tolerance."""
    cfg, ev, c = _config_case(ci, n)
    H.say("correctly rounded weights, config", ci, "n", n)
    g = H.run_gpu(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, cfg["num_phases"],
                  max_groups=2 * n, max_keys=n)
    S = _u(g["phase_total"])
    W = _u(g["wsum"])
    want = [float(w) / float(S[p]) if S[p] else 0.0 for w, p in zip(W, g["phase"])]
    assert np.array_equal(g["weight"], np.array(want)), "group weight"
    for U, w in ((_u(g["op_U"]), g["op_w"]), (_u(g["key_U"]), g["omega"])):
        tot = float(sum(U))
        assert np.array_equal(w, np.array([float(u) / tot for u in U])), "unit weight"


@pytest.mark.parametrize("path", ENGINES)
def test_negative_scale_exponents(path):
    """(app, phase) pairs whose Q96 factor 2^96 c_a / (C T) is below 2^-8 (one
    app with c_a = 1 among apps of weight 2^32 - 1, with durations near 2^62):
    rho < -8 takes the general scale word on every engine, and rho < 0 must
    come back signed."""
    rng = np.random.default_rng(17)
    n, P, A = 20000, 2, 1000
    key = ((rng.integers(0, 30, n) << 16) | rng.integers(0, 4, n)).astype(np.uint32)
    app = rng.integers(0, A, n).astype(np.uint32)
    app[: n // 2] = 0
    ph = rng.integers(0, P, n).astype(np.uint8)
    dur = rng.integers(1 << 60, 1 << 62, n).astype(np.int64)
    c = np.full(A, 2 ** 32 - 1, np.uint32)
    c[0] = 1
    o = O.run(key, app, ph, dur, c, P)
    assert o["rho"].min() < -8
    H.say("negative scale exponents", path)
    H.compare(H.run_gpu(key, app, ph, dur, c, P, path=path, max_groups=2 * n, max_keys=n), o)


@pytest.mark.parametrize("raw", [False, True])
@pytest.mark.parametrize("case", ["two_phases", "two_keys_two_phases", "one_phase", "hot_then_cold"])
def test_hot_groups_summed_across_the_wave(case, raw):
    """The LDS engine's hot groups: when at least half of a wave's lanes share
    the (key, phase) of the first lane's first event, up to two groups are
    summed per lane and then across the wave, the rest go to LDS atomics.
    two_phases: one key in two phases (70/30), both groups summed;
    two_keys_two_phases: four hot groups, two summed, two by atomics;
    one_phase: P = 1; hot_then_cold: the second group is a cold key, which
    ends the rounds.  1% of the durations are 2^32 ns or more (the wide share
    path)."""
    rng = np.random.default_rng({"two_phases": 1, "two_keys_two_phases": 2, "one_phase": 3,
                                 "hot_then_cold": 4}[case])
    n = (1 << 21) + 37
    u = rng.random(n)
    cold = 100 + rng.integers(0, 1000, n)
    if case == "two_phases":
        P = 2
        key = np.where(u < 0.95, 7, cold)
        ph = (rng.random(n) < 0.3).astype(np.int64)
    elif case == "two_keys_two_phases":
        P = 2
        key = np.select([u < 0.70, u < 0.95], [7, 9], cold)
        ph = np.select([u < 0.55, u < 0.70, u < 0.85, u < 0.95], [0, 1, 0, 1], rng.integers(0, P, n))
    elif case == "one_phase":
        P = 1
        key = np.where(u < 0.9, 7, cold)
        ph = np.zeros(n, np.int64)
    else:
        P = 3
        key = np.where(u < 0.7, 7, cold)
        ph = np.where(u < 0.7, 1, rng.integers(0, P, n))
    A = 16
    app = rng.integers(0, A, n)
    dur = rng.integers(1, 1 << 20, n)
    wide = rng.random(n) < 0.01
    dur[wide] = rng.integers(1 << 32, 1 << 40, int(wide.sum()))
    c = rng.integers(1, 1 << 20, A)
    H.say("hot groups", case, "raw", raw, "n", n)
    g = H.run_gpu(key, app, ph, dur, c, P, path="lds_hash", raw=raw, max_keys=1002, max_groups=1002 * P)
    assert g["path"] == "lds_hash", g["path"]
    o = O.run(key.astype(np.uint32), app.astype(np.uint32), ph.astype(np.uint8), dur.astype(np.int64), c, P,
              threads=8)
    H.compare(g, o, raw=raw)
