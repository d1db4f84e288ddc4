"""Target-DSL device-time share on the GPU (§4.1, Metrics) against the
oracle, through the C ABI: the plain device-time group-by (no applications,
phase = inside the target DSL) and atrex_target_share.  Keys, counts and the
128-bit DSL and total times must match bit for bit; so must every share, every
operator mean and the overall mean (each is one IEEE division, or an exact
mean rounded once, on both sides), NaN where the oracle has NaN."""
import math

import numpy as np
import pytest
import torch

import gpu_helpers as H
from oracle import oracle as O
from paper_2607_14541_amd import atrex as X
from paper_2607_14541_amd import synth

pytestmark = pytest.mark.gpu


def K(op, shape):
    return (op << 16) | shape


def _np(t):
    a = t.cpu().numpy()
    return a.view(np.uint32) if a.dtype == np.int32 else a.view(np.uint64) if a.dtype == np.int64 else a


def _same_f64(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return a.shape == b.shape and np.array_equal(np.isnan(a), np.isnan(b)) and np.array_equal(
        a[~np.isnan(a)].view(np.uint64), b[~np.isnan(b)].view(np.uint64))


def gpu_share(key, flag, dur, path="auto", max_keys=0, key_capacity=None, op_capacity=None, offset=0):
    key = np.ascontiguousarray(key, np.uint32)
    flag = np.ascontiguousarray(flag, np.uint8)
    dur = np.ascontiguousarray(dur, np.int64)
    n = key.size
    if offset:  # views that start `offset` elements into their buffers (unaligned)
        kt = H.dev(np.concatenate([np.zeros(offset, np.uint32), key]), np.int32)[offset:]
        ft = H.dev(np.concatenate([np.zeros(offset, np.uint8), flag]), np.uint8)[offset:]
        dt = H.dev(np.concatenate([np.zeros(offset, np.int64), dur]), np.int64)[offset:]
    else:
        kt, ft, dt = H.dev(key, np.int32), H.dev(flag, np.uint8), H.dev(dur, np.int64)
    ag = X.Aggregator(2, None, max_events=max(n, 1), max_keys=max_keys, path=path, device_time=True)
    try:
        ag.aggregate(kt, None, ft, dt)
        r = ag.target_share(key_capacity, op_capacity)
        out = {k: (_np(v) if isinstance(v, torch.Tensor) else v) for k, v in r.items()}
        out["path"] = ag.path_used()
        return out
    finally:
        ag.close()


def check(g, o):
    assert g["num_keys"] == o["key"].size and g["num_ops"] == o["op"].size
    assert np.array_equal(g["key"], o["key"])
    assert np.array_equal(g["count"], o["count"])
    assert np.array_equal(g["dsl_ns"].reshape(-1, 2), o["dsl_ns"])
    assert np.array_equal(g["total_ns"].reshape(-1, 2), o["total_ns"])
    assert _same_f64(g["share"], o["share"]), "per-shape shares differ"
    assert np.array_equal(g["op"], o["op"])
    assert np.array_equal(g["op_shapes"], o["op_shapes"])
    assert _same_f64(g["op_share"], o["op_share"]), "operator means differ"
    assert g["defined_ops"] == o["defined_ops"]
    assert _same_f64([g["adoption"]], [o["adoption"]]), (g["adoption"], o["adoption"])


HAND = [(K(1, 0), 1, 10), (K(1, 0), 0, 10), (K(1, 1), 1, 1), (K(1, 1), 0, 3),
        (K(1, 2), 1, 0), (K(2, 0), 1, 6), (K(2, 0), 1, 9), (K(3, 7), 0, 0)]


@pytest.mark.parametrize("path", ["lds_hash", "radix_sort", "global_hash"])
def test_hand_worked_profile(path):
    key, flag, dur = (np.array(c) for c in zip(*HAND))
    H.say("share, hand-worked profile,", path)
    g = gpu_share(key, flag, dur, path=path, max_keys=8)
    check(g, O.target_share(key, flag, dur))
    assert g["adoption"] == 11 / 16 and g["defined_ops"] == 2


@pytest.mark.parametrize("ci", [0, 2, 1])
def test_profiles_at_full_size(ci):
    cfg = synth.SHARE_CONFIGS[ci]
    p = synth.profile(cfg)
    H.say("share, full size,", cfg["slug"])
    units = synth.profile_units(cfg)
    g = gpu_share(p["key"], p["is_dsl"], p["dur_ns"], max_keys=units.size)
    H.say("  engine", g["path"], "keys", g["num_keys"], "ops", g["num_ops"])
    check(g, O.target_share(p["key"], p["is_dsl"], p["dur_ns"]))


@pytest.mark.parametrize("path", ["lds_hash", "radix_sort", "global_hash"])
@pytest.mark.parametrize("ci,n", [(0, (1 << 18) + 5), (2, (1 << 19) + 3)])
def test_engines_on_ragged_prefixes(path, ci, n):
    cfg = synth.SHARE_CONFIGS[ci]
    p = synth.profile(cfg, n=n)
    H.say("share, engine", path, cfg["slug"], "n", n)
    g = gpu_share(p["key"], p["is_dsl"], p["dur_ns"], path=path, max_keys=synth.profile_units(cfg).size)
    check(g, O.target_share(p["key"], p["is_dsl"], p["dur_ns"]))


def test_unaligned_inputs():
    p = synth.profile(synth.SHARE_CONFIGS[0], n=100003)
    H.say("share, unaligned views")
    g = gpu_share(p["key"], p["is_dsl"], p["dur_ns"], offset=1)
    assert g["path"] == "global_hash"
    check(g, O.target_share(p["key"], p["is_dsl"], p["dur_ns"]))


@pytest.mark.parametrize("path", ["lds_hash", "radix_sort"])
def test_wide_durations(path):
    # durations near 2^62: 128-bit sums, the wide share path, RN of big sums
    rng = np.random.default_rng(7)
    n = 50000
    key = (rng.integers(0, 6, n) << 16 | rng.integers(0, 9, n)).astype(np.uint32)
    flag = (rng.random(n) < 0.5).astype(np.uint8)
    dur = rng.integers(1 << 61, 1 << 62, n).astype(np.int64)
    dur[::7] = rng.integers(0, 1000, dur[::7].size)
    H.say("share, wide durations,", path)
    g = gpu_share(key, flag, dur, path=path, max_keys=64)
    check(g, O.target_share(key, flag, dur))


def test_device_time_group_by_matches_the_oracle():
    """The group-by under the share: W per (key, phase) is the plain device
    time, and the per-phase totals and counts are the pass-A ones."""
    p = synth.profile(synth.SHARE_CONFIGS[0], n=(1 << 20) + 1)
    key, flag, dur = p["key"], p["is_dsl"], p["dur_ns"]
    H.say("device-time group-by")
    ag = X.Aggregator(2, None, max_events=key.size, max_keys=512, device_time=True)
    try:
        G = ag.aggregate(H.dev(key, np.int32), None, H.dev(flag, np.uint8), H.dev(dur, np.int64))
        gr = {k: _np(v) for k, v in ag.normalize().items()}
        tot = {k: _np(v) for k, v in ag.app_totals().items()}
    finally:
        ag.close()
    o = O.run(key, np.zeros(key.size, np.uint32), flag, dur, np.ones(1, np.uint32), 2)
    assert G == o["num_groups"]
    assert np.array_equal(gr["key"], o["key"]) and np.array_equal(gr["phase"], o["phase"])
    assert np.array_equal(gr["count"], o["count"])
    assert np.array_equal(gr["wsum"].reshape(-1, 2), o["raw_ns"])
    assert np.array_equal(tot["T"].reshape(-1, 2), o["app_total"])
    assert np.array_equal(tot["n"], o["app_count"])


def test_empty_profile():
    g = gpu_share(np.zeros(0, np.uint32), np.zeros(0, np.uint8), np.zeros(0, np.int64))
    assert g["num_keys"] == 0 and g["num_ops"] == 0 and g["defined_ops"] == 0
    assert math.isnan(g["adoption"])


def test_range_errors():
    for flag, dur in (([0, 2, 1], [1, 2, 3]), ([0, 1, 1], [1, -2, 3])):
        with pytest.raises(X.AtrexError) as e:
            gpu_share(np.array([1, 2, 3]), np.array(flag), np.array(dur))
        assert e.value.status == X.E_OUT_OF_RANGE


def test_capacity_and_argument_errors():
    key, flag, dur = (np.array(c, dt) for c, dt in zip(zip(*HAND), (np.uint32, np.uint8, np.int64)))
    with pytest.raises(X.AtrexError) as e:
        gpu_share(key, flag, dur, key_capacity=3)
    assert e.value.status == X.E_CAPACITY
    with pytest.raises(X.AtrexError) as e:
        gpu_share(key, flag, dur, op_capacity=2)
    assert e.value.status == X.E_CAPACITY
    # events with applications in the device-time mode
    ag = X.Aggregator(2, None, max_events=8, device_time=True)
    try:
        with pytest.raises(X.AtrexError) as e:
            ag.aggregate(H.dev(key, np.int32), H.dev(np.zeros(8, np.uint32), np.int32), H.dev(flag, np.uint8),
                         H.dev(dur, np.int64))
        assert e.value.status == X.E_INVALID_ARG
        with pytest.raises(X.AtrexError) as e:  # before the group-by
            ag.target_share()
        assert e.value.status == X.E_STATE
    finally:
        ag.close()
    # three phases, or an application-weighted context: no target share
    ag = X.Aggregator(3, None, max_events=8, device_time=True)
    try:
        ag.aggregate(H.dev(key, np.int32), None, H.dev(flag, np.uint8), H.dev(dur, np.int64))
        with pytest.raises(X.AtrexError) as e:
            ag.target_share()
        assert e.value.status == X.E_INVALID_ARG
    finally:
        ag.close()
    ag = X.Aggregator(2, H.dev(np.ones(1, np.uint32), np.int32), max_events=8)
    try:
        ag.aggregate(H.dev(key, np.int32), H.dev(np.zeros(8, np.uint32), np.int32), H.dev(flag, np.uint8),
                     H.dev(dur, np.int64))
        with pytest.raises(X.AtrexError) as e:
            ag.target_share()
        assert e.value.status == X.E_INVALID_ARG
    finally:
        ag.close()
