"""Observed runtime per unit on the GPU (§3.1, "Baselines and weights": the
production runtime of every retained (operator, shape) unit, its deployment
baseline) against the oracle, through the C ABI: the device-time group-by,
then atrex_unit_stats on the same events.  Keys, phases, counts, 128-bit
totals, min, max and every nearest-rank quantile must match bit for bit, and
so must the mean (one IEEE division on both sides).  The workloads reach the
three paths of the kernels: units of at most 64 invocations (sorted by one
wave), of at most 8192 (one workgroup), and larger (radix select over
several rounds)."""
import numpy as np
import pytest
import torch

import gpu_helpers as H
from oracle import oracle as O
from paper_2607_14541_amd import atrex as X
from paper_2607_14541_amd import synth

pytestmark = pytest.mark.gpu


def _np(t):
    a = t.cpu().numpy()
    return a.view(np.uint32) if a.dtype == np.int32 else a


def gpu_stats(key, phase, dur, P, q, by_phase, path="auto", max_keys=0, capacity=None):
    key = np.ascontiguousarray(key, np.uint32)
    phase = np.ascontiguousarray(phase, np.uint8)
    dur = np.ascontiguousarray(dur, np.int64)
    kt, pt, dt = H.dev(key, np.int32), H.dev(phase, np.uint8), H.dev(dur, np.int64)
    ag = X.Aggregator(P, None, max_events=max(key.size, 1), max_keys=max_keys, path=path, device_time=True)
    try:
        ag.aggregate(kt, None, pt, dt)
        r = ag.unit_stats(kt, pt, dt, q_1e5=q, by_phase=by_phase, capacity=capacity)
        out = {k: (_np(v) if isinstance(v, torch.Tensor) else v) for k, v in r.items()}
        out["path"] = ag.path_used()
        return out
    finally:
        ag.close()


def check(g, o):
    assert g["num_units"] == o["key"].size
    assert np.array_equal(g["key"], o["key"])
    assert np.array_equal(g["phase"], o["phase"])
    assert np.array_equal(g["count"].view(np.uint64), o["count"])
    assert np.array_equal(g["total_ns"].view(np.uint64), o["total_ns"])
    assert np.array_equal(g["mean_ns"].view(np.uint64), o["mean_ns"].view(np.uint64)), "mean"
    assert np.array_equal(g["min_ns"], o["min_ns"]), "min"
    assert np.array_equal(g["max_ns"], o["max_ns"]), "max"
    assert np.array_equal(g["quantile_ns"].reshape(o["quantile_ns"].shape), o["quantile_ns"]), "quantiles"


Q2 = (50000, 99000)
Q8 = (1, 1000, 25000, 50000, 75000, 99000, 99900, 100000)


def _events(ci, n):
    cfg = synth.CONFIGS[ci]
    ev = synth.events(cfg, n=n)
    return ev["key"], ev["phase"], ev["dur_ns"], cfg["num_phases"], synth.key_space(cfg).size


@pytest.mark.parametrize("by_phase", [True, False])
@pytest.mark.parametrize("ci,n", [(0, (1 << 20) + 3),   # 1024 units of ~1k invocations: one workgroup each
                                  (1, (1 << 22) + 1),   # Zipf(1.1) over 4096 keys: all three paths
                                  (2, (1 << 20) + 5),   # 4M possible units, ~1 invocation each: one wave each
                                  (4, (1 << 21) + 7)])  # one key with 99% of the invocations, durations ~2^40
def test_workload_prefixes(ci, n, by_phase):
    key, phase, dur, P, K = _events(ci, n)
    H.say("unit stats, config", ci, "n", n, "by phase", by_phase)
    g = gpu_stats(key, phase, dur, P, Q8, by_phase, max_keys=K)
    check(g, O.unit_stats(key, phase, dur, P, q_1e5=Q8, by_phase=by_phase))


@pytest.mark.parametrize("path", ["lds_hash", "radix_sort", "global_hash"])
def test_engines_and_two_quantiles(path):
    key, phase, dur, P, K = _events(1, 300007)
    H.say("unit stats, engine", path)
    g = gpu_stats(key, phase, dur, P, Q2, True, path=path, max_keys=K)
    assert g["path"] == path
    check(g, O.unit_stats(key, phase, dur, P, q_1e5=Q2, by_phase=True))


def test_wide_durations_and_every_size_class():
    # units of 1..64, 65..8192 and > 8192 invocations; durations up to 2^62
    rng = np.random.default_rng(3)
    sizes = [1, 2, 63, 64, 65, 200, 4096, 8192, 8193, 30000, 70000]
    key = np.concatenate([np.full(s, (7 << 16) | i, np.uint32) for i, s in enumerate(sizes)])
    dur = rng.integers(0, 1 << 62, key.size).astype(np.int64)
    dur[::5] = rng.integers(0, 100, dur[::5].size)  # ties and small values among the large ones
    p = rng.permutation(key.size)
    key, dur = key[p], dur[p]
    phase = (rng.random(key.size) < 0.3).astype(np.uint8)
    H.say("unit stats, every size class")
    for by_phase in (True, False):
        g = gpu_stats(key, phase, dur, 2, Q8, by_phase, max_keys=64)
        check(g, O.unit_stats(key, phase, dur, 2, q_1e5=Q8, by_phase=by_phase))


def test_no_quantiles_and_all_equal_durations():
    key = np.repeat(np.arange(5, dtype=np.uint32), [1, 10, 100, 10000, 20000])
    dur = np.full(key.size, 12345, np.int64)
    dur[:3] = 0
    phase = np.zeros(key.size, np.uint8)
    for q in ((), (1, 100000)):
        g = gpu_stats(key, phase, dur, 1, q, False, max_keys=8)
        check(g, O.unit_stats(key, phase, dur, 1, q_1e5=q, by_phase=False))


def test_profile_workload_at_full_size():
    cfg = synth.SHARE_CONFIGS[1]  # 64M invocations over 440 units: the radix select on every unit
    p = synth.profile(cfg)
    H.say("unit stats, 64M-invocation profile")
    g = gpu_stats(p["key"], p["is_dsl"], p["dur_ns"], 2, Q2, False, max_keys=synth.profile_units(cfg).size)
    check(g, O.unit_stats(p["key"], p["is_dsl"], p["dur_ns"], 2, q_1e5=Q2, by_phase=False))


def test_errors():
    key, phase, dur, P, K = _events(0, 5000)
    kt, pt, dt = H.dev(key, np.int32), H.dev(phase, np.uint8), H.dev(dur, np.int64)
    ag = X.Aggregator(P, None, max_events=5000, max_keys=K, device_time=True)
    try:
        with pytest.raises(X.AtrexError) as e:  # before the group-by
            ag.unit_stats(kt, pt, dt)
        assert e.value.status == X.E_STATE
        ag.aggregate(kt, None, pt, dt)
        with pytest.raises(X.AtrexError) as e:  # other events than the aggregated ones
            ag.unit_stats(kt[:4000], pt[:4000], dt[:4000])
        assert e.value.status == X.E_INVALID_ARG
        other = kt.clone()
        other[17] = 0x7FFF0001  # a key the group-by never saw
        with pytest.raises(X.AtrexError) as e:
            ag.unit_stats(other, pt, dt)
        assert e.value.status == X.E_INVALID_ARG
        for q in ((0,), (100001,)):
            with pytest.raises(X.AtrexError) as e:
                ag.unit_stats(kt, pt, dt, q_1e5=q)
            assert e.value.status == X.E_INVALID_ARG
        with pytest.raises(X.AtrexError) as e:
            ag.unit_stats(kt, pt, dt, capacity=3)
        assert e.value.status == X.E_CAPACITY
        r = ag.unit_stats(kt, pt, dt)  # still usable
        o = O.unit_stats(key, phase, dur, P)
        assert np.array_equal(_np(r["quantile_ns"]), o["quantile_ns"])
    finally:
        ag.close()
    ag = X.Aggregator(P, H.dev(np.ones(64, np.uint32), np.int32), max_events=5000)
    try:
        ag.aggregate(kt, H.dev(np.zeros(5000, np.uint32), np.int32), pt, dt)
        with pytest.raises(X.AtrexError) as e:  # not a device-time context
            ag.unit_stats(kt, pt, dt)
        assert e.value.status == X.E_INVALID_ARG
    finally:
        ag.close()
