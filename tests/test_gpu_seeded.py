"""The LDS engine seeded with a sample's hottest keys (more keys than one
LDS table holds, most events on a few thousand of them): every output equals
the oracle's, on prefixes of the skewed workloads large enough for the
seeding (at least 2^22 events), through the separate calls and atrex_run.
With raw time, or when the image covers at least 15/16 of the sample, pass B
runs on the seeded table and spills the rest (lds_hash_seeded); otherwise a
smaller seeded table sits beside the partition scatter in one pass
(hot_scatter)."""
import numpy as np
import pytest

import gpu_helpers as H
from oracle import oracle as O
from paper_2607_14541_amd import atrex as X
from paper_2607_14541_amd import synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("ci,n,one_call_path", [(3, (1 << 22) + 5, "hot_scatter"),
                                                (4, (1 << 22) + 1, "lds_hash_seeded")])
def test_seeded_lds_engine_matches_the_oracle(ci, n, one_call_path):
    cfg = synth.CONFIGS[ci]
    ev = synth.events(cfg, n=n)
    c = synth.app_weights(cfg)
    keys = synth.key_space(cfg)
    s = synth.scores(cfg, keys, nan_frac=0.1)
    P = cfg["num_phases"]
    H.say("seeded LDS engine, config", ci, "n", n)
    o = O.run(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P, score_key=keys, s=s, threads=8)
    g = H.run_gpu(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P, score_key=keys, s=s,
                  max_keys=keys.size, max_groups=keys.size * P)
    assert g["path"] == "lds_hash_seeded", g["path"]
    H.compare(g, o, raw=True, score=True)
    g1, _, path = H.run_one_call(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P, keys, s,
                                 max_keys=keys.size, max_groups=keys.size * P)
    assert path == one_call_path
    H.compare(g1, o, raw=False, score=True)


def test_uniform_keys_are_not_seeded():
    cfg = synth.CONFIGS[2]  # 1M uniform keys: a table of the hottest few thousand covers little
    n = (1 << 22) + 3
    ev = synth.events(cfg, n=n)
    c = synth.app_weights(cfg)
    P = cfg["num_phases"]
    keys = synth.key_space(cfg)
    g = H.run_gpu(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P, max_keys=keys.size,
                  max_groups=keys.size * P)
    assert g["path"] == "radix_sort"
    o = O.run(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P, threads=8)
    H.compare(g, o, raw=True)


def test_cold_stretch_overflows_the_spill_regions():
    """55% of the events on 100 keys, then a stretch of 200k cold keys: the
    sample seeds the table, the workgroups over the cold stretch overflow
    their spill regions, and every event is partitioned instead."""
    rng = np.random.default_rng(11)
    n = (1 << 23) + 7  # a workgroup's share (~32k events) above its spill region (5/8 of it + 8k)
    hot = int(n * 0.55)
    key = np.concatenate([rng.integers(0, 100, hot), 1000 + rng.integers(0, 200000, n - hot)]).astype(np.uint32)
    cfg = synth.CONFIGS[1]
    ev = synth.events(cfg, n=n)
    c = synth.app_weights(cfg)
    P = cfg["num_phases"]
    H.say("seeded LDS engine, cold stretch, n", n)
    g = H.run_gpu(key, ev["app"], ev["phase"], ev["dur_ns"], c, P, max_keys=200100, max_groups=200100 * P)
    assert g["path"] == "lds_hash+radix_all", g["path"]
    o = O.run(key, ev["app"], ev["phase"], ev["dur_ns"], c, P, threads=8)
    H.compare(g, o, raw=True)


@pytest.mark.parametrize("n", [(1 << 22) + 3, (1 << 23) + 1001])
def test_hot_scatter_matches_the_oracle(n):
    """The seeded table beside the partition scatter, without raw time, on
    two ragged prefixes of the 1B-event workload (64k Zipf(0.9) keys, 3
    phases, 100k apps)."""
    cfg = synth.CONFIGS[3]
    ev = synth.events(cfg, n=n)
    c = synth.app_weights(cfg)
    keys = synth.key_space(cfg)
    P = cfg["num_phases"]
    H.say("hot scatter, n", n)
    g = H.run_gpu(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P, raw=False, max_keys=keys.size,
                  max_groups=keys.size * P)
    assert g["path"] == "hot_scatter", g["path"]
    o = O.run(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P, threads=8)
    H.compare(g, o, raw=False)


def test_hot_scatter_reserved_key_and_range_error():
    """The reserved key (never in an image) goes to the partition records;
    an invalid event fails the call with OUT_OF_RANGE and the context stays
    usable."""
    cfg = synth.CONFIGS[3]
    n = (1 << 22) + 9
    ev = synth.events(cfg, n=n)
    c = synth.app_weights(cfg)
    keys = synth.key_space(cfg)
    P = cfg["num_phases"]
    key = ev["key"].copy()
    key[::1000] = 0xFFFFFFFF
    H.say("hot scatter, reserved key")
    g = H.run_gpu(key, ev["app"], ev["phase"], ev["dur_ns"], c, P, raw=False, max_keys=keys.size + 1,
                  max_groups=(keys.size + 1) * P)
    assert g["path"] == "hot_scatter", g["path"]
    H.compare(g, O.run(key, ev["app"], ev["phase"], ev["dur_ns"], c, P, threads=8), raw=False)
    app = ev["app"].copy()
    app[n // 2] = cfg["num_apps"]  # one application past the table
    ag = X.Aggregator(P, H.dev(c, np.int32), max_events=n, max_keys=keys.size, max_groups=keys.size * P)
    try:
        kt = H.dev(ev["key"], np.int32)
        pt, dt = H.dev(ev["phase"], np.uint8), H.dev(ev["dur_ns"], np.int64)
        with pytest.raises(X.AtrexError) as e:
            ag.aggregate(kt, H.dev(app, np.int32), pt, dt)
        assert e.value.status == X.E_OUT_OF_RANGE
        G = ag.aggregate(kt, H.dev(ev["app"], np.int32), pt, dt)
        assert ag.path_used() == "hot_scatter"
        o = O.run(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P, threads=8)
        assert G == o["key"].size
    finally:
        ag.close()


@pytest.mark.parametrize("P", [1, 8])
def test_hot_scatter_phases_wide_durations_and_general_scale_words(P):
    """The hot scatter at 1 and 8 phases (Zipf(1.0) over 64k keys: the
    seeded image covers between half and 15/16 of the sample), with a tenth
    of the durations at 2^32 or more (the 64-bit share) and one application
    of weight 1 among weights 2^32 - 1 with durations near 2^62, whose scale
    exponent falls below -8 (the general scale word)."""
    import math
    rng = np.random.default_rng(40 + P)
    n, A = (1 << 22) + 13, 1000
    w = np.arange(1, 65537, dtype=float) ** -1.0
    cdf = np.cumsum(w) / w.sum()
    ids = rng.permutation(1 << 24)[:65536].astype(np.uint32) * np.uint32(131) + np.uint32(7)
    key = ids[np.minimum(np.searchsorted(cdf, rng.random(n)), 65535)]
    app = rng.integers(0, A, n).astype(np.uint32)
    ph = rng.integers(0, P, n).astype(np.uint8)
    dur = rng.lognormal(math.log(3e4), 2.0, n).astype(np.int64)
    big = rng.random(n) < 0.1
    dur[big] = rng.integers(1 << 32, 1 << 40, int(big.sum()))
    c = np.full(A, 2 ** 32 - 1, np.uint32)
    c[0] = 1
    z = app == 0
    dur[z] = rng.integers(1 << 60, 1 << 62, int(z.sum()))
    H.say("hot scatter, P", P)
    o = O.run(key, app, ph, dur, c, P, threads=8)
    assert o["rho"].min() < -8
    g = H.run_gpu(key, app, ph, dur, c, P, raw=False, max_keys=65536, max_groups=65536 * P)
    assert g["path"] == "hot_scatter", g["path"]
    H.compare(g, o, raw=False)
