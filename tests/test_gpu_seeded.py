"""The LDS engine seeded with a sample's hottest keys (more keys than one
LDS table holds, most events on a few thousand of them): every output equals
the oracle's, on prefixes of the skewed workloads large enough for the
seeding (at least 2^22 events), through the separate calls and atrex_run."""
import numpy as np
import pytest

import gpu_helpers as H
from oracle import oracle as O
from paper_2607_14541_amd import synth

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("ci,n", [(3, (1 << 22) + 5), (4, (1 << 22) + 1)])
def test_seeded_lds_engine_matches_the_oracle(ci, n):
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
    assert path == "lds_hash_seeded"
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
