"""Every workload at its full size (2^20 to 2^30 events) against the oracle,
through the path the benchmark times (atrex_run, AUTO engine, every key of the
workload scored): each output's digest must equal the one the committed script
tests/golden/make_digests.py wrote from the CPU oracle's outputs on the same
seeded inputs (bit for bit: keys, phases, counts, W, S, T, m, rho, U and the
fp64 weights; S_agg within 1e-12).  A second run with the per-(app, phase)
invocation counts and the raw per-group time on checks those too.
(§3.4 Eq. (2)-(3), §3.6 Eq. (4)-(6).)  Collected after the other GPU tests."""
import os
import sys

import numpy as np
import pytest
import torch

import gpu_helpers as H
from paper_2607_14541_amd import synth

sys.path.insert(0, os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden"))
import digests as D  # noqa: E402

pytestmark = pytest.mark.gpu


def _events_on_device(cfg):
    ev = synth.events(cfg)
    t = {k: H.dev(ev[k], dt) for k, dt in (("key", np.int32), ("app", np.int32), ("phase", np.uint8),
                                           ("dur_ns", np.int64))}
    del ev
    return t


@pytest.mark.parametrize("ci", [0, 1, 4, 2, 3])
def test_full_size_matches_oracle_digests(ci):
    rec = D.load()["configs"].get(str(ci))
    if rec is None:
        pytest.skip("no oracle digest for this workload in tests/golden/full_size_digests.json")
    cfg = synth.CONFIGS[ci]
    P = cfg["num_phases"]
    keys = synth.key_space(cfg)
    s = synth.scores(cfg, keys)
    c = synth.app_weights(cfg)
    H.say("full size, config", ci, cfg["name"], "events", cfg["n"])
    ev = _events_on_device(cfg)
    try:
        args = (ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P, keys, s)
        caps = dict(max_keys=keys.size, max_groups=keys.size * P)
        g, one_wait, path = H.run_one_call(*args, **caps)
        H.say("  engine", path, "one wait", one_wait, "groups", g["num_groups"])
        if ci == 1:  # the benchmark's 64M-event step: LDS engine, one host wait
            assert path == "lds_hash" and one_wait
        bad = D.mismatches(rec, H.as_oracle_names(g), s_agg=g["s_agg"])
        assert not bad, "outputs differing from the oracle: %s" % bad
        g2, _, _ = H.run_one_call(*args, **caps, raw=True, app_count=True)
        out2 = H.as_oracle_names(g2)
        bad = D.mismatches(rec, out2, s_agg=g2["s_agg"])
        assert not bad, "with raw time and app counts, outputs differing from the oracle: %s" % bad
        assert "raw_ns" in out2 and "app_count" in out2
        # every invocation counted once: per phase, sum over keys = sum over apps
        per_key = np.zeros(P, np.uint64)
        np.add.at(per_key, out2["phase"].astype(np.int64), out2["count"])
        per_app = out2["app_count"].reshape(-1, P).sum(axis=0, dtype=np.uint64)
        assert np.array_equal(per_key, per_app)
        assert int(per_key.sum()) == cfg["n"]
    finally:
        del ev
        torch.cuda.empty_cache()
