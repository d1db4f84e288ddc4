"""The oracle's sharded group-by (events split over threads, private maps
merged by exact integer addition) against its single-threaded group-by: every
output identical bit for bit, and the same status on a bad event.  Every
output is a sum over events (§3.4 Eq. (2)-(3)), so the split cannot change it;
this pins the merge (a dropped shard, a shard boundary counted twice, a field
not merged) on traces where each of those mistakes changes some output."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_14541_amd import synth
from test_oracle_bruteforce import random_trace

FIELDS = ("key", "phase", "count", "wsum", "raw_ns", "weight", "phase_total", "app_total", "app_count",
          "mant", "rho", "op", "op_U", "op_w", "ukey", "key_U", "omega")


def _same(a, b):
    assert a["num_groups"] == b["num_groups"]
    for f in FIELDS:
        x, y = np.asarray(a[f]), np.asarray(b[f])
        assert x.dtype == y.dtype and x.shape == y.shape, f
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8)), f


@pytest.mark.parametrize("seed", range(24))
@pytest.mark.parametrize("threads", [2, 3, 16, 200])
def test_sharded_equals_single_threaded_on_random_traces(seed, threads):
    key, app, ph, dur, c, P = random_trace(seed)
    _same(O.run(key, app, ph, dur, c, P, threads=threads), O.run(key, app, ph, dur, c, P))


@pytest.mark.parametrize("ci", [0, 1, 3, 4])
def test_sharded_equals_single_threaded_on_workload_prefixes(ci):
    cfg = synth.CONFIGS[ci]
    ev = synth.events(cfg, n=(1 << 17) + 5)
    c = synth.app_weights(cfg)
    keys = synth.key_space(cfg)[:3000]
    s = synth.scores(cfg, keys, nan_frac=0.1)
    args = (ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, cfg["num_phases"])
    a = O.run(*args, score_key=keys, s=s, threads=7)
    b = O.run(*args, score_key=keys, s=s)
    _same(a, b)
    for f in ("score_op", "score_op_weight", "score_op_S"):
        assert np.array_equal(a[f], b[f]), f
    assert a["s_agg"] == b["s_agg"]


def test_sharded_reports_a_bad_event_in_any_shard():
    key, app, ph, dur, c, P = random_trace(9)  # 97 events
    n = key.size
    assert n > 8
    for at in (0, n // 2, n - 1):
        bad = dur.copy()
        bad[at] = -1
        with pytest.raises(O.OracleError) as e:
            O.run(key, app, ph, bad, c, P, threads=4)
        assert e.value.status == O.E_OUT_OF_RANGE
