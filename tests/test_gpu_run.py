"""atrex_run (one call for the whole path) against the calls one by one, on
the same context type and inputs: every output bit for bit, every count, and
the same error statuses in the same order."""
import math

import numpy as np
import pytest
import torch

import gpu_helpers as H
from paper_2607_14541_amd import atrex as X
from paper_2607_14541_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _dev(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a).view(dt)).to(DEV)


def _case(ci, n, nscore=None, seed_s=0):
    cfg = synth.CONFIGS[ci]
    ev = synth.events(cfg, n=n)
    c = synth.app_weights(cfg)
    keys = synth.key_space(cfg)
    if nscore is not None:
        keys = keys[:nscore]
    s = synth.scores(cfg, keys, nan_frac=0.1)
    return cfg, ev, c, keys, s


def _tensors(ev, c, keys, s):
    return (_dev(ev["key"], np.int32), _dev(ev["app"], np.int32), _dev(ev["phase"], np.uint8),
            _dev(ev["dur_ns"], np.int64), _dev(c, np.int32), _dev(keys, np.int32), _dev(s, np.float64))


def _score_bufs(n):
    return dict(op=torch.empty(n, dtype=torch.int32, device=DEV),
                op_weight=torch.empty(n, dtype=torch.float64, device=DEV),
                op_score=torch.empty(n, dtype=torch.float64, device=DEV))


def _same(a, b, what):
    assert a.dtype == b.dtype and a.shape == b.shape, what
    assert torch.equal(a.cpu().view(torch.uint8) if a.dtype == torch.float64 else a.cpu(),
                       b.cpu().view(torch.uint8) if b.dtype == torch.float64 else b.cpu()), what


@pytest.mark.parametrize("ci,n,nscore", [(0, 1 << 20, None), (1, 1 << 21, None), (2, 1 << 20, 1 << 14),
                                         (1, (1 << 20) + 3, 100)])
def test_run_matches_the_separate_calls(ci, n, nscore):
    """nscore above 8192 takes the large score path (its own waits); up to
    8192 the normalisation and the score run back to back."""
    cfg, ev, c, keys, s = _case(ci, n, nscore)
    P = cfg["num_phases"]
    k, a, p, d, dc, sk, sv = _tensors(ev, c, keys, s)
    H.say("atrex_run vs separate calls, config", ci, "n", n, "scored", keys.size)
    mg = 2 * n
    ag = X.Aggregator(P, dc, max_events=n, max_groups=mg, max_keys=n, max_score=keys.size)
    try:
        gb = ag.group_buffers(mg)
        res = ag.run(k, a, p, d, gb, sk, sv, _score_bufs(keys.size))
        run_g = {kk: v.clone() for kk, v in res["groups"].items()}
        run_s = {kk: (v.clone() if torch.is_tensor(v) else v) for kk, v in res["score"].items()}
        run_ops, run_keys = ag.num_ops, ag.num_keys
        opw = {kk: v.clone() for kk, v in ag.op_weights().items()}
        kw = {kk: v.clone() for kk, v in ag.key_weights().items()}
        ag.reset()
        G = ag.aggregate(k, a, p, d)
        sep_g = ag.normalize(out=ag.group_buffers(mg))
        sep_s = ag.score(sk, sv)
        assert G == run_g["key"].numel()
        assert (ag.num_ops, ag.num_keys) == (run_ops, run_keys)
        for kk in sep_g:
            _same(run_g[kk], sep_g[kk], kk)
        for kk in ("op", "op_weight", "op_score"):
            _same(run_s[kk], sep_s[kk], "score " + kk)
        assert run_s["s_agg"] == sep_s["s_agg"]
        for kk, v in ag.op_weights().items():
            _same(opw[kk], v, "op " + kk)
        for kk, v in ag.key_weights().items():
            _same(kw[kk], v, "key " + kk)
    finally:
        ag.close()


def test_run_without_score_and_repeated():
    cfg, ev, c, keys, s = _case(0, 1 << 18)
    k, a, p, d, dc, sk, sv = _tensors(ev, c, keys, s)
    H.say("atrex_run without score, three times")
    ag = X.Aggregator(cfg["num_phases"], dc, max_events=1 << 18, max_groups=1 << 19, max_keys=1 << 18)
    try:
        gb = ag.group_buffers(1 << 19)
        first = {kk: v.clone() for kk, v in ag.run(k, a, p, d, gb)["groups"].items()}
        for _ in range(2):
            again = ag.run(k, a, p, d, gb)
            assert "score" not in again
            for kk in first:
                _same(first[kk], again["groups"][kk], kk)
    finally:
        ag.close()


def _status(fn):
    try:
        fn()
    except X.AtrexError as e:
        return e.status
    return X.OK


def test_run_errors_in_call_order():
    cfg, ev, c, keys, s = _case(0, 1 << 16)
    P = cfg["num_phases"]
    k, a, p, d, dc, sk, sv = _tensors(ev, c, keys, s)
    H.say("atrex_run errors")
    ag = X.Aggregator(P, dc, max_events=1 << 16, max_groups=1 << 17, max_keys=1 << 16, max_score=keys.size)
    try:
        gb = ag.group_buffers(1 << 17)
        sb = _score_bufs(keys.size)
        # fewer output rows than groups
        small = {kk: (v if kk == "phase_total" else v[:10]) for kk, v in gb.items()}
        assert _status(lambda: ag.run(k, a, p, d, small, sk, sv, sb)) == X.E_CAPACITY
        # a bad event: the group-by fails first, the score is not reached
        bad = d.clone()
        bad[12345] = -1
        assert _status(lambda: ag.run(k, a, p, bad, gb, sk, sv, sb)) == X.E_OUT_OF_RANGE
        # a score above 1: the normalisation results stand, the score fails
        s2 = sv.clone()
        s2[3] = 1.5
        assert _status(lambda: ag.run(k, a, p, d, gb, sk, s2, sb)) == X.E_OUT_OF_RANGE
        assert ag.num_ops > 0 and ag.op_weights()["w"].numel() == ag.num_ops
        # a duplicate score key
        sk2 = sk.clone()
        sk2[5] = sk2[6]
        assert _status(lambda: ag.run(k, a, p, d, gb, sk2, sv, sb)) == X.E_INVALID_ARG
        # and a clean run afterwards
        r = ag.run(k, a, p, d, gb, sk, sv, sb)
        assert math.isfinite(r["score"]["s_agg"])
    finally:
        ag.close()


@pytest.mark.parametrize("A,P", [(3, 2), (100000, 3)])
def test_repeated_runs_with_pass_a_carries(A, P):
    """Pass A's carry / high-word table is cleared once at init and then by
    every pass-A reduce after reading it: three runs on one context, with
    per-(app, phase) sums far above 2^64 (64-bit LDS partials wrap; with
    100000 apps the range engine's 32-bit counters send every high word to
    the table), each give the oracle's totals and groups."""
    from oracle import oracle as O
    rng = np.random.default_rng(A)
    n = 5000
    key = (rng.integers(1, 9, n) << 16 | rng.integers(0, 5, n)).astype(np.uint32)
    app = rng.integers(0, min(A, 7), n).astype(np.uint32)
    ph = rng.integers(0, P, n).astype(np.uint8)
    dur = rng.integers(1 << 61, 1 << 62, n).astype(np.int64)
    c = rng.integers(1, 1000, A).astype(np.uint32)
    o = O.run(key, app, ph, dur, c, P)
    H.say("repeated runs with pass-A carries, A", A, "P", P)
    ag = X.Aggregator(P, _dev(c, np.int32), max_events=n, max_groups=2 * n, max_keys=n)
    try:
        gb = ag.group_buffers(2 * n)
        for _ in range(3):
            r = ag.run(_dev(key, np.int32), _dev(app, np.int32), _dev(ph, np.uint8), _dev(dur, np.int64), gb)
            T = ag.app_totals()["T"].cpu().numpy().view(np.uint64)
            assert np.array_equal(T, o["app_total"]), "app totals"
            g = r["groups"]
            assert np.array_equal(g["wsum"].cpu().numpy().view(np.uint64), o["wsum"]), "wsum"
            assert np.array_equal(g["count"].cpu().numpy().view(np.uint64), o["count"]), "count"
    finally:
        ag.close()


def _run_vs_separate(key, app, ph, dur, c, P, sk, s, path="auto", label=""):
    n = key.size
    k, a, p, d = _dev(key, np.int32), _dev(app, np.int32), _dev(ph, np.uint8), _dev(dur, np.int64)
    dc, dsk, dsv = _dev(c, np.int32), _dev(sk, np.int32), _dev(s, np.float64)
    mg = 2 * n
    ag = X.Aggregator(P, dc, max_events=n, max_groups=mg, max_keys=n, max_score=sk.size, path=path)
    try:
        res = ag.run(k, a, p, d, ag.group_buffers(mg), dsk, dsv, _score_bufs(sk.size))
        run_g = {kk: v.clone() for kk, v in res["groups"].items()}
        run_s = {kk: (v.clone() if torch.is_tensor(v) else v) for kk, v in res["score"].items()}
        counts = (ag.num_ops, ag.num_keys, ag.path_used())
        ag.reset()
        ag.aggregate(k, a, p, d)
        sep_g = ag.normalize(out=ag.group_buffers(mg))
        sep_s = ag.score(dsk, dsv)
        assert counts == (ag.num_ops, ag.num_keys, ag.path_used()), label
        for kk in sep_g:
            _same(run_g[kk], sep_g[kk], label + " " + kk)
        for kk in ("op", "op_weight", "op_score"):
            _same(run_s[kk], sep_s[kk], label + " score " + kk)
        assert run_s["s_agg"] == sep_s["s_agg"], label
        return run_g["key"].numel(), counts[2]
    finally:
        ag.close()


def test_run_more_groups_than_the_one_workgroup_unit_kernel():
    """4300 keys x 2 phases: the LDS engine orders 8600 groups in one launch,
    more than the one-workgroup unit kernel takes, so the normalisation the
    one-call path starts before the group-by's readback is dropped and
    redone by the general one."""
    rng = np.random.default_rng(7)
    n, P, A = 1 << 20, 2, 64
    keys = np.array([(1 + i // 50) << 16 | (i % 50) for i in range(4300)], np.uint32)
    key = keys[rng.integers(0, keys.size, n)]
    key[: keys.size] = keys  # every key at least once
    app = rng.integers(0, A, n).astype(np.uint32)
    ph = np.tile(np.array([0, 1], np.uint8), n // 2)
    dur = rng.integers(1, 10 ** 6, n).astype(np.int64)
    c = rng.integers(1, 1000, A).astype(np.uint32)
    s = rng.random(keys.size) * 0.9 + 0.05
    H.say("atrex_run, 8600 groups through the LDS engine")
    G, path = _run_vs_separate(key, app, ph, dur, c, P, keys, s, path="lds_hash", label="8600 groups")
    assert G == 8600 and path == "lds_hash"


def test_run_when_the_lds_engine_falls_back():
    """1M distinct keys forced through the LDS engine: the spill regions
    overflow and the group-by falls back to partitioning every event, so the
    started normalisation is dropped; atrex_run still matches the separate
    calls."""
    cfg = synth.CONFIGS[2]
    ev = synth.events(cfg, n=1 << 23)
    c = synth.app_weights(cfg)
    keys = synth.key_space(cfg)[:4096]
    s = synth.scores(cfg, keys, nan_frac=0.1)
    H.say("atrex_run, LDS engine fallback")
    G, path = _run_vs_separate(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, cfg["num_phases"], keys, s,
                               path="lds_hash", label="fallback")
    assert path == "lds_hash+radix_all"


@pytest.mark.parametrize("ci,n", [(1, 1 << 21), (0, 1 << 20), (1, (1 << 21) + 3)])
def test_one_wait_lds_path_matches_the_oracle(ci, n):
    """The exact path the benchmark times on the 64M-event workload: atrex_run
    with the capacities the benchmark gives (max_keys = the 4096-key space,
    every key scored), so AUTO takes the LDS engine and the unit, weight and
    score kernels enqueued behind the group-by are kept (one host wait).
    Every output against the oracle, element by element (§3.4 Eq. (2)-(3),
    §3.6 Eq. (4)-(6)); the 1M-event workload at its full size."""
    from oracle import oracle as O
    cfg = synth.CONFIGS[ci]
    ev = synth.events(cfg, n=n)
    c = synth.app_weights(cfg)
    keys = synth.key_space(cfg)
    s = synth.scores(cfg, keys)
    P = cfg["num_phases"]
    H.say("one-wait LDS path vs oracle, config", ci, "n", n, "keys", keys.size)
    g, one_wait, path = H.run_one_call(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P, keys, s,
                                       max_keys=keys.size, max_groups=keys.size * P)
    assert path == "lds_hash" and one_wait, (path, one_wait)
    o = O.run(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, P, score_key=keys, s=s, threads=8)
    H.compare(g, o, raw=False, score=True)


def test_one_wait_path_with_nan_scores_and_app_counts():
    """The same one-wait path with units marked incorrect (NaN) and the
    per-(app, phase) invocation counts on."""
    from oracle import oracle as O
    cfg = synth.CONFIGS[1]
    ev = synth.events(cfg, n=1 << 20)
    c = synth.app_weights(cfg)
    keys = synth.key_space(cfg)
    s = synth.scores(cfg, keys, nan_frac=0.3)
    H.say("one-wait LDS path, NaN scores, app counts")
    g, one_wait, path = H.run_one_call(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, 2, keys, s,
                                       max_keys=keys.size, max_groups=2 * keys.size, app_count=True)
    assert path == "lds_hash" and one_wait
    assert "app_n" in g
    H.compare(g, O.run(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, 2, score_key=keys, s=s, threads=8),
              raw=False, score=True)
