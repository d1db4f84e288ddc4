"""atrex_run_noalloc (no context, no workspace, no device allocation; scratch in
a static per-GPU array) against atrex_run on the same inputs: two calls in a
row, the second smaller, every output bit for bit; sizes beyond its limits
are refused before any device work."""
import ctypes

import numpy as np
import pytest
import torch

import gpu_helpers as H
from paper_2607_14541_amd import atrex as X
from paper_2607_14541_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _d(a, dt):
    return torch.from_numpy(np.ascontiguousarray(a).view(dt)).to(DEV)


def _score_bufs(n):
    return dict(op=torch.empty(n, dtype=torch.int32, device=DEV),
                op_weight=torch.empty(n, dtype=torch.float64, device=DEV),
                op_score=torch.empty(n, dtype=torch.float64, device=DEV))


def _bits(t):
    t = t.cpu()
    return t.view(torch.int64) if t.dtype == torch.float64 else t


def _gbufs(cap, P):
    return dict(key=torch.full((cap,), -7, dtype=torch.int32, device=DEV),
                phase=torch.full((cap,), 7, dtype=torch.uint8, device=DEV),
                count=torch.full((cap,), -7, dtype=torch.int64, device=DEV),
                wsum=torch.full((cap, 2), -7, dtype=torch.int64, device=DEV),
                weight=torch.full((cap,), -7.0, dtype=torch.float64, device=DEV),
                phase_total=torch.full((P, 2), -7, dtype=torch.int64, device=DEV))


def _case(ci, n, nkeys, seed_shift=0):
    cfg = synth.CONFIGS[ci]
    ev = synth.events(cfg, n=n, begin=seed_shift)
    c = synth.app_weights(cfg)
    keys = synth.key_space(cfg)[:nkeys]
    s = synth.scores(cfg, keys, nan_frac=0.1)
    return cfg, ev, c, keys, s


def _both(ci, n, nkeys, cap, begin=0):
    cfg, ev, c, keys, s = _case(ci, n, nkeys, begin)
    P = cfg["num_phases"]
    k, a, p, d = _d(ev["key"], np.int32), _d(ev["app"], np.int32), _d(ev["phase"], np.uint8), _d(ev["dur_ns"], np.int64)
    dc, sk, sv = _d(c, np.int32), _d(keys, np.int32), _d(s, np.float64)
    ag = X.Aggregator(P, dc, max_events=n, max_groups=cap, max_keys=cap, max_score=keys.size)
    try:
        ref = ag.run(k, a, p, d, ag.group_buffers(cap), sk, sv, _score_bufs(keys.size))
        ref_counts = (ag.num_groups, ag.num_ops, ag.num_keys)
        ref = {"groups": {kk: v.clone() for kk, v in ref["groups"].items()},
               "score": {kk: (v.clone() if torch.is_tensor(v) else v) for kk, v in ref["score"].items()}}
    finally:
        ag.close()
    got = X.run_noalloc(k, a, p, d, dc, P, _gbufs(cap, P), sk, sv, _score_bufs(keys.size))
    assert (got["num_groups"], got["num_ops"], got["num_keys"]) == ref_counts
    for kk, v in ref["groups"].items():
        assert torch.equal(_bits(got["groups"][kk]), _bits(v)), kk
    for kk in ("op", "op_weight", "op_score"):
        assert torch.equal(_bits(got["score"][kk]), _bits(ref["score"][kk])), kk
    assert got["s_agg"] == ref["score"]["s_agg"]
    return got


def test_two_calls_in_a_row_match_atrex_run():
    """The second call is smaller (fewer events, keys, groups and apps) and
    must not see anything of the first one."""
    H.say("no-alloc entry, call 1: 64M-event workload prefix, 2^20 events")
    g1 = _both(1, 1 << 20, 4096, 8192)
    assert g1["num_groups"] > 4000
    H.say("no-alloc entry, call 2: 1M-event workload prefix, 2^18 + 5 events")
    g2 = _both(0, (1 << 18) + 5, 300, 1024, begin=12345)
    assert 0 < g2["num_groups"] <= 1024


def test_largest_sizes_fit_and_beyond_is_capacity():
    """At the stated limits the call fits its static array; one more event,
    group slot, scored unit or (app, phase) pair is refused with CAPACITY
    before any device work."""
    n = 1 << 24  # ATREX_NOALLOC_MAX_EVENTS
    H.say("no-alloc entry at its limits, events", n)
    rng = np.random.default_rng(3)
    A, P = 1024, 8  # 8192 (app, phase) pairs; 64 x 128 keys x 8 phases = 2^16 groups
    key = ((rng.integers(0, 64, n) << 16) | rng.integers(0, 128, n)).astype(np.uint32)
    app = rng.integers(0, A, n).astype(np.uint32)
    ph = rng.integers(0, P, n).astype(np.uint8)
    dur = rng.integers(0, 10 ** 9, n).astype(np.int64)
    c = rng.integers(1, 2 ** 20, A).astype(np.uint32)
    keys = np.unique(key)[:8192]
    s = rng.random(keys.size) * 0.9 + 0.05
    k, a, p, d = _d(key, np.int32), _d(app, np.int32), _d(ph, np.uint8), _d(dur, np.int64)
    dc, sk, sv = _d(c, np.int32), _d(keys, np.int32), _d(s, np.float64)
    cap = 1 << 16
    out = _gbufs(cap, P)
    got = X.run_noalloc(k, a, p, d, dc, P, out, sk, sv, _score_bufs(keys.size))
    assert got["num_groups"] == cap and np.isfinite(got["s_agg"])
    # beyond the limits: refused on the host (no kernel runs)
    L = X._lib()

    def status(n_ev, capacity, nsc, apps):
        prm = X._NoAllocParams(P, apps, dc.data_ptr(), torch.cuda.current_stream().cuda_stream)
        ev = X._Events(k.data_ptr(), a.data_ptr(), p.data_ptr(), d.data_ptr(), n_ev)
        g = X._Groups(*(out[kk].data_ptr() for kk in ("key", "phase", "count", "wsum", "weight", "phase_total")), 0)
        r = X._RunResult()
        return L.atrex_run_noalloc(ctypes.byref(prm), ctypes.byref(ev), ctypes.byref(g), capacity, sk.data_ptr(),
                                   sv.data_ptr(), nsc, 0, 0, 0, ctypes.byref(r))

    assert status(n + 1, cap, keys.size, A) == X.E_CAPACITY
    assert status(n, cap + 1, keys.size, A) == X.E_CAPACITY
    assert status(n, cap, 8193, A) == X.E_CAPACITY
    assert status(n, cap, keys.size, 1025) == X.E_CAPACITY  # 1025 * 8 pairs
