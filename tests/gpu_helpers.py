"""Shared helpers of the GPU parity tests: run the HIP path through the C ABI
and compare its outputs with the oracle's, element by element."""
import sys

import numpy as np
import torch

from oracle import oracle as O
from paper_2607_14541_amd import atrex as X

REL_TOL = 1e-12  # fp64 outputs (weights, S_agg); integers must match bit for bit


def say(*a):
    print("[gpu-test]", *a, flush=True)
    sys.stdout.flush()


def dev(a, dtype):
    return torch.from_numpy(np.ascontiguousarray(a).view(dtype)).cuda()


def run_gpu(key, app, phase, dur, c, P, path="auto", score_key=None, s=None, raw=True,
            max_groups=0, max_keys=0, app_count=True):
    key = np.ascontiguousarray(key, dtype=np.uint32)
    app = np.ascontiguousarray(app, dtype=np.uint32)
    phase = np.ascontiguousarray(phase, dtype=np.uint8)
    dur = np.ascontiguousarray(dur, dtype=np.int64)
    c = np.ascontiguousarray(c, dtype=np.uint32)
    args = dict(path=path, raw=raw, max_groups=max_groups, max_keys=max_keys, app_count=app_count)
    if score_key is not None:
        args["score_key"] = dev(np.asarray(score_key, np.uint32), np.int32)
        args["s"] = dev(np.asarray(s, np.float64), np.float64)
    r = X.aggregate(dev(key, np.int32), dev(app, np.int32), dev(phase, np.uint8), dev(dur, np.int64),
                    dev(c, np.int32), P, **args)
    out = {}
    for k, v in r.items():
        if isinstance(v, torch.Tensor):
            a = v.cpu().numpy()
            if a.dtype == np.int32 and k != "app_rho":  # rho is a signed exponent
                a = a.view(np.uint32)
            elif a.dtype == np.int64 and k not in ("app_rho",):
                a = a.view(np.uint64)
            out[k] = a
        else:
            out[k] = v
    out["num_groups"] = out["key"].size
    return out


def rel_err(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert a.shape == b.shape
    if a.size == 0:
        return 0.0
    zero = b == 0
    assert np.all(a[zero] == 0), "nonzero where the oracle has exactly zero"
    nz = ~zero
    return float(np.max(np.abs(a[nz] - b[nz]) / np.abs(b[nz]))) if nz.any() else 0.0


def compare(g, o, raw=True, score=False):
    assert g["num_groups"] == o["num_groups"]
    for k in ("key", "phase"):
        assert np.array_equal(g[k], o[k].astype(g[k].dtype)), k
    assert np.array_equal(g["count"], o["count"]), "count"
    assert np.array_equal(g["wsum"], o["wsum"]), "wsum"
    if raw:
        assert np.array_equal(g["raw_ns"], o["raw_ns"]), "raw_ns"
    assert np.array_equal(g["phase_total"], o["phase_total"]), "phase_total"
    assert np.array_equal(g["app_T"], o["app_total"]), "app_total"
    assert np.array_equal(g["app_mant"], o["mant"]), "mant"
    assert np.array_equal(g["app_rho"], o["rho"]), "rho"
    if "app_n" in g:  # n[a, ph] (Eq. (2)'s invocation counts) and sum_k n[k, ph] = sum_a n[a, ph]
        assert np.array_equal(g["app_n"], o["app_count"]), "app_count"
        P = g["phase_total"].shape[0]
        per_key = np.bincount(g["phase"].astype(np.int64), weights=g["count"].astype(np.float64), minlength=P)
        per_app = g["app_n"].reshape(-1, P).sum(axis=0)
        assert [int(x) for x in per_key] == [int(x) for x in per_app], "sum of counts per phase"
    assert rel_err(g["weight"], o["weight"]) <= REL_TOL, "weight"
    assert np.array_equal(g["op"], o["op"]) and np.array_equal(g["op_U"], o["op_U"]), "op U"
    assert rel_err(g["op_w"], o["op_w"]) <= REL_TOL, "op_w"
    assert np.array_equal(g["ukey"], o["ukey"]) and np.array_equal(g["key_U"], o["key_U"]), "key U"
    assert rel_err(g["omega"], o["omega"]) <= REL_TOL, "omega"
    if score:
        assert np.array_equal(g["score_op"], o["score_op"]), "score op"
        assert rel_err(g["score_op_weight"], o["score_op_weight"]) <= REL_TOL, "score w"
        assert np.array_equal(g["score_op_score"], o["score_op_S"]), "median S"
        assert abs(g["s_agg"] - o["s_agg"]) <= REL_TOL * max(abs(o["s_agg"]), 1e-300), "s_agg"


def _np_out(k, v):
    a = v.cpu().numpy()
    if a.dtype == np.int32 and k != "app_rho":  # rho is a signed exponent
        a = a.view(np.uint32)
    elif a.dtype == np.int64 and k not in ("app_rho",):
        a = a.view(np.uint64)
    return a


def run_one_call(key, app, phase, dur, c, P, score_key, s, max_keys, max_groups, max_score=None, raw=False,
                 app_count=False, path="auto"):
    """The whole path through atrex_run (one library call, as the benchmark
    times it), then the operator / key weights and app totals of the same
    context.  Inputs are numpy (uploaded here) or device tensors.  Returns
    (outputs in the layout compare() takes, one_wait flag, engine used)."""
    def up(a, dt):
        return a if isinstance(a, torch.Tensor) else dev(a, dt)
    k, a, p, d = up(key, np.int32), up(app, np.int32), up(phase, np.uint8), up(dur, np.int64)
    dc, sk, sv = up(c, np.int32), up(score_key, np.int32), up(s, np.float64)
    nsc = sk.numel()
    ag = X.Aggregator(P, dc, max_events=max(k.numel(), 1), max_groups=max_groups, max_keys=max_keys,
                      max_score=max_score or nsc, raw=raw, app_count=app_count, path=path)
    try:
        gb = ag.group_buffers(max_groups)
        sb = dict(op=torch.empty(nsc, dtype=torch.int32, device=k.device),
                  op_weight=torch.empty(nsc, dtype=torch.float64, device=k.device),
                  op_score=torch.empty(nsc, dtype=torch.float64, device=k.device))
        r = ag.run(k, a, p, d, gb, sk, sv, sb)
        out = {kk: _np_out(kk, v) for kk, v in r["groups"].items()}
        out.update({("score_" + kk): _np_out(kk, v) for kk, v in r["score"].items() if kk != "s_agg"})
        out["s_agg"] = r["score"]["s_agg"]
        out.update({("op_" + kk if kk != "op" else kk): _np_out(kk, v) for kk, v in ag.op_weights().items()})
        kw = ag.key_weights()
        out.update(ukey=_np_out("key", kw["key"]), key_U=_np_out("U", kw["U"]), omega=_np_out("omega", kw["omega"]))
        out.update({"app_" + kk: _np_out("app_" + kk, v) for kk, v in ag.app_totals().items()})
        out["num_groups"] = out["key"].size
        return out, ag.one_wait, ag.path_used()
    finally:
        ag.close()


def as_oracle_names(g):
    """GPU outputs under the names the oracle and the digests use."""
    m = {"app_T": "app_total", "app_mant": "mant", "app_rho": "rho", "app_n": "app_count"}
    return {m.get(k, k): v for k, v in g.items()}
