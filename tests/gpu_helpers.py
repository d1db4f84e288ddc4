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
            max_groups=0, max_keys=0):
    key = np.ascontiguousarray(key, dtype=np.uint32)
    app = np.ascontiguousarray(app, dtype=np.uint32)
    phase = np.ascontiguousarray(phase, dtype=np.uint8)
    dur = np.ascontiguousarray(dur, dtype=np.int64)
    c = np.ascontiguousarray(c, dtype=np.uint32)
    args = dict(path=path, raw=raw, max_groups=max_groups, max_keys=max_keys)
    if score_key is not None:
        args["score_key"] = dev(np.asarray(score_key, np.uint32), np.int32)
        args["s"] = dev(np.asarray(s, np.float64), np.float64)
    r = X.aggregate(dev(key, np.int32), dev(app, np.int32), dev(phase, np.uint8), dev(dur, np.int64),
                    dev(c, np.int32), P, **args)
    out = {}
    for k, v in r.items():
        if isinstance(v, torch.Tensor):
            a = v.cpu().numpy()
            if a.dtype == np.int32:
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
