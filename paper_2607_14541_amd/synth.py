"""Seeded synthetic trace generator (inputs only -- no aggregation arithmetic).

The paper's weights come from production inference traces (§3.1, §3.4) that
are not public; these generators stand in for them with the same structure:
labelled kernel invocations ``(key = op << 16 | shape, app, phase, dur_ns)``,
skewed (Zipf) or uniform (operator, shape) popularity, lognormal durations,
a skewed application card-hour mix (Q16 fixed point), and per-unit roofline
achievements ``S_j`` for the score.

``CONFIGS`` holds the five workloads: 1M events / 512 keys, 64M / 4096 Zipf(1.1)
keys, 256M / 1M uniform keys, 1B / 64k Zipf(0.9) keys, and 512M adversarial
events (99% on one key, durations near 2^40).  Event counts are powers of two.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "csrc", "synth.c")
_LIB = os.path.join(_HERE, "libatrex_synth.so")


class _Cfg(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("key_mode", ctypes.c_uint32),
                ("num_ops", ctypes.c_uint32), ("num_shapes", ctypes.c_uint32),
                ("zipf_n", ctypes.c_uint32), ("shape_bits", ctypes.c_uint32),
                ("op_base", ctypes.c_uint32), ("tail_n", ctypes.c_uint32),
                ("hot_p", ctypes.c_double), ("num_phases", ctypes.c_uint32),
                ("phase0_frac", ctypes.c_double), ("num_apps", ctypes.c_uint32),
                ("dur_mode", ctypes.c_uint32), ("mu", ctypes.c_double),
                ("sigma", ctypes.c_double), ("dur_lo", ctypes.c_int64),
                ("dur_hi", ctypes.c_int64)]


CONFIGS = {
    0: dict(name="1M events, 512 uniform keys, 2 phases, 64 apps", slug="1M_uniform512", n=1 << 20, seed=0,
            key_mode=0, num_ops=32, num_shapes=16, num_phases=2, num_apps=64,
            dur_mode=0, mu=math.log(2e4), sigma=1.5, weights="uniform"),
    1: dict(name="64M events, 4096 Zipf(1.1) keys, 2 phases 60/40, 1024 apps", slug="64M_zipf4096", n=1 << 26,
            seed=1, key_mode=1, zipf_n=4096, zipf_s=1.1, shape_bits=6, num_phases=2,
            phase0_frac=0.6, num_apps=1024, dur_mode=0, mu=math.log(5e4), sigma=2.0,
            weights="zipf", weights_s=1.1),
    2: dict(name="256M events, 1M uniform keys, 4 phases, 10k apps", slug="256M_uniform1M", n=1 << 28, seed=2,
            key_mode=0, num_ops=1024, num_shapes=1024, num_phases=4, num_apps=10000,
            dur_mode=0, mu=math.log(1e4), sigma=2.5, weights="uniform"),
    3: dict(name="1B events, 64k Zipf(0.9) keys, 3 phases, 100k apps", slug="1B_zipf64k", n=1 << 30, seed=3,
            key_mode=1, zipf_n=65536, zipf_s=0.9, shape_bits=8, num_phases=3,
            num_apps=100000, dur_mode=0, mu=math.log(3e4), sigma=2.0, weights="lognormal"),
    4: dict(name="512M adversarial events, 99% on one key, durations in [2^39, 2^40]", slug="512M_adversarial",
            n=1 << 29, seed=4, key_mode=2, hot_p=0.99, tail_n=1 << 18, shape_bits=10,
            op_base=1, num_phases=2, num_apps=4, dur_mode=1, dur_lo=1 << 39,
            dur_hi=1 << 40, weights="uniform"),
}


def build(force: bool = False) -> str:
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC,
                               "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _L():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        L.atrex_synth_events.argtypes = [ctypes.POINTER(_Cfg), P, P, ctypes.c_uint64,
                                         ctypes.c_uint64, P, P, P, P]
        L.atrex_synth_events.restype = None
        L.atrex_synth_u64.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                      ctypes.c_uint64, P]
        L.atrex_synth_u64.restype = None
        L.atrex_synth_normal.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64, P]
        L.atrex_synth_normal.restype = None
        _lib = L
    return _lib


def u64_stream(seed: int, stream: int, n: int, begin: int = 0) -> np.ndarray:
    out = np.empty(n, np.uint64)
    if n:
        _L().atrex_synth_u64(seed, stream, begin, n, out.ctypes.data)
    return out


def normals(seed: int, stream: int, n: int) -> np.ndarray:
    out = np.empty(n, np.float64)
    if n:
        _L().atrex_synth_normal(seed, stream, n, out.ctypes.data)
    return out


def permutation(seed: int, stream: int, n: int) -> np.ndarray:
    """A fixed pseudo-random permutation of range(n) (sort by random keys)."""
    return np.argsort(u64_stream(seed, stream, n), kind="stable").astype(np.uint32)


def zipf_cdf(n: int, s: float) -> np.ndarray:
    """Cumulative distribution of P(rank r) proportional to r^-s, r = 1..n."""
    w = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    c = np.cumsum(w)
    c /= c[-1]
    c[-1] = 1.0
    return c


def _cfg_struct(cfg: dict) -> _Cfg:
    c = _Cfg()
    c.seed = cfg["seed"]
    c.key_mode = cfg["key_mode"]
    c.num_ops = cfg.get("num_ops", 0)
    c.num_shapes = cfg.get("num_shapes", 0)
    c.zipf_n = cfg.get("zipf_n", 0)
    c.shape_bits = cfg.get("shape_bits", 0)
    c.op_base = cfg.get("op_base", 0)
    c.tail_n = cfg.get("tail_n", 0)
    c.hot_p = cfg.get("hot_p", 0.0)
    c.num_phases = cfg["num_phases"]
    c.phase0_frac = cfg.get("phase0_frac", 0.0)
    c.num_apps = cfg["num_apps"]
    c.dur_mode = cfg.get("dur_mode", 0)
    c.mu = cfg.get("mu", 0.0)
    c.sigma = cfg.get("sigma", 0.0)
    c.dur_lo = cfg.get("dur_lo", 0)
    c.dur_hi = cfg.get("dur_hi", 0)
    return c


_tables: dict = {}


def _key_tables(cfg: dict):
    if cfg["key_mode"] != 1:
        return None, None
    k = (cfg["seed"], cfg["zipf_n"], cfg["zipf_s"])
    if k not in _tables:
        _tables[k] = (zipf_cdf(cfg["zipf_n"], cfg["zipf_s"]),
                      permutation(cfg["seed"], 100, cfg["zipf_n"]))
    return _tables[k]


def events(cfg: dict, n: int | None = None, begin: int = 0, out: dict | None = None) -> dict:
    """Events [begin, begin + n) of a workload as numpy arrays.

    ``out`` may supply preallocated arrays (e.g. pinned host buffers) with keys
    key/app/phase/dur_ns; they are filled in place.
    """
    if n is None:
        n = cfg["n"] - begin
    if out is None:
        out = dict(key=np.empty(n, np.uint32), app=np.empty(n, np.uint32),
                   phase=np.empty(n, np.uint8), dur_ns=np.empty(n, np.int64))
    for k, dt in (("key", np.uint32), ("app", np.uint32), ("phase", np.uint8),
                  ("dur_ns", np.int64)):
        a = out[k]
        assert a.dtype == dt and a.size >= n and a.flags.c_contiguous
    cdf, perm = _key_tables(cfg)
    c = _cfg_struct(cfg)
    if n:
        _L().atrex_synth_events(ctypes.byref(c),
                                cdf.ctypes.data if cdf is not None else None,
                                perm.ctypes.data if perm is not None else None,
                                begin, n, out["key"].ctypes.data, out["app"].ctypes.data,
                                out["phase"].ctypes.data, out["dur_ns"].ctypes.data)
    return out


def app_weights(cfg: dict) -> np.ndarray:
    """Q16 card-hour weights c_a (uint32), one per application."""
    A, seed = cfg["num_apps"], cfg["seed"]
    kind = cfg["weights"]
    if kind == "uniform":      # round(65536 * U[1, 1000])
        u = (u64_stream(seed, 200, A) >> np.uint64(11)).astype(np.float64) * 2.0 ** -53
        c = np.rint(65536.0 * (1.0 + 999.0 * u))
    elif kind == "zipf":       # max(1, round(65536 * 1000 * rank^-s)), ranks permuted
        rank = permutation(seed, 201, A).astype(np.float64) + 1.0
        c = np.maximum(1.0, np.rint(65536.0 * 1000.0 * rank ** (-cfg["weights_s"])))
    elif kind == "lognormal":  # clamp(round(65536 * exp(N(ln 100, 1))), 1, 2^32 - 1)
        z = normals(seed, 202, A)
        c = np.clip(np.rint(65536.0 * np.exp(math.log(100.0) + z)), 1.0, 2.0 ** 32 - 1)
    else:
        raise ValueError(kind)
    return c.astype(np.uint32)


def key_space(cfg: dict) -> np.ndarray:
    """Every (operator, shape) key the workload can emit, ascending."""
    m = cfg["key_mode"]
    if m == 0:
        op = np.repeat(np.arange(cfg["num_ops"], dtype=np.uint32), cfg["num_shapes"])
        sh = np.tile(np.arange(cfg["num_shapes"], dtype=np.uint32), cfg["num_ops"])
    elif m == 1:
        ids = np.arange(cfg["zipf_n"], dtype=np.uint32)
        op, sh = ids >> np.uint32(cfg["shape_bits"]), ids & np.uint32((1 << cfg["shape_bits"]) - 1)
    else:
        ids = np.arange(cfg["tail_n"], dtype=np.uint32)
        op = np.concatenate([[0], cfg["op_base"] + (ids >> np.uint32(cfg["shape_bits"]))])
        sh = np.concatenate([[0], ids & np.uint32((1 << cfg["shape_bits"]) - 1)])
    return np.sort(((op.astype(np.uint32) << np.uint32(16)) | sh.astype(np.uint32)).astype(np.uint32))


def scores(cfg: dict, keys: np.ndarray, nan_frac: float = 0.0) -> np.ndarray:
    """Per-unit roofline achievement S_j ~ U[0.01, 1]; a fraction marked NaN
    (unit not correct)."""
    n = keys.size
    u = (u64_stream(cfg["seed"], 300, n) >> np.uint64(11)).astype(np.float64) * 2.0 ** -53
    s = 0.01 + 0.99 * u
    if nan_frac > 0:
        v = (u64_stream(cfg["seed"], 301, n) >> np.uint64(11)).astype(np.float64) * 2.0 ** -53
        s[v < nan_frac] = np.nan
    return s


# ---------------------------------------------------------------------------
# Profiles for the target-DSL device-time share (§4.1, Metrics): the kernel
# invocations of one candidate's forward passes, labelled by (operator,
# shape) unit and by whether the kernel ran inside the target DSL.  The units
# follow the benchmark's release size (30 operators, 440 shapes) or a wide
# table; each unit has its own chance of running inside the DSL (a quarter
# never do -- delegated to library or framework kernels -- a quarter always
# do, the rest mixed), a few units record only zero-length invocations (they
# do not run), and the last operator has no running shape at all.
SHARE_CONFIGS = {
    0: dict(name="1M invocations, 440 units of 30 operators", slug="share_1M_440", n=1 << 20, seed=10,
            ops=30, shapes=440, mu=math.log(2e4), sigma=1.5),
    1: dict(name="64M invocations, 440 units of 30 operators", slug="share_64M_440", n=1 << 26, seed=11,
            ops=30, shapes=440, mu=math.log(2e4), sigma=1.5),
    2: dict(name="16M invocations, 64k units of 256 operators", slug="share_16M_64k", n=1 << 24, seed=12,
            ops=256, shapes=65536, mu=math.log(2e4), sigma=2.0),
}


def _unif(seed: int, stream: int, n: int) -> np.ndarray:
    return (u64_stream(seed, stream, n) >> np.uint64(11)).astype(np.float64) * 2.0 ** -53


def profile_units(cfg: dict) -> np.ndarray:
    """The workload's (operator, shape) keys, ascending: the shapes split as
    evenly as possible over the operators."""
    I, K = cfg["ops"], cfg["shapes"]
    per = np.full(I, K // I, np.int64)
    per[: K % I] += 1
    op = np.repeat(np.arange(I, dtype=np.uint32), per)
    sh = np.concatenate([np.arange(p, dtype=np.uint32) for p in per])
    return ((op << np.uint32(16)) | sh).astype(np.uint32)


def profile(cfg: dict, n: int | None = None) -> dict:
    """Invocations [0, n) of a profile: key, is_dsl (uint8 0/1), dur_ns."""
    n = cfg["n"] if n is None else n
    seed = cfg["seed"]
    units = profile_units(cfg)
    K = units.size
    r = _unif(seed, 400, K)
    p_dsl = np.where(r < 0.25, 0.0, np.where(r < 0.5, 1.0, _unif(seed, 401, K)))
    idle = _unif(seed, 402, K) < 0.03                 # units with zero-length invocations only
    idle |= (units >> np.uint32(16)) == cfg["ops"] - 1  # the last operator never runs
    u = u64_stream(seed, 403, n)
    idx = (u % np.uint64(K)).astype(np.int64)
    key = units[idx]
    is_dsl = (_unif(seed, 404, n) < p_dsl[idx]).astype(np.uint8)
    dur = np.rint(np.exp(cfg["mu"] + cfg["sigma"] * normals(seed, 405, n)))
    dur = np.clip(dur, 0, 2.0 ** 62).astype(np.int64)
    dur[idle[idx]] = 0
    return dict(key=key, is_dsl=is_dsl, dur_ns=dur)


# ---------------------------------------------------------------------------
# Raw trace records for the host/device correlation join (§3.1): device
# kernel records (correlation id, graph anchor, stream, start, end) and the
# host records that label them -- launch records by correlation id, graph
# records by anchor, and per-stream operator intervals for kernels that carry
# neither.  Built from a labelled workload (the labels of its events are the
# ground truth): most kernels carry their launch's correlation id, some run
# inside a captured graph (anchor only), some carry no id and fall inside
# their operator's interval, and a few match nothing.
JOIN_CONFIGS = {
    0: dict(name="1M kernel records labelled from the 1M-event workload", slug="join_1M", base=0, n=1 << 20,
            seed=20, streams=8, p_corr=0.80, p_anchor=0.10, p_time=0.08),
    1: dict(name="64M kernel records labelled from the 64M-event workload", slug="join_64M", base=1, n=1 << 26,
            seed=21, streams=32, p_corr=0.80, p_anchor=0.10, p_time=0.08),
}


def join_trace(jc: dict, n: int | None = None) -> dict:
    """kernels / host / intervals record sets and the ground-truth events."""
    n = jc["n"] if n is None else n
    seed = jc["seed"]
    ev = events(CONFIGS[jc["base"]], n=n)
    S = jc["streams"]
    u = _unif(seed, 500, n)
    c1, c2, c3 = jc["p_corr"], jc["p_corr"] + jc["p_anchor"], jc["p_corr"] + jc["p_anchor"] + jc["p_time"]
    kind = (u >= c1).astype(np.uint8) + (u >= c2) + (u >= c3)
    stream = (u64_stream(seed, 501, n) % np.uint64(S)).astype(np.uint32)
    # device timeline: each stream runs its kernels back to back with gaps of
    # 1..1000 ns (a segmented prefix sum over the kernels of each stream)
    gap = (u64_stream(seed, 502, n) % np.uint64(1000)).astype(np.int64) + 1
    order = np.argsort(stream, kind="stable")
    sp = ev["dur_ns"][order] + gap[order]
    cs = np.cumsum(sp)
    first = np.searchsorted(stream[order], np.arange(S, dtype=np.uint32))
    base = np.where(first > 0, cs[np.maximum(first - 1, 0)], 0)
    start = np.empty(n, np.int64)
    start[order] = cs - sp - base[stream[order]]
    del sp, cs, order
    end = start + ev["dur_ns"]
    # correlation ids: distinct pseudo-random values (a bijection of the index)
    corr_all = u64_stream(seed, 503, n)
    assert not np.any(corr_all == 0)
    corr = np.where(kind == 0, corr_all, np.uint64(0))
    # graph anchors, one per anchored kernel
    anchored = np.nonzero(kind == 1)[0]
    anchor = np.zeros(n, np.uint64)
    anchor[anchored] = np.arange(anchored.size, dtype=np.uint64) + np.uint64(1)
    # host records in launch order: launches of the correlated kernels, a few
    # launches whose kernels were not traced (ids that no kernel carries:
    # u64_stream of another stream), then the graph records
    hk = np.nonzero(kind == 0)[0]
    extra = hk[: max(1, hk.size // 50)]
    ex_id = u64_stream(seed, 506, extra.size) | np.uint64(1)
    h_id = np.concatenate([corr[hk], ex_id, anchor[anchored]])
    h_src = np.concatenate([hk, extra, anchored])
    h_kind = np.concatenate([np.zeros(hk.size + extra.size, np.uint8), np.ones(anchored.size, np.uint8)])
    host = dict(kind=h_kind, id=h_id, key=ev["key"][h_src], app=ev["app"][h_src], phase=ev["phase"][h_src])
    # operator intervals of the kernels matched by time: [start, end + 1), inside
    # the gap before the stream's next kernel; ascending per stream
    ti = np.nonzero(kind == 2)[0]
    ib, ie = start[ti], end[ti] + 1
    o = np.lexsort((ib, stream[ti]))
    intervals = dict(stream=stream[ti][o], begin_ns=ib[o], end_ns=ie[o], key=ev["key"][ti][o], app=ev["app"][ti][o],
                     phase=ev["phase"][ti][o])
    kernels = dict(corr=corr, anchor=anchor, stream=stream, start_ns=start, end_ns=end)
    return dict(kernels=kernels, host=host, intervals=intervals, truth=ev, kind=kind)
