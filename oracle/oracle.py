"""ctypes binding of the CPU oracle (atrex_oracle*.cpp, one shared library).

TEST INFRASTRUCTURE ONLY: imported by tests/, by the smoke check and by the
benchmark's CPU-baseline leg.  The product path (the GPU library and its
binding) never imports it.

``run(...)`` executes the whole path on host arrays -- pass A, scale, pass B,
per-phase normalisation (§3.4 Eq. (2)-(3)) and, when scores are given, the
importance-weighted roofline score (§3.6 Eq. (4)-(6)) -- and returns every
intermediate as numpy arrays.  128-bit integers are returned as (lo, hi)
uint64 arrays; ``u128_to_int`` turns them into Python ints.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# every oracle source: the weighting path, and the rows built beside it
SOURCES = [os.path.join(_HERE, f) for f in ("atrex_oracle.cpp", "atrex_oracle_adoption.cpp",
                                             "atrex_oracle_stats.cpp", "atrex_oracle_join.cpp")]
_HDR = os.path.join(_HERE, "atrex_oracle.h")
# ATREX_ORACLE_SANITIZE=1: an AddressSanitizer + UndefinedBehaviorSanitizer
# build (the process must have the ASan runtime preloaded)
SANITIZE = os.environ.get("ATREX_ORACLE_SANITIZE") == "1"
_LIB = os.path.join(_HERE, "libatrex_oracle_san.so" if SANITIZE else "libatrex_oracle.so")
_SAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
              "-fno-sanitize-recover=undefined"]

OK, E_INVALID_ARG, E_OUT_OF_RANGE, E_STATE = 0, -1, -2, -3


def build(force: bool = False) -> str:
    """Compile the oracle with g++ (plain C++17, -O2; sanitized with
    ATREX_ORACLE_SANITIZE=1)."""
    newest = max(os.path.getmtime(f) for f in SOURCES + [_HDR])
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < newest:
        tmp = _LIB + ".tmp%d" % os.getpid()
        opt = _SAN_FLAGS if SANITIZE else ["-O2"]
        subprocess.check_call(["g++", *opt, "-std=c++17", "-fPIC", "-shared", "-Wall", "-pthread",
                               "-o", tmp, *SOURCES])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def library_path() -> str:
    return _LIB


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        P, U32, U64 = ctypes.c_void_p, ctypes.c_uint32, ctypes.c_uint64
        L.atrex_oracle_init.argtypes = [U32, U32, P, ctypes.POINTER(P)]
        L.atrex_oracle_aggregate_events.argtypes = [P, P, P, P, P, U64, P]
        L.atrex_oracle_aggregate_events_sharded.argtypes = [P, P, P, P, P, U64, U32, P]
        L.atrex_oracle_phase_normalize.argtypes = [P, P, P, P, P, P, P, P]
        L.atrex_oracle_app_totals.argtypes = [P, P, P, P, P]
        L.atrex_oracle_num_ops.argtypes = [P, P]
        L.atrex_oracle_op_weights.argtypes = [P, P, P, P]
        L.atrex_oracle_num_keys.argtypes = [P, P]
        L.atrex_oracle_key_weights.argtypes = [P, P, P, P]
        L.atrex_oracle_weighted_score.argtypes = [P, P, P, U64, P, P, P, P, P]
        L.atrex_oracle_destroy.argtypes = [P]
        for name in ("init", "aggregate_events", "aggregate_events_sharded", "phase_normalize", "app_totals", "num_ops",
                     "op_weights", "num_keys", "key_weights", "weighted_score"):
            getattr(L, "atrex_oracle_" + name).restype = ctypes.c_int
        L.atrex_oracle_destroy.restype = None
        # target-DSL device-time share (atrex_oracle_adoption.cpp)
        L.atrex_oracle_share_compute.argtypes = [P, P, P, U64, ctypes.POINTER(P)]
        L.atrex_oracle_share_sizes.argtypes = [P, P, P]
        L.atrex_oracle_share_keys.argtypes = [P, P, P, P, P, P]
        L.atrex_oracle_share_ops.argtypes = [P, P, P, P, P, P]
        L.atrex_oracle_share_destroy.argtypes = [P]
        L.atrex_oracle_share_destroy.restype = None
        for name in ("share_compute", "share_sizes", "share_keys", "share_ops"):
            getattr(L, "atrex_oracle_" + name).restype = ctypes.c_int
        L.atrex_oracle_exact_mean.argtypes = [P, U64]
        L.atrex_oracle_exact_mean.restype = ctypes.c_double
        # observed runtime per unit (atrex_oracle_stats.cpp)
        L.atrex_oracle_unit_stats.argtypes = [P, P, P, U64, U32, ctypes.c_int, P, U32, ctypes.POINTER(P)]
        L.atrex_oracle_stats_size.argtypes = [P, P]
        L.atrex_oracle_stats_get.argtypes = [P, P, P, P, P, P, P, P, P]
        L.atrex_oracle_stats_destroy.argtypes = [P]
        L.atrex_oracle_stats_destroy.restype = None
        for name in ("unit_stats", "stats_size", "stats_get"):
            getattr(L, "atrex_oracle_" + name).restype = ctypes.c_int
        # host/device correlation join (atrex_oracle_join.cpp)
        L.atrex_oracle_correlate.argtypes = [P] * 5 + [U64] + [P] * 5 + [U64] + [P] * 6 + [U64, ctypes.POINTER(P)]
        L.atrex_oracle_join_counts.argtypes = [P, P, P]
        L.atrex_oracle_join_get.argtypes = [P, P, P, P, P, P]
        L.atrex_oracle_join_destroy.argtypes = [P]
        L.atrex_oracle_join_destroy.restype = None
        for name in ("correlate", "join_counts", "join_get"):
            getattr(L, "atrex_oracle_" + name).restype = ctypes.c_int
        _lib = L
    return _lib


class OracleError(RuntimeError):
    def __init__(self, status: int, step: str):
        super().__init__("oracle %s returned status %d" % (step, status))
        self.status = status
        self.step = step


def _ptr(a: np.ndarray) -> ctypes.c_void_p:
    return ctypes.c_void_p(a.ctypes.data) if a.size else ctypes.c_void_p(0)


def u128_to_int(lohi: np.ndarray) -> list:
    """(n, 2) uint64 array of (lo, hi) -> list of Python ints."""
    a = np.asarray(lohi, dtype=np.uint64).reshape(-1, 2)
    return [int(lo) | (int(hi) << 64) for lo, hi in a]


def run(key, app, phase, dur_ns, app_weight_q16, num_phases, score_key=None, s=None,
        want_units: bool = True, threads: int = 1) -> dict:
    """Run the oracle end to end.  Raises OracleError on a non-OK status.
    threads > 1 splits the group-by's events over that many threads (the
    sharded form: identical results)."""
    L = lib()
    key = np.ascontiguousarray(key, dtype=np.uint32)
    app = np.ascontiguousarray(app, dtype=np.uint32)
    phase = np.ascontiguousarray(phase, dtype=np.uint8)
    dur_ns = np.ascontiguousarray(dur_ns, dtype=np.int64)
    c = np.ascontiguousarray(app_weight_q16, dtype=np.uint32)
    n = key.size
    assert app.size == n and phase.size == n and dur_ns.size == n
    P, A = int(num_phases), int(c.size)
    ctx = ctypes.c_void_p()
    st = L.atrex_oracle_init(P, A, _ptr(c), ctypes.byref(ctx))
    if st != OK:
        raise OracleError(st, "init")
    try:
        G = ctypes.c_uint64()
        if threads > 1:
            st = L.atrex_oracle_aggregate_events_sharded(ctx, _ptr(key), _ptr(app), _ptr(phase), _ptr(dur_ns),
                                                         n, int(threads), ctypes.byref(G))
        else:
            st = L.atrex_oracle_aggregate_events(ctx, _ptr(key), _ptr(app), _ptr(phase), _ptr(dur_ns),
                                                 n, ctypes.byref(G))
        if st != OK:
            raise OracleError(st, "aggregate_events")
        g = G.value
        out = {"num_groups": g}
        out["key"] = np.zeros(g, np.uint32)
        out["phase"] = np.zeros(g, np.uint8)
        out["count"] = np.zeros(g, np.uint64)
        out["wsum"] = np.zeros((g, 2), np.uint64)
        out["raw_ns"] = np.zeros((g, 2), np.uint64)
        out["weight"] = np.zeros(g, np.float64)
        out["phase_total"] = np.zeros((P, 2), np.uint64)
        AP = A * P
        out["app_total"] = np.zeros((AP, 2), np.uint64)
        out["app_count"] = np.zeros(AP, np.uint64)
        out["mant"] = np.zeros(AP, np.uint64)
        out["rho"] = np.zeros(AP, np.int32)
        st = L.atrex_oracle_app_totals(ctx, _ptr(out["app_total"]), _ptr(out["app_count"]),
                                       _ptr(out["mant"]), _ptr(out["rho"]))
        if st != OK:
            raise OracleError(st, "app_totals")
        st = L.atrex_oracle_phase_normalize(ctx, _ptr(out["key"]), _ptr(out["phase"]),
                                            _ptr(out["count"]), _ptr(out["wsum"]),
                                            _ptr(out["raw_ns"]), _ptr(out["weight"]),
                                            _ptr(out["phase_total"]))
        if st != OK:
            raise OracleError(st, "phase_normalize")
        if want_units:
            cnt = ctypes.c_uint64()
            L.atrex_oracle_num_ops(ctx, ctypes.byref(cnt))
            k = cnt.value
            out["op"] = np.zeros(k, np.uint32)
            out["op_U"] = np.zeros((k, 2), np.uint64)
            out["op_w"] = np.zeros(k, np.float64)
            if k:
                L.atrex_oracle_op_weights(ctx, _ptr(out["op"]), _ptr(out["op_U"]), _ptr(out["op_w"]))
            L.atrex_oracle_num_keys(ctx, ctypes.byref(cnt))
            k = cnt.value
            out["ukey"] = np.zeros(k, np.uint32)
            out["key_U"] = np.zeros((k, 2), np.uint64)
            out["omega"] = np.zeros(k, np.float64)
            if k:
                L.atrex_oracle_key_weights(ctx, _ptr(out["ukey"]), _ptr(out["key_U"]),
                                           _ptr(out["omega"]))
        if score_key is not None:
            sk = np.ascontiguousarray(score_key, dtype=np.uint32)
            sv = np.ascontiguousarray(s, dtype=np.float64)
            assert sk.size == sv.size
            nsc = sk.size
            nops = ctypes.c_uint64()
            sc_op = np.zeros(max(nsc, 1), np.uint32)
            sc_w = np.zeros(max(nsc, 1), np.float64)
            sc_s = np.zeros(max(nsc, 1), np.float64)
            sagg = ctypes.c_double()
            st = L.atrex_oracle_weighted_score(ctx, _ptr(sk), _ptr(sv), nsc, ctypes.byref(nops),
                                               _ptr(sc_op), _ptr(sc_w), _ptr(sc_s),
                                               ctypes.byref(sagg))
            if st != OK:
                raise OracleError(st, "weighted_score")
            k = nops.value
            out["score_op"] = sc_op[:k].copy()
            out["score_op_weight"] = sc_w[:k].copy()
            out["score_op_S"] = sc_s[:k].copy()
            out["s_agg"] = sagg.value
        return out
    finally:
        L.atrex_oracle_destroy(ctx)


def status_of(key, app, phase, dur_ns, app_weight_q16, num_phases, score_key=None, s=None) -> int:
    """Status code of the first failing step (OK when every step succeeds)."""
    try:
        run(key, app, phase, dur_ns, app_weight_q16, num_phases, score_key, s, want_units=False)
    except OracleError as e:
        return e.status
    return OK


def exact_mean(x) -> float:
    """The oracle's exact mean of finite non-negative doubles, rounded once."""
    a = np.ascontiguousarray(x, dtype=np.float64)
    return lib().atrex_oracle_exact_mean(_ptr(a), a.size)


def target_share(key, is_dsl, dur_ns) -> dict:
    """Target-DSL device-time share of one profile (§4.1, Metrics): per key
    the DSL and total device time and their ratio, per operator the exact mean
    over its running shapes, and the mean over the operators where defined.
    Raises OracleError on a non-OK status."""
    L = lib()
    key = np.ascontiguousarray(key, dtype=np.uint32)
    flag = np.ascontiguousarray(is_dsl, dtype=np.uint8)
    dur_ns = np.ascontiguousarray(dur_ns, dtype=np.int64)
    n = key.size
    assert flag.size == n and dur_ns.size == n
    h = ctypes.c_void_p()
    st = L.atrex_oracle_share_compute(_ptr(key), _ptr(flag), _ptr(dur_ns), n, ctypes.byref(h))
    if st != OK:
        raise OracleError(st, "share_compute")
    try:
        nk, no = ctypes.c_uint64(), ctypes.c_uint64()
        L.atrex_oracle_share_sizes(h, ctypes.byref(nk), ctypes.byref(no))
        K, I = nk.value, no.value
        out = {"key": np.zeros(K, np.uint32), "count": np.zeros(K, np.uint64),
               "dsl_ns": np.zeros((K, 2), np.uint64), "total_ns": np.zeros((K, 2), np.uint64),
               "share": np.zeros(K, np.float64), "op": np.zeros(I, np.uint32),
               "op_shapes": np.zeros(I, np.uint32), "op_share": np.zeros(I, np.float64)}
        st = L.atrex_oracle_share_keys(h, _ptr(out["key"]), _ptr(out["count"]), _ptr(out["dsl_ns"]),
                                       _ptr(out["total_ns"]), _ptr(out["share"]))
        if st != OK:
            raise OracleError(st, "share_keys")
        adop, nd = ctypes.c_double(), ctypes.c_uint64()
        st = L.atrex_oracle_share_ops(h, _ptr(out["op"]), _ptr(out["op_shapes"]), _ptr(out["op_share"]),
                                      ctypes.byref(adop), ctypes.byref(nd))
        if st != OK:
            raise OracleError(st, "share_ops")
        out["adoption"] = adop.value
        out["defined_ops"] = nd.value
        return out
    finally:
        L.atrex_oracle_share_destroy(h)


def unit_stats(key, phase, dur_ns, num_phases, q_1e5=(50000, 99000), by_phase=True) -> dict:
    """Observed runtime per unit (§3.1, the deployment baseline): count,
    total, mean, min, max and nearest-rank quantiles (q_1e5: q in 1e-5
    steps).  Raises OracleError on a non-OK status."""
    L = lib()
    key = np.ascontiguousarray(key, dtype=np.uint32)
    phase = np.ascontiguousarray(phase, dtype=np.uint8)
    dur_ns = np.ascontiguousarray(dur_ns, dtype=np.int64)
    q = np.ascontiguousarray(q_1e5, dtype=np.uint32)
    n = key.size
    assert phase.size == n and dur_ns.size == n
    h = ctypes.c_void_p()
    st = L.atrex_oracle_unit_stats(_ptr(key), _ptr(phase), _ptr(dur_ns), n, int(num_phases), int(bool(by_phase)),
                                   _ptr(q), q.size, ctypes.byref(h))
    if st != OK:
        raise OracleError(st, "unit_stats")
    try:
        nu = ctypes.c_uint64()
        L.atrex_oracle_stats_size(h, ctypes.byref(nu))
        U = nu.value
        out = {"key": np.zeros(U, np.uint32), "phase": np.zeros(U, np.uint8), "count": np.zeros(U, np.uint64),
               "total_ns": np.zeros((U, 2), np.uint64), "mean_ns": np.zeros(U, np.float64),
               "min_ns": np.zeros(U, np.int64), "max_ns": np.zeros(U, np.int64),
               "quantile_ns": np.zeros((U, q.size), np.int64)}
        st = L.atrex_oracle_stats_get(h, *(_ptr(out[k]) for k in ("key", "phase", "count", "total_ns", "mean_ns",
                                                                   "min_ns", "max_ns", "quantile_ns")))
        if st != OK:
            raise OracleError(st, "stats_get")
        return out
    finally:
        L.atrex_oracle_stats_destroy(h)


def correlate(kernels: dict, host: dict, intervals: dict | None = None) -> dict:
    """Host/device correlation join (§3.1).  kernels: corr, anchor, stream,
    start_ns, end_ns; host: kind, id, key, app, phase; intervals: stream,
    begin_ns, end_ns, key, app, phase.  Returns the labelled events (kernel
    order), the per-kernel source (0 corr, 1 anchor, 2 interval, 3 none) and
    the counts.  Raises OracleError on a non-OK status."""
    L = lib()
    K = {k: np.ascontiguousarray(kernels[k], dt) for k, dt in
         (("corr", np.uint64), ("anchor", np.uint64), ("stream", np.uint32), ("start_ns", np.int64),
          ("end_ns", np.int64))}
    H = {k: np.ascontiguousarray(host[k], dt) for k, dt in
         (("kind", np.uint8), ("id", np.uint64), ("key", np.uint32), ("app", np.uint32), ("phase", np.uint8))}
    iv = intervals or {k: [] for k in ("stream", "begin_ns", "end_ns", "key", "app", "phase")}
    I = {k: np.ascontiguousarray(iv[k], dt) for k, dt in
         (("stream", np.uint32), ("begin_ns", np.int64), ("end_ns", np.int64), ("key", np.uint32),
          ("app", np.uint32), ("phase", np.uint8))}
    n, m, mi = K["corr"].size, H["kind"].size, I["stream"].size
    h = ctypes.c_void_p()
    st = L.atrex_oracle_correlate(*(_ptr(K[k]) for k in ("corr", "anchor", "stream", "start_ns", "end_ns")), n,
                                  *(_ptr(H[k]) for k in ("kind", "id", "key", "app", "phase")), m,
                                  *(_ptr(I[k]) for k in ("stream", "begin_ns", "end_ns", "key", "app", "phase")), mi,
                                  ctypes.byref(h))
    if st != OK:
        raise OracleError(st, "correlate")
    try:
        lab = ctypes.c_uint64()
        by = np.zeros(4, np.uint64)
        L.atrex_oracle_join_counts(h, ctypes.byref(lab), _ptr(by))
        nl = lab.value
        out = {"key": np.zeros(nl, np.uint32), "app": np.zeros(nl, np.uint32), "phase": np.zeros(nl, np.uint8),
               "dur_ns": np.zeros(nl, np.int64), "source": np.zeros(n, np.uint8)}
        st = L.atrex_oracle_join_get(h, *(_ptr(out[k]) for k in ("key", "app", "phase", "dur_ns", "source")))
        if st != OK:
            raise OracleError(st, "join_get")
        out["by_source"] = by
        out["labelled"] = nl
        return out
    finally:
        L.atrex_oracle_join_destroy(h)
