"""Python binding of libatrex.so (C ABI in include/atrex.h).

Argument marshalling only: every step of the path runs in the library's gfx950
kernels.  PyTorch provides device memory (caller-owned tensors, including the
library's workspace) and the HIP stream.  The library must be built
(``python -m paper_2607_14541_amd.build``); there is no fallback.

Type mapping: uint32 arrays travel as torch.int32, uint64 and 128-bit (lo, hi)
pairs as torch.int64 (bit patterns unchanged), fp64 as torch.float64.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libatrex.so")

OK, E_INVALID_ARG, E_OUT_OF_RANGE, E_STATE, E_CAPACITY, E_DEVICE = 0, -1, -2, -3, -4, -5
PATHS = {"auto": 0, "lds_hash": 1, "global_hash": 2, "radix_sort": 3}
FLAG_TIMING, FLAG_RAW, FLAG_APP_COUNT, FLAG_DEVICE_TIME, FLAG_INCREMENTAL = 1, 2, 4, 8, 16


class AtrexError(RuntimeError):
    def __init__(self, status: int, call: str):
        msg = _lib().atrex_status_str(status).decode() if _LIB is not None else str(status)
        super().__init__("%s failed: %s (%d)" % (call, msg, status))
        self.status = status
        self.call = call


class _InitParams(ctypes.Structure):
    _fields_ = [("num_phases", ctypes.c_uint32), ("num_apps", ctypes.c_uint32),
                ("app_weight_q16", ctypes.c_void_p), ("max_events", ctypes.c_uint64),
                ("max_groups", ctypes.c_uint64), ("max_keys", ctypes.c_uint64),
                ("max_score", ctypes.c_uint64), ("path", ctypes.c_int),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
                ("stream", ctypes.c_void_p), ("flags", ctypes.c_uint32)]


class _Events(ctypes.Structure):
    _fields_ = [("key", ctypes.c_void_p), ("app", ctypes.c_void_p), ("phase", ctypes.c_void_p),
                ("dur_ns", ctypes.c_void_p), ("n", ctypes.c_uint64)]


class _Groups(ctypes.Structure):
    _fields_ = [("key", ctypes.c_void_p), ("phase", ctypes.c_void_p), ("count", ctypes.c_void_p),
                ("wsum", ctypes.c_void_p), ("weight", ctypes.c_void_p),
                ("phase_total", ctypes.c_void_p), ("raw_ns", ctypes.c_void_p)]


class _NoAllocParams(ctypes.Structure):
    _fields_ = [("num_phases", ctypes.c_uint32), ("num_apps", ctypes.c_uint32),
                ("app_weight_q16", ctypes.c_void_p), ("stream", ctypes.c_void_p)]


class _ShareOut(ctypes.Structure):
    _fields_ = [("key", ctypes.c_void_p), ("count", ctypes.c_void_p), ("dsl_ns", ctypes.c_void_p),
                ("total_ns", ctypes.c_void_p), ("share", ctypes.c_void_p), ("op", ctypes.c_void_p),
                ("op_shapes", ctypes.c_void_p), ("op_share", ctypes.c_void_p)]


class _StatsOut(ctypes.Structure):
    _fields_ = [("key", ctypes.c_void_p), ("phase", ctypes.c_void_p), ("count", ctypes.c_void_p),
                ("total_ns", ctypes.c_void_p), ("mean_ns", ctypes.c_void_p), ("min_ns", ctypes.c_void_p),
                ("max_ns", ctypes.c_void_p), ("quantile_ns", ctypes.c_void_p)]


class _KernelRecords(ctypes.Structure):
    _fields_ = [("corr", ctypes.c_void_p), ("anchor", ctypes.c_void_p), ("stream", ctypes.c_void_p),
                ("start_ns", ctypes.c_void_p), ("end_ns", ctypes.c_void_p), ("n", ctypes.c_uint64)]


class _HostRecords(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_void_p), ("id", ctypes.c_void_p), ("key", ctypes.c_void_p),
                ("app", ctypes.c_void_p), ("phase", ctypes.c_void_p), ("n", ctypes.c_uint64)]


class _IntervalRecords(ctypes.Structure):
    _fields_ = [("stream", ctypes.c_void_p), ("begin_ns", ctypes.c_void_p), ("end_ns", ctypes.c_void_p),
                ("key", ctypes.c_void_p), ("app", ctypes.c_void_p), ("phase", ctypes.c_void_p),
                ("n", ctypes.c_uint64)]


class _EventOut(ctypes.Structure):
    _fields_ = [("key", ctypes.c_void_p), ("app", ctypes.c_void_p), ("phase", ctypes.c_void_p),
                ("dur_ns", ctypes.c_void_p)]


class _JoinParams(ctypes.Structure):
    _fields_ = [("max_kernels", ctypes.c_uint64), ("max_host", ctypes.c_uint64), ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_size_t), ("stream", ctypes.c_void_p), ("method", ctypes.c_uint32)]


class _JoinResult(ctypes.Structure):
    _fields_ = [("labelled", ctypes.c_uint64), ("by_source", ctypes.c_uint64 * 4), ("method_used", ctypes.c_uint32)]


JOIN_METHODS = {"auto": 0, "hash": 1, "partition": 2}


class _ShareResult(ctypes.Structure):
    _fields_ = [("num_keys", ctypes.c_uint64), ("num_ops", ctypes.c_uint64), ("defined_ops", ctypes.c_uint64),
                ("adoption", ctypes.c_double)]


class _RunResult(ctypes.Structure):
    _fields_ = [("num_groups", ctypes.c_uint64), ("num_ops", ctypes.c_uint64), ("num_keys", ctypes.c_uint64),
                ("num_scored_ops", ctypes.c_uint64), ("s_agg", ctypes.c_double), ("one_wait", ctypes.c_uint32)]


_LIB = None


def _lib() -> ctypes.CDLL:
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libatrex.so is not built (%s); run: python -m paper_2607_14541_amd.build"
                               % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        P, U64, I = ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int
        sigs = {
            "atrex_workspace_bytes": [ctypes.POINTER(_InitParams), ctypes.POINTER(ctypes.c_size_t)],
            "atrex_aggregate_init": [ctypes.POINTER(_InitParams), ctypes.POINTER(P)],
            "atrex_aggregate_events": [P, ctypes.POINTER(_Events), ctypes.POINTER(U64)],
            "atrex_phase_normalize": [P, ctypes.POINTER(_Groups), ctypes.POINTER(U64), ctypes.POINTER(U64)],
            "atrex_op_weights": [P, P, P, P],
            "atrex_key_weights": [P, P, P, P],
            "atrex_weighted_score": [P, P, P, U64, P, P, P, ctypes.POINTER(U64),
                                     ctypes.POINTER(ctypes.c_double)],
            "atrex_run": [P, ctypes.POINTER(_Events), ctypes.POINTER(_Groups), U64, P, P, U64, P, P, P,
                          ctypes.POINTER(_RunResult)],
            "atrex_run_noalloc": [ctypes.POINTER(_NoAllocParams), ctypes.POINTER(_Events), ctypes.POINTER(_Groups),
                                  U64, P, P, U64, P, P, P, ctypes.POINTER(_RunResult)],
            "atrex_get_app_totals": [P, P, P, P, P],
            "atrex_target_share": [P, ctypes.POINTER(_ShareOut), U64, U64, ctypes.POINTER(_ShareResult)],
            "atrex_refresh": [P, ctypes.POINTER(_Events), U64, ctypes.POINTER(U64)],
            "atrex_join_workspace_bytes": [ctypes.POINTER(_JoinParams), ctypes.POINTER(ctypes.c_size_t)],
            "atrex_correlate": [ctypes.POINTER(_JoinParams), ctypes.POINTER(_KernelRecords),
                                ctypes.POINTER(_HostRecords), ctypes.POINTER(_IntervalRecords),
                                ctypes.POINTER(_EventOut), U64, P, ctypes.POINTER(_JoinResult)],
            "atrex_unit_stats": [P, ctypes.POINTER(_Events), I, P, ctypes.c_uint32, ctypes.POINTER(_StatsOut), U64,
                                 ctypes.POINTER(U64)],
            "atrex_refresh_state": [P, P, P, ctypes.POINTER(U64)],
            "atrex_refresh_restore": [P, P, P, U64],
            "atrex_kernel_times": [P, ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_float),
                                   ctypes.POINTER(U64), I, ctypes.POINTER(I)],
            "atrex_aggregate_reset": [P],
            "atrex_aggregate_destroy": [P],
        }
        for name, args in sigs.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = ctypes.c_int
        L.atrex_status_str.argtypes = [ctypes.c_int]
        L.atrex_status_str.restype = ctypes.c_char_p
        L.atrex_path_used.argtypes = [P]
        L.atrex_path_used.restype = ctypes.c_char_p
        _LIB = L
    return _LIB


def _ptr(t) -> ctypes.c_void_p:
    return ctypes.c_void_p(t.data_ptr()) if t is not None and t.numel() else ctypes.c_void_p(0)


def _check(st: int, call: str) -> None:
    if st != OK:
        raise AtrexError(st, call)


def _dev(t: torch.Tensor, dtype: torch.dtype, name: str) -> torch.Tensor:
    if not t.is_cuda:
        raise ValueError("%s must be a device tensor" % name)
    if t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    return t.contiguous()


def _same_items(d: dict, items: tuple) -> bool:
    """d still maps the same keys to the same objects as `items`."""
    return len(d) == len(items) and all(d.get(k) is v for k, v in items)


def _as_i32(t: torch.Tensor) -> torch.Tensor:
    """uint32 data as int32 bits."""
    if t.dtype == torch.int32:
        return t
    if t.dtype == getattr(torch, "uint32", None):
        return t.view(torch.int32)
    if t.dtype == torch.int64:
        return t.to(torch.int32)  # callers pass values < 2^31 here
    raise TypeError("expected 32-bit integer tensor, got %s" % t.dtype)


class Aggregator:
    """One aggregation context: init -> aggregate -> normalize -> weights/score.

    device_time=True: the plain device-time group-by (ATREX_FLAG_DEVICE_TIME):
    no applications (app_weight_q16 is ignored and may be None; aggregate()
    takes app=None), W = sum of dur per (key, phase); with num_phases = 2 it
    feeds target_share().

    incremental=True: the events form an append-only log (ATREX_FLAG_INCREMENTAL);
    refresh() folds the events added since the last one."""

    def __init__(self, num_phases: int, app_weight_q16: torch.Tensor | None, max_events: int,
                 max_groups: int = 0, max_keys: int = 0, max_score: int = 0, path: str = "auto",
                 timing: bool = False, raw: bool = False, app_count: bool = False,
                 stream: torch.cuda.Stream | None = None, device_time: bool = False,
                 device: torch.device | None = None, incremental: bool = False):
        L = _lib()
        self.device_time = device_time
        if device_time:
            c = None
            self.device = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
            self.A = 1
        else:
            c = _dev(_as_i32(app_weight_q16), torch.int32, "app_weight_q16")
            self.device = c.device
            self.A = int(c.numel())
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.P = int(num_phases)
        self.raw = raw
        self.app_count = app_count or device_time or incremental  # these modes always count
        p = _InitParams()
        p.num_phases, p.num_apps = self.P, self.A
        p.app_weight_q16 = c.data_ptr() if c is not None else None
        p.max_events, p.max_groups, p.max_keys, p.max_score = max_events, max_groups, max_keys, max_score
        p.path = PATHS[path]
        p.stream = self.stream.cuda_stream
        p.flags = ((FLAG_TIMING if timing else 0) | (FLAG_RAW if raw else 0) | (FLAG_APP_COUNT if app_count else 0)
                   | (FLAG_DEVICE_TIME if device_time else 0) | (FLAG_INCREMENTAL if incremental else 0))
        nbytes = ctypes.c_size_t()
        _check(L.atrex_workspace_bytes(ctypes.byref(p), ctypes.byref(nbytes)), "atrex_workspace_bytes")
        self.workspace = torch.empty(max(int(nbytes.value), 256), dtype=torch.uint8, device=self.device)
        p.workspace, p.workspace_bytes = self.workspace.data_ptr(), self.workspace.numel()
        self._app_weight = c
        ctx = ctypes.c_void_p()
        _check(L.atrex_aggregate_init(ctypes.byref(p), ctypes.byref(ctx)), "atrex_aggregate_init")
        self._ctx = ctx
        self.num_groups = None
        self.num_ops = self.num_keys = None
        self.one_wait = None
        # marshalled arguments of the last normalize()/score() call, reused
        # while the caller passes the same output tensors (and sizes) again
        self._gcache = None
        self._scache = None
        self._rviews = self._sviews = None

    # -- Eq. (2)-(3) group-by ---------------------------------------------------------
    def aggregate(self, key: torch.Tensor, app: torch.Tensor | None, phase: torch.Tensor,
                  dur_ns: torch.Tensor) -> int:
        key = _dev(_as_i32(key), torch.int32, "key")
        app = _dev(_as_i32(app), torch.int32, "app") if app is not None else None
        phase = _dev(phase, torch.uint8, "phase")
        dur_ns = _dev(dur_ns, torch.int64, "dur_ns")
        n = key.numel()
        if not ((app is None or app.numel() == n) and phase.numel() == n and dur_ns.numel() == n):
            raise ValueError("event arrays differ in length")
        self._events = (key, app, phase, dur_ns)  # keep alive for the call
        ev = _Events(_ptr(key), _ptr(app), _ptr(phase), _ptr(dur_ns), n)
        G = ctypes.c_uint64()
        _check(_lib().atrex_aggregate_events(self._ctx, ctypes.byref(ev), ctypes.byref(G)),
               "atrex_aggregate_events")
        self._events = None
        self.num_groups = G.value
        return self.num_groups

    def refresh(self, key: torch.Tensor, app: torch.Tensor, phase: torch.Tensor, dur_ns: torch.Tensor,
                n_new: int) -> int:
        """Incremental refresh (incremental=True): the tensors hold the whole
        log, whose last n_new events are new since the last refresh; the
        results equal a group-by of the whole log.  Returns the group count."""
        key = _dev(_as_i32(key), torch.int32, "key")
        app = _dev(_as_i32(app), torch.int32, "app")
        phase = _dev(phase, torch.uint8, "phase")
        dur_ns = _dev(dur_ns, torch.int64, "dur_ns")
        n = key.numel()
        if not (app.numel() == n and phase.numel() == n and dur_ns.numel() == n):
            raise ValueError("event arrays differ in length")
        self._events = (key, app, phase, dur_ns)
        ev = _Events(_ptr(key), _ptr(app), _ptr(phase), _ptr(dur_ns), n)
        G = ctypes.c_uint64()
        _check(_lib().atrex_refresh(self._ctx, ctypes.byref(ev), int(n_new), ctypes.byref(G)), "atrex_refresh")
        self._events = None
        self.num_groups = G.value
        return self.num_groups

    def refresh_state(self) -> dict:
        """The folded per-(app, phase) totals T, counts n and n_folded."""
        GA, dev = self.A * self.P, self.device
        T = torch.empty((GA, 2), dtype=torch.int64, device=dev)
        n = torch.empty(GA, dtype=torch.int64, device=dev)
        nf = ctypes.c_uint64()
        _check(_lib().atrex_refresh_state(self._ctx, _ptr(T), _ptr(n), ctypes.byref(nf)), "atrex_refresh_state")
        return dict(T=T, n=n, n_folded=nf.value)

    def refresh_restore(self, state: dict) -> None:
        """Resume from refresh_state() of a context with the same parameters."""
        _check(_lib().atrex_refresh_restore(self._ctx, _ptr(state["T"].contiguous()), _ptr(state["n"].contiguous()),
                                            int(state["n_folded"])), "atrex_refresh_restore")

    def reset(self) -> None:
        """Back to the initialised state: the next batch reuses the workspace."""
        _check(_lib().atrex_aggregate_reset(self._ctx), "atrex_aggregate_reset")
        self.num_groups = self.num_ops = self.num_keys = None

    def group_buffers(self, capacity: int) -> dict:
        """Output tensors for normalize() with room for `capacity` groups."""
        dev = self.device
        out = dict(key=torch.empty(capacity, dtype=torch.int32, device=dev),
                   phase=torch.empty(capacity, dtype=torch.uint8, device=dev),
                   count=torch.empty(capacity, dtype=torch.int64, device=dev),
                   wsum=torch.empty((capacity, 2), dtype=torch.int64, device=dev),
                   weight=torch.empty(capacity, dtype=torch.float64, device=dev),
                   phase_total=torch.empty((self.P, 2), dtype=torch.int64, device=dev))
        if self.raw:
            out["raw_ns"] = torch.empty((capacity, 2), dtype=torch.int64, device=dev)
        return out

    def normalize(self, out: dict | None = None) -> dict:
        G = self.num_groups
        if out is None:
            out = self.group_buffers(G)
        c = self._gcache
        if c is None or c[0] is not out or c[1] != G or not _same_items(out, c[2]):
            if out["key"].numel() < G:
                raise ValueError("output buffers hold %d groups, need %d" % (out["key"].numel(), G))
            g = _Groups(_ptr(out["key"]), _ptr(out["phase"]), _ptr(out["count"]), _ptr(out["wsum"]),
                        _ptr(out["weight"]), _ptr(out["phase_total"]), _ptr(out.get("raw_ns")))
            views = {k: (v if k == "phase_total" else v[:G]) for k, v in out.items()}
            c = self._gcache = (out, G, tuple(out.items()), g, views)
        nops, nkeys = ctypes.c_uint64(), ctypes.c_uint64()
        _check(_lib().atrex_phase_normalize(self._ctx, ctypes.byref(c[3]), ctypes.byref(nops),
                                            ctypes.byref(nkeys)), "atrex_phase_normalize")
        self.num_ops, self.num_keys = nops.value, nkeys.value
        return dict(c[4])

    def run(self, key: torch.Tensor, app: torch.Tensor, phase: torch.Tensor, dur_ns: torch.Tensor,
            out: dict, score_key: torch.Tensor | None = None, s: torch.Tensor | None = None,
            score_out: dict | None = None) -> dict:
        """reset + aggregate + normalize (+ score when score_key, s are given) in
        one library call (atrex_run): the same results as the calls one by one.
        `out` comes from group_buffers(); `score_out` holds op / op_weight /
        op_score tensors of at least len(score_key) entries."""
        key = _dev(_as_i32(key), torch.int32, "key")
        app = _dev(_as_i32(app), torch.int32, "app")
        phase = _dev(phase, torch.uint8, "phase")
        dur_ns = _dev(dur_ns, torch.int64, "dur_ns")
        n = key.numel()
        if not (app.numel() == n and phase.numel() == n and dur_ns.numel() == n):
            raise ValueError("event arrays differ in length")
        ev = _Events(_ptr(key), _ptr(app), _ptr(phase), _ptr(dur_ns), n)
        c = self._gcache
        if c is None or c[0] is not out or c[1] != -1 or not _same_items(out, c[2]):
            g = _Groups(_ptr(out["key"]), _ptr(out["phase"]), _ptr(out["count"]), _ptr(out["wsum"]),
                        _ptr(out["weight"]), _ptr(out["phase_total"]), _ptr(out.get("raw_ns")))
            c = self._gcache = (out, -1, tuple(out.items()), g, None)
        nsc, sp = 0, (ctypes.c_void_p(0),) * 5
        if score_key is not None:
            score_key = _dev(_as_i32(score_key), torch.int32, "score_key")
            s = _dev(s, torch.float64, "s")
            nsc = score_key.numel()
            if s.numel() != nsc:
                raise ValueError("score_key and s differ in length")
            if any(score_out[k].numel() < nsc for k in ("op", "op_weight", "op_score")):
                raise ValueError("score output buffers too small")
            sp = (_ptr(score_key), _ptr(s), _ptr(score_out["op"]), _ptr(score_out["op_weight"]),
                  _ptr(score_out["op_score"]))
        r = _RunResult()
        st = _lib().atrex_run(self._ctx, ctypes.byref(ev), ctypes.byref(c[3]), out["key"].numel(), sp[0], sp[1],
                              nsc, sp[2], sp[3], sp[4], ctypes.byref(r))
        # counts of the stages that completed (as after the separate calls)
        self.num_groups, self.num_ops, self.num_keys = r.num_groups, r.num_ops, r.num_keys
        self.one_wait = bool(r.one_wait)
        _check(st, "atrex_run")
        G, k = r.num_groups, r.num_scored_ops
        v = self._rviews  # views of the first G groups / k operators, kept while they stay the same
        if v is None or v[0] is not out or v[1] != G:
            v = self._rviews = (out, G, {kk: (t if kk == "phase_total" else t[:G]) for kk, t in out.items()})
        res = {"groups": dict(v[2])}
        if score_key is not None:
            w = self._sviews
            if w is None or w[0] is not score_out or w[1] != k:
                w = self._sviews = (score_out, k, {kk: score_out[kk][:k] for kk in ("op", "op_weight", "op_score")})
            res["score"] = dict(w[2], s_agg=r.s_agg)
        return res

    def op_weights(self) -> dict:
        k, dev = self.num_ops, self.device
        op = torch.empty(k, dtype=torch.int32, device=dev)
        U = torch.empty((k, 2), dtype=torch.int64, device=dev)
        w = torch.empty(k, dtype=torch.float64, device=dev)
        _check(_lib().atrex_op_weights(self._ctx, _ptr(op), _ptr(U), _ptr(w)), "atrex_op_weights")
        return dict(op=op, U=U, w=w)

    def key_weights(self) -> dict:
        k, dev = self.num_keys, self.device
        key = torch.empty(k, dtype=torch.int32, device=dev)
        U = torch.empty((k, 2), dtype=torch.int64, device=dev)
        w = torch.empty(k, dtype=torch.float64, device=dev)
        _check(_lib().atrex_key_weights(self._ctx, _ptr(key), _ptr(U), _ptr(w)), "atrex_key_weights")
        return dict(key=key, U=U, omega=w)

    # -- Eq. (4)-(6) ---------------------------------------------------------------------
    def score(self, score_key: torch.Tensor, s: torch.Tensor, out: dict | None = None) -> dict:
        score_key = _dev(_as_i32(score_key), torch.int32, "score_key")
        s = _dev(s, torch.float64, "s")
        n = score_key.numel()
        if s.numel() != n:
            raise ValueError("score_key and s differ in length")
        dev = self.device
        if out is None:
            out = dict(op=torch.empty(max(n, 1), dtype=torch.int32, device=dev),
                       op_weight=torch.empty(max(n, 1), dtype=torch.float64, device=dev),
                       op_score=torch.empty(max(n, 1), dtype=torch.float64, device=dev))
        c = self._scache
        if c is None or c[0] is not out or c[1] != n or not _same_items(out, c[2]):
            op, ow, osc = out["op"], out["op_weight"], out["op_score"]
            if op.numel() < n or ow.numel() < n or osc.numel() < n:
                raise ValueError("score output buffers too small")
            c = self._scache = [out, n, tuple(out.items()), (_ptr(op), _ptr(ow), _ptr(osc)), None]
        nops = ctypes.c_uint64()
        sagg = ctypes.c_double()
        _check(_lib().atrex_weighted_score(self._ctx, _ptr(score_key), _ptr(s), n, *c[3], ctypes.byref(nops),
                                           ctypes.byref(sagg)), "atrex_weighted_score")
        k = nops.value
        if c[4] is None or c[4][0] != k:  # views of the first k entries
            c[4] = (k, out["op"][:k], out["op_weight"][:k], out["op_score"][:k])
        return dict(s_agg=sagg.value, op=c[4][1], op_weight=c[4][2], op_score=c[4][3])

    # -- inspection ------------------------------------------------------------------------
    def app_totals(self) -> dict:
        """D_a^phi, the scale (m, rho) and, with app_count=True at construction,
        the invocation count n of every (app, phase), index a * P + phase."""
        GA, dev = self.A * self.P, self.device
        T = torch.empty((GA, 2), dtype=torch.int64, device=dev)
        n = torch.empty(GA, dtype=torch.int64, device=dev) if self.app_count else None
        m = torch.empty(GA, dtype=torch.int64, device=dev)
        r = torch.empty(GA, dtype=torch.int32, device=dev)
        _check(_lib().atrex_get_app_totals(self._ctx, _ptr(T), _ptr(n), _ptr(m), _ptr(r)), "atrex_get_app_totals")
        out = dict(T=T, mant=m, rho=r)
        if n is not None:
            out["n"] = n
        return out

    # -- target-DSL device-time share (§4.1, Metrics) ----------------------------------
    def share_buffers(self, key_capacity: int, op_capacity: int) -> dict:
        """Output tensors for target_share()."""
        dev, kc, oc = self.device, max(int(key_capacity), 1), max(int(op_capacity), 1)
        return dict(key=torch.empty(kc, dtype=torch.int32, device=dev),
                    count=torch.empty(kc, dtype=torch.int64, device=dev),
                    dsl_ns=torch.empty((kc, 2), dtype=torch.int64, device=dev),
                    total_ns=torch.empty((kc, 2), dtype=torch.int64, device=dev),
                    share=torch.empty(kc, dtype=torch.float64, device=dev),
                    op=torch.empty(oc, dtype=torch.int32, device=dev),
                    op_shapes=torch.empty(oc, dtype=torch.int32, device=dev),
                    op_share=torch.empty(oc, dtype=torch.float64, device=dev))

    def target_share(self, key_capacity: int | None = None, op_capacity: int | None = None,
                     out: dict | None = None) -> dict:
        """Per key the DSL (phase 1) and total device time and their ratio, per
        operator the exact mean over its running shapes, and the mean over the
        operators where it is defined (device_time=True, num_phases=2, after
        aggregate()).  Capacities default to the group count, or to the sizes
        of `out` (from share_buffers())."""
        G = self.num_groups or 0
        if out is not None:
            kc = out["key"].numel() if key_capacity is None else int(key_capacity)
            oc = out["op"].numel() if op_capacity is None else int(op_capacity)
        else:
            kc = G if key_capacity is None else int(key_capacity)
            oc = min(G, 65536) if op_capacity is None else int(op_capacity)
            out = self.share_buffers(kc, oc)
        so = _ShareOut(*(_ptr(out[k]) for k in ("key", "count", "dsl_ns", "total_ns", "share", "op", "op_shapes",
                                                 "op_share")))
        r = _ShareResult()
        _check(_lib().atrex_target_share(self._ctx, ctypes.byref(so), kc, oc, ctypes.byref(r)), "atrex_target_share")
        K, I = r.num_keys, r.num_ops
        res = {k: v[:K] for k, v in out.items() if not k.startswith("op")}
        res.update({k: v[:I] for k, v in out.items() if k.startswith("op")})
        res.update(adoption=r.adoption, defined_ops=r.defined_ops, num_keys=K, num_ops=I)
        return res

    # -- observed runtime per unit (§3.1, the deployment baseline) ----------------------
    def stats_buffers(self, capacity: int, nq: int) -> dict:
        """Output tensors for unit_stats()."""
        dev, c = self.device, max(int(capacity), 1)
        return dict(key=torch.empty(c, dtype=torch.int32, device=dev),
                    phase=torch.empty(c, dtype=torch.uint8, device=dev),
                    count=torch.empty(c, dtype=torch.int64, device=dev),
                    total_ns=torch.empty((c, 2), dtype=torch.int64, device=dev),
                    mean_ns=torch.empty(c, dtype=torch.float64, device=dev),
                    min_ns=torch.empty(c, dtype=torch.int64, device=dev),
                    max_ns=torch.empty(c, dtype=torch.int64, device=dev),
                    quantile_ns=torch.empty((c, max(nq, 1)), dtype=torch.int64, device=dev))

    def unit_stats(self, key: torch.Tensor, phase: torch.Tensor, dur_ns: torch.Tensor, q_1e5=(50000, 99000),
                   by_phase: bool = True, capacity: int | None = None, out: dict | None = None) -> dict:
        """Count, total, mean, min, max and nearest-rank quantiles (q in 1e-5
        steps) of the durations of every unit, after aggregate() on the same
        events (device_time=True).  Capacity defaults to the group count."""
        key = _dev(_as_i32(key), torch.int32, "key")
        phase = _dev(phase, torch.uint8, "phase")
        dur_ns = _dev(dur_ns, torch.int64, "dur_ns")
        n = key.numel()
        if not (phase.numel() == n and dur_ns.numel() == n):
            raise ValueError("event arrays differ in length")
        q = (ctypes.c_uint32 * 8)(*[int(x) for x in q_1e5])
        nq = len(q_1e5)
        if out is None:
            out = self.stats_buffers((self.num_groups or 0) if capacity is None else capacity, nq)
        cap = out["key"].numel() if capacity is None else int(capacity)
        so = _StatsOut(*(_ptr(out[k]) for k in ("key", "phase", "count", "total_ns", "mean_ns", "min_ns", "max_ns",
                                                 "quantile_ns")))
        ev = _Events(_ptr(key), None, _ptr(phase), _ptr(dur_ns), n)
        U = ctypes.c_uint64()
        _check(_lib().atrex_unit_stats(self._ctx, ctypes.byref(ev), int(bool(by_phase)), q, nq, ctypes.byref(so), cap,
                                       ctypes.byref(U)), "atrex_unit_stats")
        u = U.value
        res = {k: v[:u] for k, v in out.items()}
        res["quantile_ns"] = out["quantile_ns"][:u, :nq]
        res["num_units"] = u
        return res

    def kernel_times(self) -> list:
        cap = 64
        names = (ctypes.c_char_p * cap)()
        ms = (ctypes.c_float * cap)()
        items = (ctypes.c_uint64 * cap)()
        cnt = ctypes.c_int()
        _check(_lib().atrex_kernel_times(self._ctx, names, ms, items, cap, ctypes.byref(cnt)),
               "atrex_kernel_times")
        return [(names[i].decode(), float(ms[i]), int(items[i])) for i in range(cnt.value)]

    def path_used(self) -> str:
        return _lib().atrex_path_used(self._ctx).decode()

    def close(self) -> None:
        if getattr(self, "_ctx", None):
            _lib().atrex_aggregate_destroy(self._ctx)
            self._ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def aggregate(key, app, phase, dur_ns, app_weight_q16, num_phases, path="auto", raw=False,
              score_key=None, s=None, max_groups=0, max_keys=0, app_count=False) -> dict:
    """Whole path in one call: returns groups, per-op and per-key weights, and
    the score when (score_key, s) are given."""
    n = key.numel()
    nsc = score_key.numel() if score_key is not None else 0
    ag = Aggregator(num_phases, app_weight_q16, max_events=max(n, 1), max_groups=max_groups,
                    max_keys=max_keys, max_score=max(nsc, 1) if nsc else 0, path=path, raw=raw,
                    app_count=app_count)
    try:
        ag.aggregate(key, app, phase, dur_ns)
        out = ag.normalize()
        out.update({"op_" + k if k != "op" else k: v for k, v in ag.op_weights().items()})
        kw = ag.key_weights()
        out.update(ukey=kw["key"], key_U=kw["U"], omega=kw["omega"])
        out.update({"app_" + k: v for k, v in ag.app_totals().items()})
        out["path"] = ag.path_used()
        if score_key is not None:
            out.update({"score_" + k if k != "s_agg" else k: v for k, v in ag.score(score_key, s).items()})
        return out
    finally:
        ag.close()


def score(ctx: "Aggregator", score_key, s) -> float:
    """S_agg of Eq. (6) (§3.6) for an Aggregator whose group-by and
    normalisation have run: score_key (u32 keys) and s (fp64 S_j, NaN = not
    correct) as device tensors.  Repeatable; ctx.score() also returns the
    per-operator weights and medians."""
    return ctx.score(score_key, s)["s_agg"]


def target_share(key, is_dsl, dur_ns, path="auto", max_keys=0) -> dict:
    """The target-DSL device-time share of one profile (§4.1, Metrics) in one
    call: the device-time group-by with phase = is_dsl (1 inside the target
    DSL, 0 outside), then atrex_target_share."""
    n = key.numel()
    ag = Aggregator(2, None, max_events=max(n, 1), max_keys=max_keys, path=path, device_time=True,
                    device=key.device)
    try:
        ag.aggregate(key, None, is_dsl, dur_ns)
        out = ag.target_share()
        out["path"] = ag.path_used()
        return out
    finally:
        ag.close()


def unit_stats(key, phase, dur_ns, num_phases, q_1e5=(50000, 99000), by_phase=True, path="auto",
               max_keys=0, max_groups=0) -> dict:
    """Observed runtime per unit (§3.1) in one call: the device-time group-by
    of the events, then atrex_unit_stats on the same events."""
    n = key.numel()
    ag = Aggregator(num_phases, None, max_events=max(n, 1), max_keys=max_keys, max_groups=max_groups, path=path,
                    device_time=True, device=key.device)
    try:
        ag.aggregate(key, None, phase, dur_ns)
        out = ag.unit_stats(key, phase, dur_ns, q_1e5=q_1e5, by_phase=by_phase)
        out["path"] = ag.path_used()
        return out
    finally:
        ag.close()


class Correlator:
    """Host/device correlation join (§3.1) with a workspace for up to
    max_kernels kernel records and max_host host records: run() labels
    kernel records by correlation id, graph anchor or stream interval and
    returns the labelled events in kernel-record order.  method: "auto",
    "hash" or "partition" (include/atrex.h, ATREX_JOIN_*); run() reports the
    one used."""

    KERNEL_FIELDS = (("corr", torch.int64), ("anchor", torch.int64), ("stream", torch.int32),
                     ("start_ns", torch.int64), ("end_ns", torch.int64))
    HOST_FIELDS = (("kind", torch.uint8), ("id", torch.int64), ("key", torch.int32), ("app", torch.int32),
                   ("phase", torch.uint8))
    INTERVAL_FIELDS = (("stream", torch.int32), ("begin_ns", torch.int64), ("end_ns", torch.int64),
                       ("key", torch.int32), ("app", torch.int32), ("phase", torch.uint8))

    def __init__(self, max_kernels: int, max_host: int, device=None, stream: torch.cuda.Stream | None = None,
                 method: str = "auto"):
        self.device = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        self.p = _JoinParams(int(max_kernels), int(max_host), None, 0, self.stream.cuda_stream, JOIN_METHODS[method])
        nb = ctypes.c_size_t()
        _check(_lib().atrex_join_workspace_bytes(ctypes.byref(self.p), ctypes.byref(nb)), "atrex_join_workspace_bytes")
        self.workspace = torch.empty(max(int(nb.value), 256), dtype=torch.uint8, device=self.device)
        self.p.workspace, self.p.workspace_bytes = self.workspace.data_ptr(), self.workspace.numel()

    def buffers(self, capacity: int) -> dict:
        c, dev = max(int(capacity), 1), self.device
        return dict(key=torch.empty(c, dtype=torch.int32, device=dev), app=torch.empty(c, dtype=torch.int32, device=dev),
                    phase=torch.empty(c, dtype=torch.uint8, device=dev),
                    dur_ns=torch.empty(c, dtype=torch.int64, device=dev))

    @staticmethod
    def _fields(d: dict, spec, name: str) -> tuple:
        ts = []
        for f, dt in spec:
            t = d[f]
            if dt in (torch.int32, torch.int64) and t.dtype != dt:
                t = t.view(dt) if t.element_size() == torch.empty(0, dtype=dt).element_size() else t.to(dt)
            ts.append(_dev(t, dt, name + "." + f))
        n = ts[0].numel()
        if any(t.numel() != n for t in ts):
            raise ValueError(name + " arrays differ in length")
        return tuple(ts), n

    def run(self, kernels: dict, host: dict, intervals: dict | None = None, out: dict | None = None,
            source: torch.Tensor | None = None) -> dict:
        kt, nk = self._fields(kernels, self.KERNEL_FIELDS, "kernels")
        ht, nh = self._fields(host, self.HOST_FIELDS, "host")
        kr = _KernelRecords(*(_ptr(t) for t in kt), nk)
        hr = _HostRecords(*(_ptr(t) for t in ht), nh)
        ir = None
        if intervals is not None:
            it, ni = self._fields(intervals, self.INTERVAL_FIELDS, "intervals")
            ir = _IntervalRecords(*(_ptr(t) for t in it), ni)
        if out is None:
            out = self.buffers(nk)
        if source is None:
            source = torch.empty(max(nk, 1), dtype=torch.uint8, device=self.device)
        eo = _EventOut(*(_ptr(out[k]) for k in ("key", "app", "phase", "dur_ns")))
        r = _JoinResult()
        _check(_lib().atrex_correlate(ctypes.byref(self.p), ctypes.byref(kr), ctypes.byref(hr),
                                      ctypes.byref(ir) if ir is not None else None, ctypes.byref(eo),
                                      out["key"].numel(), _ptr(source), ctypes.byref(r)), "atrex_correlate")
        L = r.labelled
        res = {k: v[:L] for k, v in out.items()}
        res.update(source=source[:nk], labelled=L, by_source=list(r.by_source),
                   method={v: k for k, v in JOIN_METHODS.items()}[r.method_used])
        return res


def run_noalloc(key, app, phase, dur_ns, app_weight_q16, num_phases, out: dict, score_key=None, s=None,
                score_out: dict | None = None, stream: torch.cuda.Stream | None = None) -> dict:
    """The whole path through atrex_run_noalloc: no context, no workspace, no
    device allocation by the library (caller-owned inputs and outputs only).
    `out` as from Aggregator.group_buffers(); `score_out` holds op / op_weight /
    op_score tensors of at least len(score_key) entries.  Returns the counts,
    s_agg and views of the first num_groups / num_scored_ops entries."""
    key = _dev(_as_i32(key), torch.int32, "key")
    app = _dev(_as_i32(app), torch.int32, "app")
    phase = _dev(phase, torch.uint8, "phase")
    dur_ns = _dev(dur_ns, torch.int64, "dur_ns")
    c = _dev(_as_i32(app_weight_q16), torch.int32, "app_weight_q16")
    n = key.numel()
    if not (app.numel() == n and phase.numel() == n and dur_ns.numel() == n):
        raise ValueError("event arrays differ in length")
    st = stream if stream is not None else torch.cuda.current_stream(key.device)
    p = _NoAllocParams(int(num_phases), c.numel(), c.data_ptr(), st.cuda_stream)
    ev = _Events(_ptr(key), _ptr(app), _ptr(phase), _ptr(dur_ns), n)
    g = _Groups(_ptr(out["key"]), _ptr(out["phase"]), _ptr(out["count"]), _ptr(out["wsum"]),
                _ptr(out["weight"]), _ptr(out["phase_total"]), _ptr(out.get("raw_ns")))
    nsc, sp = 0, (ctypes.c_void_p(0),) * 5
    if score_key is not None:
        score_key = _dev(_as_i32(score_key), torch.int32, "score_key")
        s = _dev(s, torch.float64, "s")
        nsc = score_key.numel()
        if s.numel() != nsc:
            raise ValueError("score_key and s differ in length")
        if any(score_out[k].numel() < nsc for k in ("op", "op_weight", "op_score")):
            raise ValueError("score output buffers too small")
        sp = (_ptr(score_key), _ptr(s), _ptr(score_out["op"]), _ptr(score_out["op_weight"]),
              _ptr(score_out["op_score"]))
    r = _RunResult()
    _check(_lib().atrex_run_noalloc(ctypes.byref(p), ctypes.byref(ev), ctypes.byref(g), out["key"].numel(), sp[0],
                                    sp[1], nsc, sp[2], sp[3], sp[4], ctypes.byref(r)), "atrex_run_noalloc")
    G, k = r.num_groups, r.num_scored_ops
    res = dict(num_groups=G, num_ops=r.num_ops, num_keys=r.num_keys, num_scored_ops=k, s_agg=r.s_agg,
               groups={kk: (t if kk == "phase_total" else t[:G]) for kk, t in out.items()})
    if score_key is not None:
        res["score"] = {kk: score_out[kk][:k] for kk in ("op", "op_weight", "op_score")}
    return res
