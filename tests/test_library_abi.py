"""The C-ABI library loads and exports every entry point include/atrex.h
declares; host-only entry points behave (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "atrex.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(atrex_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    from paper_2607_14541_amd import atrex
    return atrex._lib()


def test_header_declares_the_four_boundary_calls():
    names = declared_functions()
    for n in ("atrex_aggregate_init", "atrex_aggregate_events", "atrex_phase_normalize",
              "atrex_weighted_score"):
        assert n in names


def test_every_declared_symbol_is_exported(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    assert lib.atrex_status_str(0) == b"ok"
    assert lib.atrex_status_str(-4) == b"capacity exceeded"


def test_workspace_bytes_validates_parameters(lib):
    from paper_2607_14541_amd import atrex as X
    p = X._InitParams()
    b = ctypes.c_size_t()
    for P, A, ok in ((2, 1024, True), (0, 4, False), (9, 4, False), (8, 0, False)):
        p.num_phases, p.num_apps, p.max_events = P, A, 1 << 20
        st = lib.atrex_workspace_bytes(ctypes.byref(p), ctypes.byref(b))
        assert (st == 0) == ok
    p.num_phases, p.num_apps, p.max_events = 2, 4, 1 << 31  # n must stay below 2^31
    assert lib.atrex_workspace_bytes(ctypes.byref(p), ctypes.byref(b)) == X.E_INVALID_ARG


def test_init_rejects_bad_arguments_before_touching_the_device(lib):
    from paper_2607_14541_amd import atrex as X
    p = X._InitParams()
    ctx = ctypes.c_void_p()
    p.num_phases, p.num_apps, p.max_events = 2, 4, 100
    assert lib.atrex_aggregate_init(ctypes.byref(p), ctypes.byref(ctx)) == X.E_INVALID_ARG  # no weights
    assert ctx.value is None
    assert lib.atrex_aggregate_events(None, None, None) == X.E_INVALID_ARG


def test_device_time_flag_validation(lib):
    """The plain device-time mode takes one application and no raw-time flag."""
    from paper_2607_14541_amd import atrex as X
    p = X._InitParams()
    b = ctypes.c_size_t()
    p.max_events = 1000
    for A, flags, ok in ((1, X.FLAG_DEVICE_TIME, True), (2, X.FLAG_DEVICE_TIME, False),
                         (1, X.FLAG_DEVICE_TIME | X.FLAG_RAW, False),
                         (1, X.FLAG_DEVICE_TIME | X.FLAG_APP_COUNT | X.FLAG_TIMING, True)):
        p.num_phases, p.num_apps, p.flags = 2, A, flags
        assert (lib.atrex_workspace_bytes(ctypes.byref(p), ctypes.byref(b)) == 0) == ok, (A, flags)
    assert lib.atrex_target_share(None, None, 0, 0, None) == X.E_INVALID_ARG


def test_incremental_flag_validation(lib):
    """An incremental context cannot also be a device-time one."""
    from paper_2607_14541_amd import atrex as X
    p = X._InitParams()
    b = ctypes.c_size_t()
    p.max_events, p.num_phases, p.num_apps = 1000, 2, 4
    p.flags = X.FLAG_INCREMENTAL
    assert lib.atrex_workspace_bytes(ctypes.byref(p), ctypes.byref(b)) == 0
    p.num_apps, p.flags = 1, X.FLAG_INCREMENTAL | X.FLAG_DEVICE_TIME
    assert lib.atrex_workspace_bytes(ctypes.byref(p), ctypes.byref(b)) == X.E_INVALID_ARG
    assert lib.atrex_refresh(None, None, 0, None) == X.E_INVALID_ARG
    assert lib.atrex_refresh_state(None, None, None, None) == X.E_INVALID_ARG
    assert lib.atrex_refresh_restore(None, None, None, 0) == X.E_INVALID_ARG
    assert lib.atrex_unit_stats(None, None, 0, None, 0, None, 0, None) == X.E_INVALID_ARG


def test_join_parameters(lib):
    from paper_2607_14541_amd import atrex as X
    p = X._JoinParams(1 << 20, 1 << 20, None, 0, None)
    b = ctypes.c_size_t()
    assert lib.atrex_join_workspace_bytes(ctypes.byref(p), ctypes.byref(b)) == 0 and b.value > 0
    sizes = {}
    for name, m in X.JOIN_METHODS.items():
        p.method = m
        assert lib.atrex_join_workspace_bytes(ctypes.byref(p), ctypes.byref(b)) == 0
        sizes[name] = b.value
    assert sizes["auto"] == sizes["partition"] >= sizes["hash"]
    p.method = 3  # no such method
    assert lib.atrex_join_workspace_bytes(ctypes.byref(p), ctypes.byref(b)) == X.E_INVALID_ARG
    p.method, p.max_host = X.JOIN_METHODS["partition"], (2048 << 15) + 1  # beyond the partitioned join's buckets
    assert lib.atrex_join_workspace_bytes(ctypes.byref(p), ctypes.byref(b)) == X.E_INVALID_ARG
    p.method = X.JOIN_METHODS["auto"]  # takes the hash join there: the hash join's workspace
    assert lib.atrex_join_workspace_bytes(ctypes.byref(p), ctypes.byref(b)) == 0
    auto_big = b.value
    p.method = X.JOIN_METHODS["hash"]
    assert lib.atrex_join_workspace_bytes(ctypes.byref(p), ctypes.byref(b)) == 0 and b.value == auto_big
    p.max_kernels = 1 << 31
    assert lib.atrex_join_workspace_bytes(ctypes.byref(p), ctypes.byref(b)) == X.E_INVALID_ARG
    assert lib.atrex_correlate(None, None, None, None, None, 0, None, None) == X.E_INVALID_ARG
