"""Host/device correlation join on the GPU (§3.1) against the oracle, through
the C ABI (atrex_correlate): every kernel record's source and every labelled
event (key, app, phase, duration, in kernel-record order) must match bit for
bit; at sizes where the oracle is slow, against the labelled events the raw
records were built from (the oracle recovers them exactly at the sizes the
CPU tests run).  The labelled events then run through the weighting path."""
import numpy as np
import pytest
import torch

import gpu_helpers as H
from oracle import oracle as O
from paper_2607_14541_amd import atrex as X
from paper_2607_14541_amd import synth

pytestmark = pytest.mark.gpu

KF = (("corr", np.uint64, np.int64), ("anchor", np.uint64, np.int64), ("stream", np.uint32, np.int32),
      ("start_ns", np.int64, np.int64), ("end_ns", np.int64, np.int64))
HF = (("kind", np.uint8, np.uint8), ("id", np.uint64, np.int64), ("key", np.uint32, np.int32),
      ("app", np.uint32, np.int32), ("phase", np.uint8, np.uint8))
IF = (("stream", np.uint32, np.int32), ("begin_ns", np.int64, np.int64), ("end_ns", np.int64, np.int64),
      ("key", np.uint32, np.int32), ("app", np.uint32, np.int32), ("phase", np.uint8, np.uint8))


def up(d, spec):
    return {f: H.dev(np.ascontiguousarray(d[f], nt), dt) for f, nt, dt in spec}


def gpu_join(kernels, host, intervals=None, capacity=None, method="auto"):
    n = len(kernels["corr"])
    c = X.Correlator(max(n, 1), max(len(host["id"]), 1), method=method)
    k, h = up(kernels, KF), up(host, HF)
    iv = up(intervals, IF) if intervals is not None else None
    out = c.buffers(n if capacity is None else capacity)
    r = c.run(k, h, iv, out=out)
    res = {f: r[f].cpu().numpy() for f in ("key", "app", "phase", "dur_ns", "source")}
    res["key"], res["app"] = res["key"].view(np.uint32), res["app"].view(np.uint32)
    res.update(labelled=r["labelled"], by_source=r["by_source"], method=r["method"])
    if method != "auto":
        assert r["method"] == method
    return res


def check(g, o):
    assert np.array_equal(g["source"], o["source"])
    assert g["labelled"] == o["labelled"] and g["by_source"] == o["by_source"].tolist()
    for f in ("key", "app", "phase", "dur_ns"):
        assert np.array_equal(g[f], o[f]), f


HAND = (dict(corr=[5, 0, 9, 0, 5], anchor=[3, 3, 0, 0, 0], stream=[1, 1, 2, 2, 1],
             start_ns=[10, 20, 30, 40, 50], end_ns=[15, 26, 31, 47, 50]),
        dict(kind=[0, 1], id=[5, 3], key=[100, 200], app=[1, 2], phase=[0, 1]),
        dict(stream=[1, 2], begin_ns=[0, 35], end_ns=[100, 45], key=[7, 300], app=[9, 3], phase=[2, 1]))


METHODS = ["hash", "partition"]


@pytest.mark.parametrize("method", METHODS)
def test_hand_worked_trace(method):
    g = gpu_join(*HAND, method=method)
    check(g, O.correlate(*HAND))
    assert g["source"].tolist() == [0, 1, 3, 2, 0]


@pytest.mark.parametrize("method", METHODS)
@pytest.mark.parametrize("n", [(1 << 20), 100003])
def test_synthetic_trace_against_the_oracle(n, method):
    tr = synth.join_trace(synth.JOIN_CONFIGS[0], n=n)
    H.say("join, synthetic trace", n, method)
    g = gpu_join(tr["kernels"], tr["host"], tr["intervals"], method=method)
    check(g, O.correlate(tr["kernels"], tr["host"], tr["intervals"]))


@pytest.mark.parametrize("method", ["auto", "hash"])
def test_large_trace_recovers_the_labelled_events(method):
    tr = synth.join_trace(synth.JOIN_CONFIGS[1], n=1 << 24)
    H.say("join, 16M kernel records", method)
    g = gpu_join(tr["kernels"], tr["host"], tr["intervals"], method=method)
    if method == "auto":
        assert g["method"] == "partition"
    m = tr["kind"] < 3
    assert np.array_equal(g["source"], tr["kind"])
    for f in ("key", "app", "phase", "dur_ns"):
        assert np.array_equal(g[f], tr["truth"][f][m]), f


@pytest.mark.parametrize("method", METHODS)
def test_without_intervals_or_host_records(method):
    tr = synth.join_trace(synth.JOIN_CONFIGS[0], n=50000)
    g = gpu_join(tr["kernels"], tr["host"], None, method=method)
    check(g, O.correlate(tr["kernels"], tr["host"], None))
    empty = {f: np.zeros(0, nt) for f, nt, _ in HF}
    g = gpu_join(tr["kernels"], empty, tr["intervals"], method=method)
    check(g, O.correlate(tr["kernels"], empty, tr["intervals"]))
    ek = {f: np.zeros(0, nt) for f, nt, _ in KF}
    g = gpu_join(ek, tr["host"], tr["intervals"], method=method)
    assert g["labelled"] == 0 and g["by_source"] == [0, 0, 0, 0]


def test_partition_ids_crowding_one_bucket():
    """Host ids chosen to share one bucket of the partitioned join beyond its
    LDS tables' room: the call falls back to the hash join, same results."""
    rng = np.random.default_rng(5)
    nh = 6000  # 16 buckets (the fewest) of 4096 slots per id space
    ids = []
    cand = rng.integers(1, 1 << 62, 400000, dtype=np.uint64)
    top = (_id_hash(cand) >> np.uint32(28)).astype(np.int64)
    ids = cand[top == 3][:nh]
    assert ids.size == nh
    host = dict(kind=np.zeros(nh, np.uint8), id=ids, key=np.arange(nh, dtype=np.uint32),
                app=np.zeros(nh, np.uint32), phase=np.zeros(nh, np.uint8))
    nk = 3 * nh
    kern = dict(corr=np.where(np.arange(nk) % 3 == 2, np.uint64(0), ids[np.arange(nk) % nh]).astype(np.uint64),
                anchor=np.zeros(nk, np.uint64), stream=np.zeros(nk, np.uint32),
                start_ns=np.arange(nk, dtype=np.int64), end_ns=np.arange(nk, dtype=np.int64) + 5)
    g = gpu_join(kern, host, None)
    assert g["method"] == "hash"
    check(g, O.correlate(kern, host, None))


def _id_hash(ids):
    """hash32(lo ^ hash32(hi)) of 64-bit ids, hash32 being the library's
    xorshift-multiply mixer (shifts 16, 15, 16; multipliers 0x7feb352d and
    0x846ca68b), to pick ids that land in one bucket."""
    def h32(x):
        x = x.astype(np.uint64) & np.uint64(0xFFFFFFFF)
        x ^= x >> np.uint64(16)
        x = (x * np.uint64(0x7feb352d)) & np.uint64(0xFFFFFFFF)
        x ^= x >> np.uint64(15)
        x = (x * np.uint64(0x846ca68b)) & np.uint64(0xFFFFFFFF)
        x ^= x >> np.uint64(16)
        return x
    lo = ids & np.uint64(0xFFFFFFFF)
    hi = ids >> np.uint64(32)
    return h32(lo ^ h32(hi)).astype(np.uint32)


def test_labelled_events_through_the_weighting_path():
    """Raw records -> labelled events -> weights, against the oracle's
    weights of the events the records were built from."""
    tr = synth.join_trace(synth.JOIN_CONFIGS[0], n=(1 << 20) + 3)
    cfg = synth.CONFIGS[0]
    c = X.Correlator(tr["kind"].size, tr["host"]["id"].size)
    r = c.run(up(tr["kernels"], KF), up(tr["host"], HF), up(tr["intervals"], IF))
    m = tr["kind"] < 3
    truth = {f: tr["truth"][f][m] for f in ("key", "app", "phase", "dur_ns")}
    cw = synth.app_weights(cfg)
    g = H.run_gpu(r["key"].cpu().numpy().view(np.uint32), r["app"].cpu().numpy().view(np.uint32),
                  r["phase"].cpu().numpy(), r["dur_ns"].cpu().numpy(), cw, cfg["num_phases"])
    o = O.run(truth["key"], truth["app"], truth["phase"], truth["dur_ns"], cw, cfg["num_phases"])
    H.compare(g, o, raw=True)


@pytest.mark.parametrize("method", METHODS)
def test_errors(method):
    k, h, iv = HAND
    bad_h = [dict(h, id=[5, 5], kind=[0, 0]), dict(h, id=[0, 3]), dict(h, kind=[2, 1])]
    for hh in bad_h:
        with pytest.raises(X.AtrexError) as e:
            gpu_join(k, hh, iv, method=method)
        assert e.value.status == X.E_INVALID_ARG
    for ii in (dict(iv, stream=[2, 1]), dict(iv, begin_ns=[0, 35], end_ns=[100, 34]),
               dict(stream=[1, 1], begin_ns=[0, 50], end_ns=[60, 70], key=[1, 2], app=[0, 0], phase=[0, 0])):
        with pytest.raises(X.AtrexError) as e:
            gpu_join(k, h, ii, method=method)
        assert e.value.status == X.E_INVALID_ARG
    with pytest.raises(X.AtrexError) as e:
        gpu_join(dict(k, end_ns=[15, 26, 31, 47, 49]), h, iv, method=method)
    assert e.value.status == X.E_OUT_OF_RANGE
    with pytest.raises(X.AtrexError) as e:
        gpu_join(k, h, iv, capacity=2, method=method)
    assert e.value.status == X.E_CAPACITY
