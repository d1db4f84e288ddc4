"""Status codes of the GPU library match the oracle's on the same bad inputs,
and calls out of order are refused."""
import math

import numpy as np
import pytest
import torch

import gpu_helpers as H
from oracle import oracle as O
from paper_2607_14541_amd import atrex as X

pytestmark = pytest.mark.gpu


def status(key, app, ph, dur, c, P, sk=None, s=None, path="auto"):
    try:
        H.run_gpu(key, app, ph, dur, c, P, path=path, score_key=sk, s=s)
    except X.AtrexError as e:
        return e.status
    return X.OK


@pytest.mark.parametrize("path", ["lds_hash", "global_hash"])
@pytest.mark.parametrize("ev", [
    dict(key=[1, 2, 3, 4, 5], app=[0, 1, 9, 0, 1], phase=[0, 0, 0, 1, 1], dur=[5] * 5),
    dict(key=[1, 2, 3, 4, 5], app=[0, 1, 1, 0, 1], phase=[0, 0, 2, 1, 1], dur=[5] * 5),
    dict(key=[1, 2, 3, 4, 5], app=[0, 1, 1, 0, 1], phase=[0, 0, 0, 1, 1], dur=[5, 5, -7, 5, 5]),
])
def test_event_range_errors(path, ev):
    H.say("range error", path)
    o = O.status_of(ev["key"], ev["app"], ev["phase"], ev["dur"], [1, 1], 2)
    assert o == O.E_OUT_OF_RANGE
    assert status(ev["key"], ev["app"], ev["phase"], ev["dur"], [1, 1], 2, path=path) == o


@pytest.mark.parametrize("sk,s", [
    ([1 << 16], [1.5]), ([1 << 16], [0.0]), ([1 << 16], [-1.0]), ([1 << 16], [math.inf]),
    ([1 << 16, 1 << 16], [0.5, 0.5]), ([7 << 16], [0.5]),
])
def test_score_errors(sk, s):
    H.say("score error", sk, s)
    o = O.status_of([1 << 16], [0], [0], [5], [1], 1, score_key=sk, s=s)
    assert o != O.OK
    assert status([1 << 16], [0], [0], [5], [1], 1, sk=sk, s=s) == o


def test_zero_card_hours_rejected():
    H.say("zero weights")
    c = torch.zeros(3, dtype=torch.int32, device="cuda")
    with pytest.raises(X.AtrexError) as e:
        X.Aggregator(2, c, max_events=10)
    assert e.value.status == X.E_INVALID_ARG


def test_call_order():
    H.say("call order")
    c = torch.ones(2, dtype=torch.int32, device="cuda")
    ag = X.Aggregator(2, c, max_events=8)
    with pytest.raises(X.AtrexError) as e:
        ag.num_groups = 0
        ag.normalize()
    assert e.value.status == X.E_STATE
    k = torch.tensor([1, 2], dtype=torch.int32, device="cuda")
    a = torch.tensor([0, 1], dtype=torch.int32, device="cuda")
    p = torch.tensor([0, 1], dtype=torch.uint8, device="cuda")
    d = torch.tensor([3, 4], dtype=torch.int64, device="cuda")
    assert ag.aggregate(k, a, p, d) == 2
    with pytest.raises(X.AtrexError) as e:
        ag.aggregate(k, a, p, d)
    assert e.value.status == X.E_STATE
    with pytest.raises(X.AtrexError) as e:
        ag.score(k, torch.tensor([0.5, 0.5], dtype=torch.float64, device="cuda"))
    assert e.value.status == X.E_STATE
    ag.normalize()
    r = ag.score(k, torch.tensor([0.5, 0.25], dtype=torch.float64, device="cuda"))
    assert r["op"].numel() == 1
    # the module-level form returns the same S_agg (keys 1 and 2 are one
    # operator: the median of 0.5 and 0.25, weight 1)
    assert X.score(ag, k, torch.tensor([0.5, 0.25], dtype=torch.float64, device="cuda")) == r["s_agg"] == 0.375
    ag.close()


def test_capacity_error():
    H.say("capacity")
    c = torch.ones(1, dtype=torch.int32, device="cuda")
    ag = X.Aggregator(1, c, max_events=100, max_groups=4, max_keys=4)
    n = 50
    k = torch.arange(n, dtype=torch.int32, device="cuda")
    z = torch.zeros(n, dtype=torch.int32, device="cuda")
    with pytest.raises(X.AtrexError) as e:
        ag.aggregate(k, z, torch.zeros(n, dtype=torch.uint8, device="cuda"), torch.ones(n, dtype=torch.int64, device="cuda"))
    assert e.value.status == X.E_CAPACITY
    ag.close()


@pytest.mark.parametrize("bad", ["app", "phase", "duration"])
@pytest.mark.parametrize("where", [0, 77777, 199999])
def test_event_range_errors_range_split_pass_a(bad, where):
    """30000 apps x 2 phases do not fit one LDS table: pass A is split into
    ranges of the (app, phase) table; a wave that meets an invalid event
    checks its events one by one, in every range's workgroups."""
    rng = np.random.default_rng(where)
    n, A, P = 200000, 30000, 2
    key = rng.integers(0, 50, n).astype(np.uint32)
    app = rng.integers(0, A, n).astype(np.uint32)
    ph = rng.integers(0, P, n).astype(np.uint8)
    dur = rng.integers(1, 10 ** 6, n).astype(np.int64)
    c = rng.integers(1, 1000, A).astype(np.uint32)
    if bad == "app":
        app[where] = A + 3
    elif bad == "phase":
        ph[where] = P
    else:
        dur[where] = -1
    H.say("range error, range-split pass A", bad, where)
    o = O.status_of(key, app, ph, dur, c, P)
    assert o == O.E_OUT_OF_RANGE
    assert status(key, app, ph, dur, c, P) == o
    app[where], ph[where], dur[where] = 1, 0, 5  # the repaired trace aggregates
    assert status(key, app, ph, dur, c, P) == X.OK
