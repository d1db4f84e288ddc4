"""Pins of the oracle's host/device correlation join (§3.1: host and device
events are matched through correlation ids when available, otherwise through
graph anchors or timestamps).

Pinned by a hand-worked trace, a round trip (raw records built from labelled
events must give those events back, each kernel by the path it was built
for), a Python brute force with the precedence written out (dict lookups and
a linear interval scan), interval boundaries, and the validation rules."""
import random

import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_14541_amd import synth


def test_hand_worked_trace():
    kernels = dict(corr=[5, 0, 9, 0, 5], anchor=[3, 3, 0, 0, 0], stream=[1, 1, 2, 2, 1],
                   start_ns=[10, 20, 30, 40, 50], end_ns=[15, 26, 31, 47, 50])
    host = dict(kind=[0, 1], id=[5, 3], key=[100, 200], app=[1, 2], phase=[0, 1])
    intervals = dict(stream=[1, 2], begin_ns=[0, 35], end_ns=[100, 45], key=[7, 300], app=[9, 3], phase=[2, 1])
    r = O.correlate(kernels, host, intervals)
    # 1: corr 5 (wins over anchor 3 and the interval); 2: anchor 3; 3: corr 9
    # unknown, no anchor, start 30 outside [35, 45); 4: interval; 5: corr 5
    assert r["source"].tolist() == [0, 1, 3, 2, 0]
    assert r["key"].tolist() == [100, 200, 300, 100]
    assert r["app"].tolist() == [1, 2, 3, 1]
    assert r["phase"].tolist() == [0, 1, 1, 0]
    assert r["dur_ns"].tolist() == [5, 6, 7, 0]
    assert r["by_source"].tolist() == [2, 1, 1, 1] and r["labelled"] == 4


def test_round_trip_recovers_the_labelled_events():
    tr = synth.join_trace(synth.JOIN_CONFIGS[0], n=1 << 18)
    r = O.correlate(tr["kernels"], tr["host"], tr["intervals"])
    m = tr["kind"] < 3
    assert np.array_equal(r["source"], tr["kind"])
    for k in ("key", "app", "phase", "dur_ns"):
        assert np.array_equal(r[k], tr["truth"][k][m]), k


def _brute(k, h, iv):
    lab = {}
    for j in range(len(h["id"])):
        lab[(h["kind"][j], h["id"][j])] = (h["key"][j], h["app"][j], h["phase"][j])
    out, src = [], []
    for e in range(len(k["corr"])):
        s, v = 3, None
        for kind, ident in ((0, k["corr"][e]), (1, k["anchor"][e])):
            if s == 3 and ident != 0 and (kind, ident) in lab:
                s, v = kind, lab[(kind, ident)]
        if s == 3:
            for j in range(len(iv["stream"])):
                if iv["stream"][j] == k["stream"][e] and iv["begin_ns"][j] <= k["start_ns"][e] < iv["end_ns"][j]:
                    s, v = 2, (iv["key"][j], iv["app"][j], iv["phase"][j])
                    break
        src.append(s)
        if v is not None:
            out.append(v + (k["end_ns"][e] - k["start_ns"][e],))
    return src, out


@pytest.mark.parametrize("seed", range(15))
def test_brute_force(seed):
    rng = random.Random(seed)
    n = rng.randint(0, 200)
    S = rng.randint(1, 3)
    ids = rng.sample(range(1, 60), 20)
    host = dict(kind=[], id=[], key=[], app=[], phase=[])
    for kind in (0, 1):
        for i in rng.sample(ids, rng.randint(0, 12)):
            host["kind"].append(kind)
            host["id"].append(i)
            host["key"].append(rng.randrange(1 << 20))
            host["app"].append(rng.randrange(50))
            host["phase"].append(rng.randrange(3))
    iv = dict(stream=[], begin_ns=[], end_ns=[], key=[], app=[], phase=[])
    for s in range(S):
        t = 0
        for _ in range(rng.randint(0, 6)):
            b = t + rng.randint(0, 30)
            e = b + rng.randint(0, 40)
            t = e
            for f, v in (("stream", s), ("begin_ns", b), ("end_ns", e), ("key", rng.randrange(1 << 20)),
                         ("app", rng.randrange(50)), ("phase", rng.randrange(3))):
                iv[f].append(v)
    k = dict(corr=[], anchor=[], stream=[], start_ns=[], end_ns=[])
    for _ in range(n):
        st = rng.randint(0, 250)
        for f, v in (("corr", rng.choice([0] + ids)), ("anchor", rng.choice([0, 0] + ids)), ("stream", rng.randrange(S)),
                     ("start_ns", st), ("end_ns", st + rng.randint(0, 20))):
            k[f].append(v)
    src, out = _brute(k, host, iv)
    r = O.correlate(k, host, iv)
    assert r["source"].tolist() == src
    assert [tuple(x) for x in zip(r["key"].tolist(), r["app"].tolist(), r["phase"].tolist(),
                                  r["dur_ns"].tolist())] == out


def test_interval_boundaries():
    host = dict(kind=[], id=[], key=[], app=[], phase=[])
    iv = dict(stream=[0, 0], begin_ns=[10, 20], end_ns=[20, 30], key=[1, 2], app=[0, 0], phase=[0, 0])
    k = dict(corr=[0] * 5, anchor=[0] * 5, stream=[0, 0, 0, 0, 1], start_ns=[9, 10, 19, 20, 15],
             end_ns=[9, 11, 19, 40, 16])
    r = O.correlate(k, host, iv)
    assert r["source"].tolist() == [3, 2, 2, 2, 3]  # begin is inside, end is not; other streams never match
    assert r["key"].tolist() == [1, 1, 2]


def test_validation():
    k = dict(corr=[1], anchor=[0], stream=[0], start_ns=[5], end_ns=[6])
    good_h = dict(kind=[0], id=[1], key=[1], app=[0], phase=[0])
    for h in (dict(kind=[0, 0], id=[1, 1], key=[1, 2], app=[0, 0], phase=[0, 0]),  # the same id twice
              dict(kind=[0], id=[0], key=[1], app=[0], phase=[0]),                 # id 0
              dict(kind=[2], id=[1], key=[1], app=[0], phase=[0])):                # unknown kind
        with pytest.raises(O.OracleError) as e:
            O.correlate(k, h)
        assert e.value.status == O.E_INVALID_ARG
    # one id may serve as a correlation id and as an anchor
    O.correlate(k, dict(kind=[0, 1], id=[1, 1], key=[1, 2], app=[0, 0], phase=[0, 0]))
    for iv in (dict(stream=[0, 0], begin_ns=[10, 15], end_ns=[20, 30], key=[1, 2], app=[0, 0], phase=[0, 0]),  # overlap
               dict(stream=[1, 0], begin_ns=[10, 50], end_ns=[20, 60], key=[1, 2], app=[0, 0], phase=[0, 0]),  # order
               dict(stream=[0], begin_ns=[10], end_ns=[9], key=[1], app=[0], phase=[0])):                      # end < begin
        with pytest.raises(O.OracleError) as e:
            O.correlate(k, good_h, iv)
        assert e.value.status == O.E_INVALID_ARG
    with pytest.raises(O.OracleError) as e:
        O.correlate(dict(corr=[1], anchor=[0], stream=[0], start_ns=[5], end_ns=[4]), good_h)
    assert e.value.status == O.E_OUT_OF_RANGE
