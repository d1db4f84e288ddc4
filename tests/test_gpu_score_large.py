"""The score for more scored units than the one-workgroup kernels take
(n > 8192), through the C ABI against the oracle: per-operator segments
sorted in LDS (every operator with at most 8192 scored units), and the global
sorts taken when one operator has more.  Medians and U bit for bit, weights
and S_agg within 1e-12; duplicate keys and S outside (0, 1] give the oracle's
status."""
import math

import numpy as np
import pytest

import gpu_helpers as H
from oracle import oracle as O
from paper_2607_14541_amd import atrex as X

pytestmark = pytest.mark.gpu


def _case(layout, seed=11):
    rng = np.random.default_rng(seed)
    if layout == "many_ops":  # 40 operators x 500 shapes = 20000 scored units
        sk = np.array([(op << 16) | sh for op in range(40) for sh in range(500)], np.uint32)
    else:  # one operator with 12000 scored shapes, ten with 100
        sk = np.array([(3 << 16) | sh for sh in range(12000)] +
                      [(op << 16) | sh for op in (0, 1, 2, 4, 5, 6, 7, 8, 9, 10) for sh in range(100)], np.uint32)
    sk = sk[rng.permutation(sk.size)]
    s = rng.uniform(0.01, 1.0, sk.size)
    s[rng.random(sk.size) < 0.1] = math.nan
    # a trace over a subset of the scored keys plus a few keys nobody scores
    n, P, A = 150000, 2, 16
    pool = np.concatenate([sk[: sk.size // 2], np.array([(99 << 16) | 1, (98 << 16) | 2], np.uint32)])
    key = pool[rng.integers(0, pool.size, n)]
    app = rng.integers(0, A, n).astype(np.uint32)
    ph = rng.integers(0, P, n).astype(np.uint8)
    dur = rng.integers(1, 10 ** 7, n).astype(np.int64)
    c = rng.integers(1, 2 ** 20, A).astype(np.uint32)
    return key, app, ph, dur, c, P, sk, s


@pytest.mark.parametrize("layout", ["many_ops", "one_long_op"])
def test_large_score_parity(layout):
    key, app, ph, dur, c, P, sk, s = _case(layout)
    H.say("large score", layout, sk.size)
    g = H.run_gpu(key, app, ph, dur, c, P, score_key=sk, s=s)
    o = O.run(key, app, ph, dur, c, P, score_key=sk, s=s)
    H.compare(g, o, score=True)


@pytest.mark.parametrize("layout", ["many_ops", "one_long_op"])
@pytest.mark.parametrize("bad", ["duplicate", "above_one", "zero"])
def test_large_score_errors(layout, bad):
    key, app, ph, dur, c, P, sk, s = _case(layout, seed=5)
    sk = sk.copy()
    s = s.copy()
    if bad == "duplicate":
        sk[-1] = sk[17]
    elif bad == "above_one":
        s[123] = 1.25
    else:
        s[4567] = 0.0
    H.say("large score error", layout, bad)
    o = O.status_of(key, app, ph, dur, c, P, score_key=sk, s=s)
    assert o != O.OK
    try:
        H.run_gpu(key, app, ph, dur, c, P, score_key=sk, s=s)
        st = X.OK
    except X.AtrexError as e:
        st = e.status
    assert st == o
