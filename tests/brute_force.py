"""Exact-rational brute force for small traces (test helper, <= ~100 events).

Two independent computations, both in Python ``fractions``/big ints:

* ``real_valued``: the paper's Eq. (2)-(3) (§3.4) literally, in the paper's
  nesting order -- for each operator, sum over applications of
  p_a * mean over phi in Phi_i of D_{i,a}^phi / D_a^phi -- then the
  normalisation over operators.  Same for keys and for per-phase shares.
* ``fixed_point``: the Q96 fixed-point definition the oracle implements, from
  the rational r = 2^96 c_a / (C T) with ``Fraction`` floors instead of limb
  arithmetic and shifts.
"""
from __future__ import annotations

from collections import defaultdict
from fractions import Fraction
from math import floor, lcm

MANT_BITS = 56


def real_valued(key, app, phase, dur, c, P):
    """Eq. (2)-(3) with exact rationals.  Phi = phases with >= 1 invocation."""
    C = sum(int(x) for x in c)
    p = [Fraction(int(x), C) for x in c]
    D_a = defaultdict(int)                       # (a, phi) -> D_a^phi
    D_unit = {"op": defaultdict(int), "key": defaultdict(int)}  # (unit, a, phi)
    phases = {"op": defaultdict(set), "key": defaultdict(set)}
    for k, a, ph, d in zip(key, app, phase, dur):
        k, a, ph, d = int(k), int(a), int(ph), int(d)
        D_a[(a, ph)] += d
        for kind, u in (("op", k >> 16), ("key", k)):
            D_unit[kind][(u, a, ph)] += d
            phases[kind][u].add(ph)
    out = {}
    for kind in ("op", "key"):
        wt = {}
        for u, Phi in phases[kind].items():
            s = Fraction(0)
            for a in range(len(c)):
                inner = Fraction(0)
                for ph in Phi:
                    if D_a[(a, ph)] > 0:
                        inner += Fraction(D_unit[kind][(u, a, ph)], D_a[(a, ph)])
                s += p[a] * inner / len(Phi)
            wt[u] = s
        tot = sum(wt.values())
        out[kind] = {u: (w / tot if tot else Fraction(0)) for u, w in wt.items()}
        out[kind + "_raw"] = wt
    # per-(key, phase) share, normalised per phase
    share = defaultdict(Fraction)
    for (k, a, ph), dk in D_unit["key"].items():
        if D_a[(a, ph)] > 0:
            share[(k, ph)] += p[a] * Fraction(dk, D_a[(a, ph)])
    for (k, a, ph) in D_unit["key"]:
        share.setdefault((k, ph), Fraction(0))
    per_phase = defaultdict(Fraction)
    for (k, ph), v in share.items():
        per_phase[ph] += v
    out["group"] = {g: (v / per_phase[g[1]] if per_phase[g[1]] else Fraction(0))
                    for g, v in share.items()}
    out["group_raw"] = dict(share)
    return out


def floor_log2(r: Fraction) -> int:
    e = r.numerator.bit_length() - r.denominator.bit_length()
    while Fraction(2) ** e > r:
        e -= 1
    while Fraction(2) ** (e + 1) <= r:
        e += 1
    return e


def scale(c_a: int, C: int, T: int):
    """(m, rho): m * 2^(rho-55) <= 2^96 c_a/(C T) < (m+1) * 2^(rho-55)."""
    if T == 0 or c_a == 0:
        return 0, 0
    r = Fraction(c_a * 2 ** 96, C * T)
    rho = floor_log2(r)
    m = floor(r * Fraction(2) ** (MANT_BITS - 1 - rho))
    return m, rho


def fixed_point(key, app, phase, dur, c, P):
    C = sum(int(x) for x in c)
    T = defaultdict(int)
    n_app = defaultdict(int)
    for a, ph, d in zip(app, phase, dur):
        T[(int(a), int(ph))] += int(d)
        n_app[(int(a), int(ph))] += 1
    sc = {ap: scale(int(c[ap[0]]), C, t) for ap, t in T.items()}
    W = defaultdict(int)
    n = defaultdict(int)
    raw = defaultdict(int)
    for k, a, ph, d in zip(key, app, phase, dur):
        m, rho = sc[(int(a), int(ph))]
        v = floor(Fraction(int(d) * m) * Fraction(2) ** (rho - (MANT_BITS - 1)))
        g = (int(k), int(ph))
        W[g] += v
        n[g] += 1
        raw[g] += int(d)
    S = defaultdict(int)
    for (k, ph), w in W.items():
        S[ph] += w
    L = lcm(*range(1, P + 1))
    U = {"op": {}, "key": {}}
    for kind, unit in (("op", lambda k: k >> 16), ("key", lambda k: k)):
        Wu = defaultdict(lambda: defaultdict(int))
        nu = defaultdict(lambda: defaultdict(int))
        for (k, ph), w in W.items():
            Wu[unit(k)][ph] += w
            nu[unit(k)][ph] += n[(k, ph)]
        for u in Wu:
            Phi = [ph for ph in range(P) if nu[u][ph] > 0]
            U[kind][u] = (L // len(Phi)) * sum(Wu[u][ph] for ph in Phi)
    return dict(T=dict(T), n_app=dict(n_app), scale=sc, W=dict(W), n=dict(n), raw=dict(raw),
                S=dict(S), U=U)


def median(vals):
    v = sorted(vals)
    h = len(v) // 2
    return v[h] if len(v) % 2 else (v[h - 1] + v[h]) / 2
