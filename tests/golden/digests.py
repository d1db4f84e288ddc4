"""Canonical digests of the path's outputs, for parity checks on workloads too
large to compare element by element in a test (test infrastructure).

Every output array is hashed (SHA-256) over its elements as little-endian
values of a fixed type and shape, in the order the path defines (groups
ascending by (key, phase), (app, phase) pairs at index a * P + phase,
operators and keys ascending).  128-bit values are (low, high) pairs of
uint64.  Floating-point arrays are hashed bit for bit: every fp64 output of
the path is one correctly rounded operation on exact integers (or a median of
the inputs), so equal integers give equal bits.  S_agg, a compensated sum, is
stored as a number and compared within the parity tolerance.
"""
from __future__ import annotations

import hashlib
import json
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
DIGEST_FILE = os.path.join(HERE, "full_size_digests.json")

# output name -> (numpy type, elements per entry)
FIELDS = {
    "key": ("<u4", 1), "phase": ("<u1", 1), "count": ("<u8", 1), "wsum": ("<u8", 2),
    "raw_ns": ("<u8", 2), "weight": ("<f8", 1), "phase_total": ("<u8", 2),
    "app_total": ("<u8", 2), "app_count": ("<u8", 1), "mant": ("<u8", 1), "rho": ("<i4", 1),
    "op": ("<u4", 1), "op_U": ("<u8", 2), "op_w": ("<f8", 1),
    "ukey": ("<u4", 1), "key_U": ("<u8", 2), "omega": ("<f8", 1),
    "score_op": ("<u4", 1), "score_op_weight": ("<f8", 1), "score_op_S": ("<f8", 1),
}


def digest(name: str, a) -> str:
    """SHA-256 of output `name` as its canonical little-endian array."""
    dt, per = FIELDS[name]
    x = np.ascontiguousarray(np.asarray(a))
    # reinterpret (not convert) values that travelled as signed integers
    want = np.dtype(dt)
    if x.dtype.kind in "iu" and want.kind in "iu" and x.dtype.itemsize == want.itemsize:
        x = x.view(want)
    x = x.astype(want, copy=False).reshape(-1, per)
    return hashlib.sha256(x.tobytes()).hexdigest()


def digests(outputs: dict) -> dict:
    """Digests of every known output present in `outputs`."""
    return {k: digest(k, v) for k, v in outputs.items() if k in FIELDS}


def load() -> dict:
    with open(DIGEST_FILE) as f:
        return json.load(f)


def mismatches(record: dict, outputs: dict, s_agg=None, rel_tol: float = 1e-12) -> list:
    """Names of the outputs whose digests differ from `record` (only outputs
    present on both sides are compared), plus 's_agg' when it differs by more
    than rel_tol relative.  Also 'num_groups' when the counts differ."""
    bad = []
    if "key" in outputs and len(outputs["key"]) != record["num_groups"]:
        bad.append("num_groups")
    mine = digests(outputs)
    for k, h in record["digests"].items():
        if k in mine and mine[k] != h:
            bad.append(k)
    if s_agg is not None and "s_agg" in record:
        want = float.fromhex(record["s_agg"])
        if abs(s_agg - want) > rel_tol * max(abs(want), 1e-300):
            bad.append("s_agg")
    return bad
