#!/usr/bin/env python3
"""Writes tests/golden/full_size_digests.json: digests of the oracle's outputs
on every workload at its full size, for the full-size GPU parity tests and the
benchmark's self-check.

Calls only the CPU oracle (oracle/, its sharded group-by on every core) and the
seeded input generator; nothing here touches the GPU library.  Inputs are
those the benchmark times: all events of the workload, every key of its key
space scored with S_j ~ U[0.01, 1] (no unit marked incorrect).

    python tests/golden/make_digests.py [--configs 0,1,4,2,3] [--threads N]

Takes about an hour on 8 cores (the 256M- and 1B-event workloads dominate);
the file is rewritten after each workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)
sys.path.insert(0, HERE)

import digests as D  # noqa: E402
from oracle import oracle as O  # noqa: E402
from paper_2607_14541_amd import synth  # noqa: E402


def one(ci: int, threads: int) -> dict:
    cfg = synth.CONFIGS[ci]
    t0 = time.time()
    ev = synth.events(cfg)
    c = synth.app_weights(cfg)
    keys = synth.key_space(cfg)
    s = synth.scores(cfg, keys)
    t1 = time.time()
    o = O.run(ev["key"], ev["app"], ev["phase"], ev["dur_ns"], c, cfg["num_phases"], score_key=keys, s=s,
              threads=threads)
    t2 = time.time()
    del ev
    outputs = {k: o[k] for k in D.FIELDS if k in o}
    P = cfg["num_phases"]
    rec = {
        "workload": cfg["name"], "events": cfg["n"], "seed": cfg["seed"], "phases": P,
        "apps": cfg["num_apps"], "scored_keys": int(keys.size),
        "num_groups": int(o["num_groups"]), "num_ops": int(o["op"].size), "num_keys": int(o["ukey"].size),
        "num_scored_ops": int(o["score_op"].size),
        "s_agg": float(o["s_agg"]).hex(),
        "phase_total": [str(int(lo) | (int(hi) << 64)) for lo, hi in o["phase_total"]],
        "first_groups": [[int(o["key"][i]), int(o["phase"][i]), int(o["count"][i]),
                          str(int(o["wsum"][i][0]) | (int(o["wsum"][i][1]) << 64))]
                         for i in range(min(4, o["num_groups"]))],
        "digests": D.digests(outputs),
        "oracle_seconds": round(t2 - t1, 1), "oracle_threads": threads,
    }
    print("config %d: %s, %d groups, generated in %.1fs, oracle %.1fs on %d threads"
          % (ci, cfg["name"], o["num_groups"], t1 - t0, t2 - t1, threads), flush=True)
    return rec


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--configs", default="0,1,4,2,3")
    ap.add_argument("--threads", type=int, default=os.cpu_count() or 1)
    args = ap.parse_args()
    data = D.load() if os.path.exists(D.DIGEST_FILE) else {}
    data["note"] = ("SHA-256 digests of the CPU oracle's outputs on each workload at full size; "
                    "written by tests/golden/make_digests.py (oracle only)")
    data.setdefault("configs", {})
    for ci in [int(x) for x in args.configs.split(",")]:
        data["configs"][str(ci)] = one(ci, args.threads)
        tmp = D.DIGEST_FILE + ".tmp"
        with open(tmp, "w") as f:
            json.dump(data, f, indent=1, sort_keys=True)
        os.replace(tmp, D.DIGEST_FILE)
    return 0


if __name__ == "__main__":
    sys.exit(main())
