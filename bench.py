#!/usr/bin/env python3
"""Benchmark of the trace-event -> importance-weight path on one MI355X.

One step = the whole path over one batch of events already resident in HBM:
pass A (per-(app, phase) time, Eq. (2)), the Q96 scale (Eq. (3)), pass B
(per-(key, phase) shares), compaction/ordering, per-phase normalisation and
Eq. (3) per operator and key, and the importance-weighted score (Eq. (4)-(6)).
Prints one JSON line: throughput in G events/s, the roofline of the dominant
kernel (per-kernel hipEvent times from the library, taken on the stream the
kernels run on) and the CPU oracle timed on a bounded sample.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 1] [--path auto]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E peak, GB/s
BYTES_PASS_A = 13              # app u32 + phase u8 + dur i64 per event
BYTES_PASS_B = 17              # key u32 + app u32 + phase u8 + dur i64 per event
# algorithmic HBM bytes per event of the streaming kernels: the event fields
# each one must read, plus the 16-byte partition records written and re-read
KERNEL_BYTES = {"pass_a": BYTES_PASS_A, "pass_a_global": BYTES_PASS_A,
                "pass_b_lds": BYTES_PASS_B, "pass_b_global": BYTES_PASS_B,
                "part_hist": 4, "part_scatter": BYTES_PASS_B + 16, "part_aggregate": 16}
KERNEL_SOURCES = ["paper_2607_14541_amd/csrc/kernels_aggregate.hip",
                  "paper_2607_14541_amd/csrc/kernels_rows.hip",
                  "paper_2607_14541_amd/csrc/atrex_kernels.h",
                  "paper_2607_14541_amd/csrc/atrex_device.hpp"]


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def traffic_from_profile(slug: str, kernel: str, n: int):
    """HBM bytes per launch from committed rocprofv3 counter summaries, or
    None when none exists for this kernel/workload or the kernel source has
    changed since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic_%s.json" % slug)
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    k = rec.get("kernels", {}).get(kernel)
    if not k or rec.get("kernel_source_hash") != kernel_source_hash() or rec.get("events") != n:
        return None
    return k.get("hbm_bytes_per_launch")


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=1, help="workload index (0..4)")
    ap.add_argument("--path", default="auto", choices=["auto", "lds_hash", "global_hash", "radix_sort"])
    ap.add_argument("--cpu-sample-log2", type=int, default=26,
                    help="events of the workload the CPU oracle is timed on (2^k)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        return 2

    import numpy as np
    import torch
    from paper_2607_14541_amd import atrex as X
    from paper_2607_14541_amd import synth

    cfg = synth.CONFIGS[args.config]
    n, P = cfg["n"], cfg["num_phases"]
    keys = synth.key_space(cfg)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log("config", args.config, cfg["name"], "n", n)
    t = time.time()
    ev = synth.events(cfg)
    c = synth.app_weights(cfg)
    s = synth.scores(cfg, keys)
    log("generated in %.1fs" % (time.time() - t))
    d_key = torch.from_numpy(ev["key"].view(np.int32)).to(dev)
    d_app = torch.from_numpy(ev["app"].view(np.int32)).to(dev)
    d_ph = torch.from_numpy(ev["phase"]).to(dev)
    d_dur = torch.from_numpy(ev["dur_ns"]).to(dev)
    d_c = torch.from_numpy(c.view(np.int32)).to(dev)
    d_sk = torch.from_numpy(keys.view(np.int32)).to(dev)
    d_s = torch.from_numpy(s).to(dev)
    torch.cuda.synchronize()
    max_groups = keys.size * P

    def make(timing: bool):
        return X.Aggregator(P, d_c, max_events=n, max_groups=max_groups, max_keys=keys.size,
                            max_score=keys.size, path=args.path, timing=timing)

    ag = make(False)
    gbuf = ag.group_buffers(max_groups)
    sbuf = dict(op=torch.empty(keys.size, dtype=torch.int32, device=dev),
                op_weight=torch.empty(keys.size, dtype=torch.float64, device=dev),
                op_score=torch.empty(keys.size, dtype=torch.float64, device=dev))
    result = {}

    def step(a, times=None):
        if times is None:  # the whole path in one library call (atrex_run)
            r = a.run(d_key, d_app, d_ph, d_dur, gbuf, d_sk, d_s, sbuf)
            result["groups"], result["score"] = r["groups"], r["score"]
            return
        # per-kernel times: the calls one by one (times are kept per call)
        a.reset()
        a.aggregate(d_key, d_app, d_ph, d_dur)
        if times is not None:
            times.extend(a.kernel_times())
        out = a.normalize(out=gbuf)
        if times is not None:
            times.extend(a.kernel_times())
        result["groups"] = out
        result["score"] = a.score(d_sk, d_s, out=sbuf)
        if times is not None:
            times.extend(a.kernel_times())

    for _ in range(args.warmup):
        step(ag)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(ag)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0
    ms_step = 1e3 * elapsed / args.steps
    value = n * args.steps / elapsed / 1e9
    log("step %.3f ms, %.2f G events/s, path %s" % (ms_step, value, ag.path_used()))

    # sanity of the timed result: every invocation counted, each phase sums to 1
    g = result["groups"]
    assert int(g["count"].sum().item()) == n, "event count mismatch"
    wsum_phase = torch.zeros(P, dtype=torch.float64, device=dev).index_add_(0, g["phase"].long(), g["weight"])
    assert torch.allclose(wsum_phase, torch.ones_like(wsum_phase), atol=1e-9), "phase weights"

    # per-kernel device times (hipEvents recorded by the library on its stream)
    agt = make(True)
    per = {}
    for _ in range(3):
        times = []
        step(agt, times)
        for name, ms, items in times:
            per.setdefault(name, []).append((ms, items))
    kernels = {k: dict(avg_ms=sum(m for m, _ in v) / len(v), items=v[0][1]) for k, v in per.items()}
    agt.close()
    dom = max((k for k in kernels if k in KERNEL_BYTES), key=lambda k: kernels[k]["avg_ms"])
    alg = KERNEL_BYTES[dom] * n
    achieved = alg / (kernels[dom]["avg_ms"] * 1e-3) / 1e9
    traffic = traffic_from_profile(cfg["slug"], dom, n)
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "algorithmic_bytes_per_launch": alg, "avg_launch_ms": round(kernels[dom]["avg_ms"], 4)}
    log("kernels", json.dumps({k: round(v["avg_ms"], 4) for k, v in kernels.items()}))

    cpu = None
    if not args.no_cpu_baseline:
        from oracle import oracle as O  # the CPU baseline leg is the oracle, timed as it stands
        m = min(n, 1 << args.cpu_sample_log2)
        log("cpu oracle on the first %d events" % m)
        tc = time.perf_counter()
        O.run(ev["key"][:m], ev["app"][:m], ev["phase"][:m], ev["dur_ns"][:m], c, P,
              score_key=keys, s=s, want_units=True)
        dt = time.perf_counter() - tc
        cpu = {"value": round(m / dt / 1e9, 6), "unit": "G events/s", "cores": 1, "kind": "oracle",
               "sample": "first %d events of the same workload (full path incl. score), %.1f s" % (m, dt)}

    line = {
        "metric": "trace events aggregated/sec (G ev/s) + % of MI355X peak HBM BW",
        "value": round(value, 3),
        "unit": "G events/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u128",
        "data": "synthetic",
        "config": {"workload": cfg["name"], "events": n, "keys": int(keys.size), "phases": P,
                   "apps": cfg["num_apps"], "seed": cfg["seed"], "path": ag.path_used(),
                   "parallelism": "none", "entry": "atrex_run"},
        "hbm_frac_30B": round(30 * value * 1e9 / (HBM_PEAK_GBS * 1e9), 4),
        "hbm_frac_17B": round(17 * value * 1e9 / (HBM_PEAK_GBS * 1e9), 4),
        "kernels_ms": {k: round(v["avg_ms"], 4) for k, v in kernels.items()},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    ag.close()
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
