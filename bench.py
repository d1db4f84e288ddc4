#!/usr/bin/env python3
"""Benchmark of the trace-event -> importance-weight path on one MI355X.

One step = the whole path over one batch of events already resident in HBM:
pass A (per-(app, phase) time, Eq. (2)), the Q96 scale (Eq. (3)), pass B
(per-(key, phase) shares), compaction/ordering, per-phase normalisation and
Eq. (3) per operator and key, and the importance-weighted score (Eq. (4)-(6)),
in one library call (atrex_run).  The default workload is the largest: 1B
events over 64k Zipf(0.9) keys, 3 phases, 100k apps.

Prints one JSON line: throughput in G events/s; the roofline of the dominant
kernel (the event bytes the method reads -- 13 per event in pass A, 17 in
pass B -- over its hipEvent time, taken by the library on the stream the
kernels run on); a parity self-check of the timed step's outputs against the
CPU oracle's (digests written by tests/golden/make_digests.py; a mismatch
makes the run fail); and the CPU oracle timed on bounded samples of the same
workload, on one core and sharded over the host's cores.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3] [--path auto]

--row share measures the target-DSL device-time share instead (§4.1, Metrics:
the plain device-time group-by of one profile's kernel invocations and the
per-shape, per-operator and overall shares), on the 64M-invocation profile by
default (--config picks 0..2 of the profile workloads).  --row refresh
measures an incremental refresh of the weights over an append-only log (the
workload's events, the last eighth new), beside a from-scratch run.  --row
stats measures the observed runtime per unit (count, total, mean, min, max,
median, p99) on a profile workload; --row join the host/device correlation
join that labels raw kernel records.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E peak, GB/s
BYTES_PASS_A = 13              # app u32 + phase u8 + dur i64 per event
BYTES_PASS_B = 17              # key u32 + app u32 + phase u8 + dur i64 per event
# the event bytes of the method each kernel reads (the kernels that stream
# the events); the other kernels' traffic is the engine's own
METHOD_BYTES = {"pass_a": BYTES_PASS_A, "pass_a_range": BYTES_PASS_A, "pass_a_global": BYTES_PASS_A,
                "pass_b_lds": BYTES_PASS_B, "pass_b_global": BYTES_PASS_B, "part_scatter": BYTES_PASS_B,
                "hot_scatter": BYTES_PASS_B}
PASS_A_KERNELS = ("pass_a", "pass_a_range", "pass_a_global", "pass_a_reduce", "scale")
# pass B: every kernel from the scale words to the (key, phase) rows
PASS_B_KERNELS = ("seed", "seed_image", "pass_b_lds", "pass_b_global", "compact_rows", "owner_finish",
                  "part_hist", "part_scatter", "part_aggregate", "part_hist_spill", "part_scatter_spill",
                  "part_aggregate_spill", "part_hist_cold", "hot_scatter", "part_aggregate_cold")
# bytes per event each partition-engine kernel moves besides the method's:
# histogram (key re-read), scatter (16-byte record written), aggregate (record
# read); the hot scatter writes records only for the events of keys outside
# its table, so its figures are upper bounds
ENGINE_BYTES = {"part_hist": 4, "part_scatter": 16, "part_aggregate": 16,
                "part_hist_cold": 4, "hot_scatter": 16, "part_aggregate_cold": 16}
KERNEL_SOURCES = ["paper_2607_14541_amd/csrc/kernels_aggregate.hip",
                  "paper_2607_14541_amd/csrc/kernels_rows.hip",
                  "paper_2607_14541_amd/csrc/kernels_share.hip",
                  "paper_2607_14541_amd/csrc/atrex_kernels.h",
                  "paper_2607_14541_amd/csrc/atrex_device.hpp"]
DEFAULT_STEPS = {0: 200, 1: 200, 2: 40, 3: 20, 4: 30}
# events of each workload the CPU oracle is timed on: (one thread, all threads)
CPU_SAMPLE_LOG2 = {0: (20, 20), 1: (24, 26), 2: (20, 22), 3: (21, 23), 4: (24, 26)}


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """Hash of the streaming kernels' sources without comments and blank lines
    (a change to the code, not to its comments, invalidates stored counters)."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, f)) as fh:
            text = re.sub(r"/\*.*?\*/", "", fh.read(), flags=re.S)
        for line in text.splitlines():
            code = line.split("//", 1)[0].rstrip()
            if code.strip():
                h.update(code.encode() + b"\n")
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


def host_threads() -> int:
    """Threads for the sharded CPU oracle: the host's share of cores (the
    OMP_NUM_THREADS the environment sets, else the CPUs this process may run
    on), at most 16."""
    env = os.environ.get("OMP_NUM_THREADS")
    n = int(env) if env and env.isdigit() else len(os.sched_getaffinity(0))
    return max(1, min(16, n))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def kernel_averages(runs) -> dict:
    """{name: {avg_ms, items}} from lists of (name, ms, items) per repetition:
    a name's launches within one repetition are summed, then averaged over
    the repetitions."""
    per = {}
    for times in runs:
        tot = {}
        for name, ms, items in times:
            t = tot.setdefault(name, [0.0, items])
            t[0] += ms
        for name, (ms, items) in tot.items():
            per.setdefault(name, []).append((ms, items))
    return {k: dict(avg_ms=sum(m for m, _ in v) / len(v), items=v[0][1]) for k, v in per.items()}


# event bytes the target-share kernels read: phase + dur in the per-phase
# totals, key + phase + dur in the per-(key, phase) group-by
SHARE_METHOD_BYTES = {"time_totals": 9, "pass_b_lds": 13, "pass_b_global": 13, "part_scatter": 13}
SHARE_DEFAULT_STEPS = {0: 200, 1: 100, 2: 100}


def bench_share(args) -> int:
    import numpy as np
    import torch
    from paper_2607_14541_amd import atrex as X
    from paper_2607_14541_amd import synth

    ci = 1 if args.config is None else args.config
    cfg = synth.SHARE_CONFIGS[ci]
    n = cfg["n"]
    steps = args.steps if args.steps is not None else SHARE_DEFAULT_STEPS[ci]
    units = synth.profile_units(cfg)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log("target share, profile", ci, cfg["name"])
    p = synth.profile(cfg)
    d_key = torch.from_numpy(p["key"].view(np.int32)).to(dev)
    d_flag = torch.from_numpy(p["is_dsl"]).to(dev)
    d_dur = torch.from_numpy(p["dur_ns"]).to(dev)
    torch.cuda.synchronize()
    K = units.size

    def make(timing: bool):
        return X.Aggregator(2, None, max_events=n, max_keys=K, max_groups=2 * K, path=args.path, timing=timing,
                            device_time=True)

    ag = make(False)
    sbuf = ag.share_buffers(K, min(K, 65536))
    res = {}

    def step(a):  # one profile: device-time group-by, then the shares
        a.reset()
        a.aggregate(d_key, None, d_flag, d_dur)
        res["r"] = a.target_share(out=sbuf)

    for _ in range(args.warmup):
        step(ag)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step(ag)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = 1e3 * elapsed / steps
    value = n * steps / elapsed / 1e9
    log("step %.3f ms, %.2f G invocations/s, path %s" % (ms_step, value, ag.path_used()))

    parity = None
    o = None
    if not args.no_parity or not args.no_cpu_baseline:
        from oracle import oracle as O  # checker and CPU baseline: the oracle as it stands
        tc = time.perf_counter()
        o = O.target_share(p["key"], p["is_dsl"], p["dur_ns"])
        t_oracle = time.perf_counter() - tc
    if not args.no_parity:
        r = res["r"]

        def f64_same(a, b):
            a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
            return a.shape == b.shape and np.array_equal(np.isnan(a), np.isnan(b)) and np.array_equal(
                a[~np.isnan(a)].view(np.uint64), b[~np.isnan(b)].view(np.uint64))
        bad = [k for k, ok in (
            ("key", np.array_equal(r["key"].cpu().numpy().view(np.uint32), o["key"])),
            ("count", np.array_equal(r["count"].cpu().numpy().view(np.uint64), o["count"])),
            ("dsl_ns", np.array_equal(r["dsl_ns"].cpu().numpy().view(np.uint64), o["dsl_ns"])),
            ("total_ns", np.array_equal(r["total_ns"].cpu().numpy().view(np.uint64), o["total_ns"])),
            ("share", f64_same(r["share"].cpu().numpy(), o["share"])),
            ("op", np.array_equal(r["op"].cpu().numpy().view(np.uint32), o["op"])),
            ("op_shapes", np.array_equal(r["op_shapes"].cpu().numpy().view(np.uint32), o["op_shapes"])),
            ("op_share", f64_same(r["op_share"].cpu().numpy(), o["op_share"])),
            ("adoption", f64_same([r["adoption"]], [o["adoption"]]))) if not ok]
        parity = {"checked": True, "against": "CPU oracle on the same profile, every output", "ok": not bad,
                  "mismatch": bad}
        log("parity", "ok" if not bad else "MISMATCH %s" % bad)

    agt = make(True)
    runs = []
    for _ in range(5):
        agt.reset()
        agt.aggregate(d_key, None, d_flag, d_dur)
        t = agt.kernel_times()
        agt.target_share(out=sbuf)
        runs.append(t + agt.kernel_times())
    agt.close()
    kernels = kernel_averages(runs)
    dom = max((k for k in kernels if k in SHARE_METHOD_BYTES), key=lambda k: kernels[k]["avg_ms"])
    alg = SHARE_METHOD_BYTES[dom] * n
    achieved = alg / (kernels[dom]["avg_ms"] * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                "algorithmic_bytes_per_launch": alg, "avg_launch_ms": round(kernels[dom]["avg_ms"], 4)}
    log("kernels", json.dumps({k: round(v["avg_ms"], 4) for k, v in kernels.items()}))
    cpu = None
    if not args.no_cpu_baseline:
        cpu = {"value": round(n / t_oracle / 1e9, 6), "unit": "G invocations/s", "cores": 1, "kind": "oracle",
               "sample": "the whole %d-invocation profile, one thread (%.1f s)" % (n, t_oracle),
               "nproc": os.cpu_count(), "cpu_model": cpu_model()}
    r = res["r"]
    line = {
        "metric": "profile kernel invocations folded into the target-DSL device-time share per second",
        "value": round(value, 3), "unit": "G invocations/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "u128+f64", "data": "synthetic",
        "config": {"workload": cfg["name"], "invocations": n, "units": int(K), "operators": cfg["ops"],
                   "seed": cfg["seed"], "path": ag.path_used(), "parallelism": "none",
                   "entry": "atrex_aggregate_events + atrex_target_share"},
        "adoption": r["adoption"], "defined_ops": r["defined_ops"],
        "kernels_ms": {k: round(v["avg_ms"], 4) for k, v in kernels.items()},
        "parity": parity, "roofline": roofline, "cpu_baseline": cpu,
    }
    ag.close()
    print(json.dumps(line), flush=True)
    return 1 if parity is not None and not parity["ok"] else 0


# event bytes the unit-statistics kernels read per event: key + phase + dur
# while placing the durations, the duration in each select round
STATS_METHOD_BYTES = {"stats_scatter": 13}
STATS_Q = (50000, 99000)


def bench_stats(args) -> int:
    """Observed runtime per unit (§3.1, the deployment baseline): a step is the
    device-time group-by of a profile's invocations and the per-unit count,
    total, mean, min, max, median and p99 (atrex_unit_stats), units = keys
    with their phases merged."""
    import numpy as np
    import torch
    from paper_2607_14541_amd import atrex as X
    from paper_2607_14541_amd import synth

    ci = 1 if args.config is None else args.config
    cfg = synth.SHARE_CONFIGS[ci]
    n = cfg["n"]
    steps = args.steps if args.steps is not None else SHARE_DEFAULT_STEPS[ci] // 2
    units = synth.profile_units(cfg)
    K = units.size
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log("unit statistics, profile", ci, cfg["name"])
    p = synth.profile(cfg)
    d_key = torch.from_numpy(p["key"].view(np.int32)).to(dev)
    d_ph = torch.from_numpy(p["is_dsl"]).to(dev)
    d_dur = torch.from_numpy(p["dur_ns"]).to(dev)
    torch.cuda.synchronize()

    def make(timing: bool):
        return X.Aggregator(2, None, max_events=n, max_keys=K, max_groups=2 * K, path=args.path, timing=timing,
                            device_time=True)

    ag = make(False)
    sbuf = ag.stats_buffers(2 * K, len(STATS_Q))
    res = {}

    def step(a):
        a.reset()
        a.aggregate(d_key, None, d_ph, d_dur)
        res["r"] = a.unit_stats(d_key, d_ph, d_dur, q_1e5=STATS_Q, by_phase=False, out=sbuf)

    for _ in range(args.warmup):
        step(ag)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step(ag)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_step = 1e3 * elapsed / steps
    value = n * steps / elapsed / 1e9
    log("step %.3f ms, %.2f G invocations/s, path %s" % (ms_step, value, ag.path_used()))
    parity, cpu = None, None
    if not args.no_parity:
        from oracle import oracle as O  # the checker
        o = O.unit_stats(p["key"], p["is_dsl"], p["dur_ns"], 2, q_1e5=STATS_Q, by_phase=False)
        r = res["r"]
        bad = [k for k, a, b in (
            ("key", r["key"].cpu().numpy().view(np.uint32), o["key"]),
            ("count", r["count"].cpu().numpy().view(np.uint64), o["count"]),
            ("total_ns", r["total_ns"].cpu().numpy().view(np.uint64), o["total_ns"]),
            ("mean_ns", r["mean_ns"].cpu().numpy().view(np.uint64), o["mean_ns"].view(np.uint64)),
            ("min_ns", r["min_ns"].cpu().numpy(), o["min_ns"]), ("max_ns", r["max_ns"].cpu().numpy(), o["max_ns"]),
            ("quantile_ns", r["quantile_ns"].cpu().numpy(), o["quantile_ns"])) if not np.array_equal(a, b)]
        parity = {"checked": True, "against": "CPU oracle on the same profile, every output", "ok": not bad,
                  "mismatch": bad}
        log("parity", "ok" if not bad else "MISMATCH %s" % bad)
    agt = make(True)
    runs = []
    for _ in range(5):
        agt.reset()
        agt.aggregate(d_key, None, d_ph, d_dur)
        t = agt.kernel_times()
        agt.unit_stats(d_key, d_ph, d_dur, q_1e5=STATS_Q, by_phase=False, out=sbuf)
        runs.append(t + agt.kernel_times())
    agt.close()
    kernels = kernel_averages(runs)
    dom = "stats_scatter"
    alg = STATS_METHOD_BYTES[dom] * n
    achieved = alg / (kernels[dom]["avg_ms"] * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                "algorithmic_bytes_per_launch": alg, "avg_launch_ms": round(kernels[dom]["avg_ms"], 4),
                "select_rounds_ms": round(kernels.get("stats_select", {}).get("avg_ms", 0.0), 4)}
    log("kernels", json.dumps({k: round(v["avg_ms"], 4) for k, v in kernels.items()}))
    if not args.no_cpu_baseline:
        from oracle import oracle as O
        m = min(n, 1 << 24)
        tc = time.perf_counter()
        O.unit_stats(p["key"][:m], p["is_dsl"][:m], p["dur_ns"][:m], 2, q_1e5=STATS_Q, by_phase=False)
        dt = time.perf_counter() - tc
        cpu = {"value": round(m / dt / 1e9, 6), "unit": "G invocations/s", "cores": 1, "kind": "oracle",
               "sample": "first %d invocations of the same profile, one thread (%.1f s)" % (m, dt),
               "nproc": os.cpu_count(), "cpu_model": cpu_model()}
    line = {
        "metric": "profile kernel invocations summarised into per-unit runtime statistics per second",
        "value": round(value, 3), "unit": "G invocations/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "int64+u128", "data": "synthetic",
        "config": {"workload": cfg["name"], "invocations": n, "units": int(K), "quantiles_1e5": list(STATS_Q),
                   "seed": cfg["seed"], "path": ag.path_used(), "parallelism": "none",
                   "entry": "atrex_aggregate_events + atrex_unit_stats"},
        "kernels_ms": {k: round(v["avg_ms"], 4) for k, v in kernels.items()},
        "parity": parity, "roofline": roofline, "cpu_baseline": cpu,
    }
    ag.close()
    print(json.dumps(line), flush=True)
    return 1 if parity is not None and not parity["ok"] else 0


# bytes the correlation join must move per kernel record (corr 8, anchor 8,
# stream 4, start 8, end 8 read) and per labelled event (key 4, app 4,
# phase 1, dur 8 written); host records (kind 1, id 8, key 4, app 4, phase 1)
# are read once
JOIN_READ_PER_KERNEL, JOIN_WRITE_PER_EVENT, JOIN_READ_PER_HOST = 36, 17, 18
JOIN_DEFAULT_STEPS = {0: 100, 1: 20}


def bench_join(args) -> int:
    """Host/device correlation join (§3.1): a step labels one trace's device
    kernel records from its host records (correlation ids, graph anchors,
    stream intervals) and writes the labelled events (atrex_correlate)."""
    import numpy as np
    import torch
    from paper_2607_14541_amd import atrex as X
    from paper_2607_14541_amd import synth

    ci = 1 if args.config is None else args.config
    jc = synth.JOIN_CONFIGS[ci]
    steps = args.steps if args.steps is not None else JOIN_DEFAULT_STEPS[ci]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log("correlation join", ci, jc["name"])
    t = time.time()
    tr = synth.join_trace(jc)
    log("generated in %.1fs" % (time.time() - t))
    n, m, mi = tr["kind"].size, tr["host"]["id"].size, tr["intervals"]["stream"].size

    np_of = {torch.int64: np.int64, torch.int32: np.int32, torch.uint8: np.uint8}

    def up(d, spec):
        return {f: torch.from_numpy(np.ascontiguousarray(d[f]).view(np_of[dt])).to(dev) for f, dt in spec}
    k = up(tr["kernels"], X.Correlator.KERNEL_FIELDS)
    h = up(tr["host"], X.Correlator.HOST_FIELDS)
    iv = up(tr["intervals"], X.Correlator.INTERVAL_FIELDS)
    c = X.Correlator(n, m, device=dev)
    out = c.buffers(n)
    src = torch.empty(n, dtype=torch.uint8, device=dev)
    res = {}

    def step():
        res["r"] = c.run(k, h, iv, out=out, source=src)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record()
    for _ in range(steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_dev = ev0.elapsed_time(ev1) / steps
    ms_step = 1e3 * elapsed / steps
    value = n * steps / elapsed / 1e9
    r = res["r"]
    L = r["labelled"]
    log("step %.3f ms (%.3f ms between hipEvents), %.2f G records/s, labelled %d, method %s" % (
        ms_step, ms_dev, value, L, r["method"]))
    # the other method on the same trace, for comparison (not the metric)
    other = "hash" if r["method"] == "partition" else None
    ms_other = None
    if other:
        c2 = X.Correlator(n, m, device=dev, method=other)
        c2.run(k, h, iv, out=out, source=src)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        reps = max(3, steps // 4)
        for _ in range(reps):
            c2.run(k, h, iv, out=out, source=src)
        e1.record()
        torch.cuda.synchronize()
        ms_other = e0.elapsed_time(e1) / reps
        del c2
        log("the %s join on the same trace: %.3f ms" % (other, ms_other))
        step()  # the timed method's outputs again, for the parity check
        torch.cuda.synchronize()
        r = res["r"]
    parity = None
    if not args.no_parity:
        msk = tr["kind"] < 3
        bad = [f for f, a, b in (("source", r["source"].cpu().numpy(), tr["kind"]),
                                 ("key", r["key"].cpu().numpy().view(np.uint32), tr["truth"]["key"][msk]),
                                 ("app", r["app"].cpu().numpy().view(np.uint32), tr["truth"]["app"][msk]),
                                 ("phase", r["phase"].cpu().numpy(), tr["truth"]["phase"][msk]),
                                 ("dur_ns", r["dur_ns"].cpu().numpy(), tr["truth"]["dur_ns"][msk]))
               if not np.array_equal(a, b)]
        parity = {"checked": True, "against": "the labelled events the records were built from (the oracle "
                  "recovers them exactly at the sizes its tests run)", "ok": not bad, "mismatch": bad}
        log("parity", "ok" if not bad else "MISMATCH %s" % bad)
    alg = JOIN_READ_PER_KERNEL * n + JOIN_WRITE_PER_EVENT * L + JOIN_READ_PER_HOST * m
    achieved = alg / (ms_dev * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": "atrex_correlate (%s join: every kernel of the call)" % r["method"],
                "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                "algorithmic_bytes_per_launch": alg, "avg_launch_ms": round(ms_dev, 4)}
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import oracle as O  # the CPU baseline leg: the oracle as it stands
        sub = synth.join_trace(jc, n=1 << 21)
        tc = time.perf_counter()
        O.correlate(sub["kernels"], sub["host"], sub["intervals"])
        dt = time.perf_counter() - tc
        cpu = {"value": round((1 << 21) / dt / 1e9, 6), "unit": "G records/s", "cores": 1, "kind": "oracle",
               "sample": "a 2097152-record trace of the same recipe, one thread (%.1f s)" % dt,
               "nproc": os.cpu_count(), "cpu_model": cpu_model()}
    line = {
        "metric": "device kernel records labelled by the host/device correlation join per second",
        "value": round(value, 3), "unit": "G records/s", "n_gpus": 1, "steps": steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "u64 ids", "data": "synthetic",
        "config": {"workload": jc["name"], "kernel_records": n, "host_records": m, "intervals": mi,
                   "streams": jc["streams"], "seed": jc["seed"], "parallelism": "none", "entry": "atrex_correlate"},
        "labelled": L, "by_source": r["by_source"], "ms_between_events": round(ms_dev, 4),
        "method": r["method"], "ms_hash_join": round(ms_other, 4) if ms_other else None,
        "parity": parity, "roofline": roofline, "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 1 if parity is not None and not parity["ok"] else 0


def bench_refresh(args) -> int:
    """Incremental refresh: the workload's events are an append-only log whose
    last eighth is new; a step restores the folded totals of the first seven
    eighths (a checkpoint), folds the new events (pass A over them only),
    re-runs pass B over the whole log, orders, normalises and scores.  The
    same log re-weighted from scratch (atrex_run) is timed beside it."""
    import numpy as np
    import torch
    from paper_2607_14541_amd import atrex as X
    from paper_2607_14541_amd import synth

    ci = 3 if args.config is None else args.config
    cfg = synth.CONFIGS[ci]
    n, P = cfg["n"], cfg["num_phases"]
    n_new = n // 8
    n_old = n - n_new
    steps = args.steps if args.steps is not None else max(5, DEFAULT_STEPS[ci] // 2)
    keys = synth.key_space(cfg)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log("refresh, config", ci, cfg["name"], "log", n, "new", n_new)
    ev = synth.events(cfg)
    c = synth.app_weights(cfg)
    s = synth.scores(cfg, keys)
    d = {k: torch.from_numpy(ev[k].view(dt)).to(dev) for k, dt in (("key", np.int32), ("app", np.int32),
                                                                     ("phase", np.uint8), ("dur_ns", np.int64))}
    d_c = torch.from_numpy(c.view(np.int32)).to(dev)
    d_sk = torch.from_numpy(keys.view(np.int32)).to(dev)
    d_s = torch.from_numpy(s).to(dev)
    torch.cuda.synchronize()
    if args.no_cpu_baseline:
        del ev
    G = keys.size * P
    kw = dict(max_events=n, max_groups=G, max_keys=keys.size, max_score=keys.size, path=args.path)
    ag = X.Aggregator(P, d_c, incremental=True, **kw)
    old = {k: v[:n_old] for k, v in d.items()}
    ag.refresh(old["key"], old["app"], old["phase"], old["dur_ns"], n_old)
    state = ag.refresh_state()
    gbuf = ag.group_buffers(G)
    sbuf = dict(op=torch.empty(keys.size, dtype=torch.int32, device=dev),
                op_weight=torch.empty(keys.size, dtype=torch.float64, device=dev),
                op_score=torch.empty(keys.size, dtype=torch.float64, device=dev))
    res = {}

    def step(a):
        a.reset()
        a.refresh_restore(state)
        a.refresh(d["key"], d["app"], d["phase"], d["dur_ns"], n_new)
        res["groups"] = a.normalize(out=gbuf)
        res["score"] = a.score(d_sk, d_s, out=sbuf)

    def timed(fn, k):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(k):
            fn()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) / k

    t_refresh = timed(lambda: step(ag), steps)
    full = X.Aggregator(P, d_c, **kw)
    fb = full.group_buffers(G)
    t_full = timed(lambda: full.run(d["key"], d["app"], d["phase"], d["dur_ns"], fb, d_sk, d_s, sbuf), steps)
    full.close()
    log("refresh %.3f ms, whole log from scratch %.3f ms" % (1e3 * t_refresh, 1e3 * t_full))

    parity = None
    if not args.no_parity:
        sys.path.insert(0, os.path.join(ROOT, "tests", "golden"))
        import digests as D
        rec = D.load()["configs"].get(str(ci)) if os.path.exists(D.DIGEST_FILE) else None
        if rec is None:
            parity = {"checked": False, "reason": "no oracle digest for this workload"}
        else:
            out = {k: v.cpu().numpy() for k, v in res["groups"].items()}
            out.update(score_op=res["score"]["op"].cpu().numpy(),
                       score_op_weight=res["score"]["op_weight"].cpu().numpy(),
                       score_op_S=res["score"]["op_score"].cpu().numpy())
            ow, kwt, at = ag.op_weights(), ag.key_weights(), ag.app_totals()
            out.update(op=ow["op"].cpu().numpy(), op_U=ow["U"].cpu().numpy(), op_w=ow["w"].cpu().numpy(),
                       ukey=kwt["key"].cpu().numpy(), key_U=kwt["U"].cpu().numpy(), omega=kwt["omega"].cpu().numpy(),
                       app_total=at["T"].cpu().numpy(), mant=at["mant"].cpu().numpy(), rho=at["rho"].cpu().numpy())
            bad = D.mismatches(rec, out, s_agg=res["score"]["s_agg"])
            parity = {"checked": True, "against": "CPU oracle over the whole log (digests of its outputs)",
                      "ok": not bad, "mismatch": bad}
            log("parity", "ok" if not bad else "MISMATCH %s" % bad)

    agt = X.Aggregator(P, d_c, incremental=True, timing=True, **kw)
    runs = []
    for _ in range(3):
        agt.reset()
        agt.refresh_restore(state)
        agt.refresh(d["key"], d["app"], d["phase"], d["dur_ns"], n_new)
        runs.append(agt.kernel_times())
    agt.close()
    kernels = kernel_averages(runs)
    dom = max((k for k in kernels if k in METHOD_BYTES), key=lambda k: kernels[k]["avg_ms"])
    # pass-A kernels read the new events only
    units = n_new if dom in ("pass_a", "pass_a_range", "pass_a_global") else n
    alg = METHOD_BYTES[dom] * units
    achieved = alg / (kernels[dom]["avg_ms"] * 1e-3) / 1e9
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                "algorithmic_bytes_per_launch": alg, "avg_launch_ms": round(kernels[dom]["avg_ms"], 4)}
    log("kernels", json.dumps({k: round(v["avg_ms"], 4) for k, v in kernels.items()}))
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import oracle as O  # a refresh's result is the oracle over the whole log
        l1, lt = CPU_SAMPLE_LOG2[ci]
        threads = host_threads()
        m = min(n, 1 << lt)
        tc = time.perf_counter()
        O.run(ev["key"][:m], ev["app"][:m], ev["phase"][:m], ev["dur_ns"][:m], c, P, score_key=keys, s=s,
              threads=threads)
        dt = time.perf_counter() - tc
        cpu = {"value": round(m / dt / 1e9, 6), "unit": "G events/s", "cores": threads, "kind": "oracle",
               "sample": "first %d events of the log, whole path incl. score, group-by sharded over %d threads "
                         "(%.1f s)" % (m, threads, dt), "nproc": os.cpu_count(), "cpu_model": cpu_model()}
    line = {
        "metric": "log events re-weighted per second by an incremental refresh (1/8 of the log new)",
        "value": round(n / t_refresh / 1e9, 3), "unit": "G events/s", "n_gpus": 1, "steps": steps,
        "warmup": args.warmup, "ms_per_step": round(1e3 * t_refresh, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u128", "data": "synthetic",
        "config": {"workload": cfg["name"], "log_events": n, "new_events": n_new, "seed": cfg["seed"],
                   "path": ag.path_used(), "parallelism": "none",
                   "entry": "atrex_refresh_restore + atrex_refresh + atrex_phase_normalize + atrex_weighted_score"},
        "ms_whole_log_from_scratch": round(1e3 * t_full, 4), "speedup_vs_from_scratch": round(t_full / t_refresh, 3),
        "kernels_ms": {k: round(v["avg_ms"], 4) for k, v in kernels.items()},
        "parity": parity, "roofline": roofline, "cpu_baseline": cpu,
    }
    ag.close()
    print(json.dumps(line), flush=True)
    return 1 if parity is not None and parity.get("checked") and not parity["ok"] else 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=None, help="workload index (0..4); default 3 = 1B events")
    ap.add_argument("--row", default="weights", choices=["weights", "share", "refresh", "stats", "join"],
                    help="weights: the importance-weight path (default); share: the target-DSL share; "
                         "refresh: an incremental refresh of an append-only log; stats: runtime statistics per unit; "
                         "join: the host/device correlation join")
    ap.add_argument("--path", default="auto", choices=["auto", "lds_hash", "global_hash", "radix_sort"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-parity", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(--gpus %d requested)" % args.gpus, file=sys.stderr)
        return 2
    if args.row == "share":
        return bench_share(args)
    if args.row == "refresh":
        return bench_refresh(args)
    if args.row == "stats":
        return bench_stats(args)
    if args.row == "join":
        return bench_join(args)
    if args.config is None:
        args.config = 3
    steps = args.steps if args.steps is not None else DEFAULT_STEPS[args.config]

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
    if args.no_cpu_baseline:
        del ev
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

    def step(a):  # the whole path in one library call (atrex_run)
        r = a.run(d_key, d_app, d_ph, d_dur, gbuf, d_sk, d_s, sbuf)
        result["groups"], result["score"] = r["groups"], r["score"]

    for _ in range(args.warmup):
        step(ag)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step(ag)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0
    ms_step = 1e3 * elapsed / steps
    value = n * steps / elapsed / 1e9
    log("step %.3f ms, %.2f G events/s, path %s, one wait %s" % (ms_step, value, ag.path_used(), ag.one_wait))

    # parity of the timed step's outputs with the CPU oracle's (digests)
    parity = None
    if not args.no_parity:
        sys.path.insert(0, os.path.join(ROOT, "tests", "golden"))
        import digests as D
        rec = D.load()["configs"].get(str(args.config)) if os.path.exists(D.DIGEST_FILE) else None
        if rec is None:
            parity = {"checked": False, "reason": "no oracle digest for this workload"}
        else:
            def h(x):
                a = x.cpu().numpy()
                return a
            out = {k: h(v) for k, v in result["groups"].items()}
            out.update(score_op=h(result["score"]["op"]), score_op_weight=h(result["score"]["op_weight"]),
                       score_op_S=h(result["score"]["op_score"]))
            ow, kw, at = ag.op_weights(), ag.key_weights(), ag.app_totals()
            out.update(op=h(ow["op"]), op_U=h(ow["U"]), op_w=h(ow["w"]), ukey=h(kw["key"]), key_U=h(kw["U"]),
                       omega=h(kw["omega"]), app_total=h(at["T"]), mant=h(at["mant"]), rho=h(at["rho"]))
            bad = D.mismatches(rec, out, s_agg=result["score"]["s_agg"])
            parity = {"checked": True, "against": "CPU oracle (digests of its outputs on this workload)",
                      "outputs": len([k for k in rec["digests"] if k in out]) + 1, "ok": not bad,
                      "mismatch": bad}
            log("parity", "ok" if not bad else "MISMATCH %s" % bad)

    # aggregate-only time (pass A, scale, pass B, ordering) and the whole step
    # with a 512 MB write before each repetition (no cache residency), medians
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    reps = max(3, min(10, steps))
    t_agg, t_flush = [], []
    for _ in range(reps):
        flush.fill_(1)
        torch.cuda.synchronize()
        ta = time.perf_counter()
        ag.reset()
        ag.aggregate(d_key, d_app, d_ph, d_dur)
        t_agg.append(time.perf_counter() - ta)
        flush.fill_(2)
        torch.cuda.synchronize()
        ta = time.perf_counter()
        step(ag)
        t_flush.append(time.perf_counter() - ta)
    del flush

    # per-kernel device times (hipEvents recorded by the library on its stream)
    agt = make(True)
    runs = []
    for _ in range(3):
        times = []
        agt.reset()
        agt.aggregate(d_key, d_app, d_ph, d_dur)
        times.extend(agt.kernel_times())
        out_g = agt.normalize(out=gbuf)
        times.extend(agt.kernel_times())
        agt.score(d_sk, d_s, out=sbuf)
        times.extend(agt.kernel_times())
        del out_g
        runs.append(times)
    kernels = kernel_averages(runs)
    agt.close()
    dom = max((k for k in kernels if k in METHOD_BYTES), key=lambda k: kernels[k]["avg_ms"])
    alg = METHOD_BYTES[dom] * n
    achieved = alg / (kernels[dom]["avg_ms"] * 1e-3) / 1e9
    traffic = traffic_from_profile(cfg["slug"], dom, n)
    t_a = sum(v["avg_ms"] for k, v in kernels.items() if k in PASS_A_KERNELS)
    t_b = sum(v["avg_ms"] for k, v in kernels.items() if k in PASS_B_KERNELS)
    engine_extra = sum(b for k, b in ENGINE_BYTES.items() if k in kernels)
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": traffic,
                "algorithmic_bytes_per_launch": alg, "avg_launch_ms": round(kernels[dom]["avg_ms"], 4),
                "pass_a_frac": round(BYTES_PASS_A * n / (t_a * 1e-3) / 1e9 / HBM_PEAK_GBS, 4) if t_a else None,
                "pass_b_frac": round(BYTES_PASS_B * n / (t_b * 1e-3) / 1e9 / HBM_PEAK_GBS, 4) if t_b else None,
                "engine_extra_bytes_per_event": engine_extra}
    log("kernels", json.dumps({k: round(v["avg_ms"], 4) for k, v in kernels.items()}))

    cpu = None
    if not args.no_cpu_baseline:
        from oracle import oracle as O  # the CPU baseline leg is the oracle, timed as it stands
        l1, lt = CPU_SAMPLE_LOG2[args.config]
        threads = host_threads()
        res = {}
        for th, lg in ((1, l1), (threads, lt)):
            m = min(n, 1 << lg)
            log("cpu oracle on the first %d events, %d thread(s)" % (m, th))
            tc = time.perf_counter()
            O.run(ev["key"][:m], ev["app"][:m], ev["phase"][:m], ev["dur_ns"][:m], c, P,
                  score_key=keys, s=s, want_units=True, threads=th)
            dt = time.perf_counter() - tc
            res[th] = (m, dt)
        m, dt = res[threads]
        m1, dt1 = res[1]
        cpu = {"value": round(m / dt / 1e9, 6), "unit": "G events/s", "cores": threads, "kind": "oracle",
               "sample": "first %d events of the same workload, full path incl. score, group-by sharded over "
                         "%d threads (%.1f s)" % (m, threads, dt),
               "single_thread": {"value": round(m1 / dt1 / 1e9, 6), "cores": 1,
                                 "sample": "first %d events, one thread (%.1f s)" % (m1, dt1)},
               "nproc": os.cpu_count(), "cpu_model": cpu_model()}

    line = {
        "metric": "trace events aggregated/sec (G ev/s) + % of MI355X peak HBM BW",
        "value": round(value, 3),
        "unit": "G events/s",
        "n_gpus": 1,
        "steps": steps,
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
        "t_aggregate_ms": round(1e3 * statistics.median(t_agg), 4),
        "t_pipeline_ms_flushed": round(1e3 * statistics.median(t_flush), 4),
        "kernels_ms": {k: round(v["avg_ms"], 4) for k, v in kernels.items()},
        "parity": parity,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    ag.close()
    print(json.dumps(line), flush=True)
    if parity is not None and parity.get("checked") and not parity["ok"]:
        log("parity check FAILED:", parity["mismatch"])
        return 1
    return 0


if __name__ == "__main__":
    sys.exit(main())
