#!/usr/bin/env python3
"""Benchmark of the trace analyzer on one MI355X.

One step = one full analysis (every output: timelines, gaps, join and
latency histogram, containment with per-op aggregates, per-name
aggregates, cross-stream overlap) of the decode-step trace: 1 process,
4 streams, a 30 s window, 1,000 steps of 1,000 kernels (about 1M kernel
records, 1M launches, 1M CPU ops: 2.99M rows).  The input is resident in
HBM before timing.  Prints one JSON line: events (all input rows) per
second, the roofline of the dominant kernel measured live with HIP events
on the library's stream (the radix-sort passes), and the CPU oracle timed
on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
METRIC = "trace events analyzed/sec (M ev/s) at 1 MI355X + achieved HBM GB/s % peak"
HBM_PEAK_GBS = 8000.0
# Stage used for the roofline (the radix passes: the largest share of the
# device time) and the sources that define its kernels (the profiled traffic
# is only trusted while these files are unchanged).
ROOFLINE_STAGE = "sort"
ROOFLINE_KERNEL = "k_radix_pass"
STAGE_SOURCES = {"sort": ["paper_2609_40247_amd/csrc/radix.hip", "paper_2609_40247_amd/csrc/common.hpp",
                          "paper_2609_40247_amd/csrc/internal.hpp"]}
BYTES_PER_KEY_PASS = 24  # a digit pass reads and writes one 8-byte key and one 4-byte row index


def source_hash(stage: str) -> str:
    h = hashlib.sha256()
    for f in STAGE_SOURCES[stage]:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def sort_units(stats):
    """Key-passes the radix launches of the sort stage must make, and the
    number of those launches.  Pass p of a sort is its digit first + p, where
    first is 1 when the sort leaves its lowest digit to the refine pass (bit
    31 of its skipped-digit mask).  The stage makes as many passes as the
    timeline and containment sorts need; the join sort (which moves data only
    when the correlation table cannot be used) runs its passes in the same
    launches.  A sort moves its keys once per pass whose digit is not
    skipped."""
    def first(skipped):
        return 1 if (skipped >> 31) & 1 else 0
    passes = max(nd - first(skipped) for _, skipped, nd in (stats[0], stats[2]))
    units = 0
    for nkeys, skipped, nd in stats:
        f = first(skipped)
        units += nkeys * sum(1 for d in range(f, min(nd, f + passes)) if not (skipped >> d) & 1)
    return units, passes


def profiled_traffic(stage: str, workload: str):
    """HBM bytes per call of the stage from the committed rocprofv3 counter
    summary, if it was taken on the current sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{ROOFLINE_KERNEL}_{workload}.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    m_sha = re.search(r"kernel_source_sha256:\s*([0-9a-f]+)", txt)
    m_b = re.search(r"hbm_bytes_per_call:\s*([0-9]+)", txt)
    if not m_sha or not m_b or m_sha.group(1) != source_hash(stage):
        return None
    return int(m_b.group(1))


def cpu_baseline(cols, params, n, budget_s=12.0, max_calls=30):
    import oracle  # the CPU oracle: test infrastructure, used here only as the baseline
    oracle.analyze(cols, params)  # load / build outside the timing
    calls, t0 = 0, time.perf_counter()
    while calls < max_calls:
        oracle.analyze(cols, params)
        calls += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    dt = time.perf_counter() - t0
    return {"value": round(n * calls / dt / 1e6, 3), "unit": "M ev/s", "cores": 1, "kind": "oracle",
            "sample": f"the same 2.99M-row trace analyzed {calls} times by the single-threaded C oracle "
                      f"({dt:.1f} s on {os.cpu_count()} host cores, 1 used)"}


def _config4_trace(t):
    from paper_2609_40247_amd import synth
    tr = synth.config4_trace(t)
    return tr.columns(), tr.params


def run_config4(args) -> int:
    """One chunk of the 256-trace batch (traces 32c .. 32c+31, about 105M
    rows) through the batch entry point, device-resident; then the same chunk
    streamed from pinned host memory with double-buffered uploads."""
    import multiprocessing as mp
    import numpy as np
    first = 32 * args.chunk
    ids = list(range(first, first + 32))
    with mp.get_context("fork").Pool(min(16, os.cpu_count() or 1)) as pool:  # before the GPU is touched
        gen = pool.map(_config4_trace, ids)
    cols_l = [c for c, _ in gen]
    params_l = [p for _, p in gen]
    ns = [len(c["ts"]) for c in cols_l]
    n = int(sum(ns))
    offs = np.cumsum([0] + ns).astype(np.int64)
    keys = list(cols_l[0].keys())
    cols = {k: np.concatenate([c[k] for c in cols_l]) for k in keys}
    kernels = int(sum(int(np.count_nonzero(c["kind"] == 2)) for c in cols_l))

    import torch
    from paper_2609_40247_amd import herschel as H
    big = int(np.argmax(ns))
    ans = [H.Analyzer(p, ns[t], workspace=(t == big)) for t, p in enumerate(params_l)]
    p0 = ans[0]._params_struct(ans[big].ws.data_ptr(), ans[big].ws_bytes)
    plist = [p0] + [a.params for a in ans[1:]]
    outs = [a.outs for a in ans]
    dev = [H.device_columns(cols)]
    ev = H.events_struct(dev[0])
    torch.cuda.synchronize()

    def call(e):
        code = H.herschel_trace_analyze_batch(e, offs, plist, outs)
        if code != 0:
            raise RuntimeError(f"batch analysis failed: {H.herschel_strerror(code)}")

    for _ in range(args.warmup):
        call(ev)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        call(ev)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps

    # streamed: chunk i+1 uploads on a copy stream while chunk i is analyzed
    host = {k: torch.from_numpy(np.ascontiguousarray(v)).pin_memory() for k, v in cols.items()}
    dev.append({k: torch.empty_like(v) for k, v in dev[0].items()})
    evs = [H.events_struct(d) for d in dev]
    cs = torch.cuda.Stream()
    main = torch.cuda.current_stream()
    nbytes = sum(v.numel() * v.element_size() for v in host.values())
    done = [torch.cuda.Event() for _ in range(2)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    with torch.cuda.stream(cs):
        for k in host:
            dev[0][k].copy_(host[k], non_blocking=True)
    done[0].record(cs)
    torch.cuda.synchronize()
    h2d_s = time.perf_counter() - t0
    reps = max(args.steps, 2)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    with torch.cuda.stream(cs):
        for k in host:
            dev[0][k].copy_(host[k], non_blocking=True)
    done[0].record(cs)
    for i in range(reps):
        if i + 1 < reps:
            b = (i + 1) % 2
            with torch.cuda.stream(cs):
                for k in host:
                    dev[b][k].copy_(host[k], non_blocking=True)
            done[b].record(cs)
        main.wait_event(done[i % 2])
        call(evs[i % 2])
    torch.cuda.synchronize()
    stream_ms = (time.perf_counter() - t0) * 1e3 / reps

    out = {
        "metric": METRIC, "value": round(n / (ms * 1e-3) / 1e6, 3), "unit": "M ev/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int64", "data": "synthetic",
        "config": {"workload": f"batch chunk {args.chunk} of the 256-trace set: traces {first}-{first + 31} "
                               "(decode-step traces of 200k-2M kernels, windows of ceil(L/1000) x 30 ms), "
                               "names, busy/idle, gaps, latency histogram",
                   "rows": n, "kernels": kernels, "traces": 32,
                   "kernel_records_per_s_M": round(kernels / (ms * 1e-3) / 1e6, 3),
                   "est_ms_for_256_traces": round(ms * 8, 1)},
        "streamed": {"value": round(n / (stream_ms * 1e-3) / 1e6, 3), "unit": "M ev/s", "ms_per_chunk":
                     round(stream_ms, 3), "h2d_bytes_per_chunk": nbytes,
                     "h2d_GBps": round(nbytes / h2d_s / 1e9, 2)},
        "roofline": None,
    }
    if not args.no_cpu_baseline:
        import oracle
        oracle.analyze(cols_l[0], params_l[0])
        t0, done_rows, used = time.perf_counter(), 0, 0
        for c, p in zip(cols_l, params_l):
            oracle.analyze(c, p)
            done_rows += len(c["ts"])
            used += 1
            if time.perf_counter() - t0 >= 12.0:
                break
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": round(done_rows / dt / 1e6, 3), "unit": "M ev/s", "cores": 1,
                               "kind": "oracle", "sample": f"the first {used} traces of the chunk "
                               f"({done_rows} rows) analyzed once each by the single-threaded C oracle "
                               f"({dt:.1f} s)"}
    print(json.dumps(out), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--stages", action="store_true", help="also print a per-stage breakdown to stderr")
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="first copy a buffer of this many MiB on the device (a plain copy kernel of known "
                         "size, for scaling rocprofv3 byte counters)")
    ap.add_argument("--workload", choices=("config1", "config4"), default="config1",
                    help="config1: the decode-step trace (the headline line); config4: one 32-trace chunk of "
                         "the batch workload through the batch entry point")
    ap.add_argument("--chunk", type=int, default=0, help="config4: which of the 8 chunks")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              "run it with --gpus 1", file=sys.stderr)
        return 2
    if args.workload == "config4":
        return run_config4(args)

    import numpy as np
    import torch
    from paper_2609_40247_amd import herschel as H
    from paper_2609_40247_amd import synth

    if args.copy_mb > 0:
        src = torch.empty(args.copy_mb << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    tr = synth.config1()
    n = tr.n
    an = H.Analyzer(tr.params, n)
    dcols = H.device_columns(tr.columns())
    ev = H.events_struct(dcols)
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        code = an.run(ev, n)
        if code != 0:
            raise RuntimeError(f"analysis failed: {H.herschel_strerror(code)}")
    c = an.results(n)["counters"]
    units, launches = sort_units(H.herschel_sort_stats(an.params))

    # the timed region: K calls as a user makes them (repeated calls with the
    # same arguments replay the library's captured graph of the launches)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        code = an.run(ev, n)
        if code != 0:
            raise RuntimeError(f"analysis failed: {H.herschel_strerror(code)}")
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / args.steps

    # the roofline kernel: HIP events around the sort stage, recorded on the
    # stream its passes run on, over another K calls (launched directly, since
    # a call with stage events is not replayed from the graph)
    stage_id = H.STAGES.index(ROOFLINE_STAGE)
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    stream = torch.cuda.current_stream()
    for a, b in pairs:  # create the events
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    for a, b in pairs:
        H.herschel_time_stage(stage_id, a, b)
        code = an.run(ev, n)
        if code != 0:
            raise RuntimeError(f"analysis failed: {H.herschel_strerror(code)}")
    torch.cuda.synchronize()
    H.herschel_time_stage(stage_id, None, None)
    stage_ms = sum(a.elapsed_time(b) for a, b in pairs) / args.steps

    if args.stages:
        for sid, name in enumerate(H.STAGES):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            e1.record(stream)
            torch.cuda.synchronize()
            tot = 0.0
            for _ in range(5):
                H.herschel_time_stage(sid, e0, e1)
                an.run(ev, n)
                tot += e0.elapsed_time(e1)
            H.herschel_time_stage(sid, None, None)
            print(f"stage {name:14s} {tot / 5 * 1e3:9.1f} us", file=sys.stderr)

    # per launch of k_radix_pass: the stage's bytes and time over its launches
    alg = BYTES_PER_KEY_PASS * units / launches
    launch_s = stage_ms * 1e-3 / launches
    achieved = alg / launch_s / 1e9
    traffic = profiled_traffic(ROOFLINE_STAGE, "config1")
    traffic = None if traffic is None else round(traffic / launches)
    out = {
        "metric": METRIC, "value": round(n / (ms * 1e-3) / 1e6, 3), "unit": "M ev/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int64", "data": "synthetic",
        "config": {"workload": "decode-step trace: 1 process, 4 streams, 30 s window, 1000 steps x 1000 kernels",
                   "rows": n, "kernels": c["n_admitted_kernel"], "launches": c["n_admitted_launch"],
                   "cpu_ops": c["n_admitted_cpu"], "outputs": "all"},
        "roofline": {"kernel": ROOFLINE_KERNEL, "bound": "hbm", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "algorithmic_bytes": round(alg), "launch_us": round(launch_s * 1e6, 2),
                     "launches_per_step": launches, "key_passes_per_step": units},
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(tr.columns(), tr.params, n)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
