#!/usr/bin/env python3
"""Benchmark of the trace analyzer on one MI355X.

One step = one full analysis of one synthetic profiling window (every output:
timelines, gaps, join and latency histogram, containment with per-op
aggregates, per-name aggregates, cross-stream overlap, dependency waits).
The default workload is the decode-step trace: 1 process, 4 streams, a 30 s
window, 1,000 steps of 1,000 kernels (about 1M kernel records, 1M launches,
1M CPU ops: 2.99M rows).  ``--workload`` picks another: the tiny trace, the
mixed prefill/decode trace, the 8-process node trace, or one 32-trace chunk
of the 256-trace batch through the batch entry point.  The input is resident
in HBM before timing.

Prints one JSON line: events (all input rows) per second; the roofline of the
dominant kernel (the radix digit passes) measured live with HIP events on the
stream they run on; the whole call's algorithmic bytes over its wall time,
warm and with a cold cache, beside the HBM traffic the committed rocprofv3
counter profile measured over all analysis kernels; and the CPU oracle timed
on this host.
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
METRIC = "trace events analyzed/sec (M ev/s) at 1 MI355X + achieved HBM GB/s % peak"
HBM_PEAK_GBS = 8000.0
ROOFLINE_STAGE = "sort"
ROOFLINE_KERNEL = "k_radix_pass"
BYTES_PER_KEY_PASS = 24  # a digit pass reads and writes one 8-byte key and one 4-byte row index
CSRC = os.path.join(ROOT, "paper_2609_40247_amd", "csrc")

WORKLOADS = {
    "config0": "tiny trace: 1 process, 2 streams, 10 s window, 20k kernels, 20k launches, 20k CPU ops",
    "config1": "decode-step trace: 1 process, 4 streams, 30 s window, 1000 steps x 1000 kernels",
    "config2": "mixed prefill/decode trace: 1 process, 8 streams (compute, comm, copy), 30 s window, 5M rows",
    "config3": "node trace: 8 decode-step processes with clock offsets, 20k cross-process dependency edges",
}


def sources_hash() -> str:
    """Hash of every library source: a counter profile is trusted only while
    the kernels it measured are unchanged."""
    h = hashlib.sha256()
    for d, pat in ((CSRC, (".hip", ".hpp")), (os.path.join(ROOT, "include"), (".h",))):
        for f in sorted(os.listdir(d)):
            if f.endswith(pat):
                with open(os.path.join(d, f), "rb") as fh:
                    h.update(f.encode())
                    h.update(fh.read())
    return h.hexdigest()[:16]


def profile_fields(workload: str):
    """Per-call HBM traffic and summed kernel time of the analysis from the
    committed rocprofv3 summary of this workload, if taken on the current
    sources."""
    path = os.path.join(ROOT, "profiles", f"pipeline_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    txt = open(path).read()
    want = {"sources_sha256": r"sources_sha256:\s*([0-9a-f]+)", "hbm_bytes_per_call": r"hbm_bytes_per_call:\s*([0-9]+)",
            "kernel_us_per_call": r"kernel_us_per_call:\s*([0-9.]+)",
            "radix_hbm_bytes_per_launch": r"radix_hbm_bytes_per_launch:\s*([0-9]+)"}
    got = {}
    for k, pat in want.items():
        m = re.search(pat, txt)
        if not m:
            return None
        got[k] = m.group(1)
    if got["sources_sha256"] != sources_hash():
        return None
    return {"hbm_bytes_per_call": int(got["hbm_bytes_per_call"]), "kernel_us_per_call": float(got["kernel_us_per_call"]),
            "radix_hbm_bytes_per_launch": int(got["radix_hbm_bytes_per_launch"])}


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def algorithmic_bytes(n: int, counters: dict, params: dict, n_gaps: int) -> int:
    """Bytes the analysis must read and write once: every input column
    (37 B a row), the per-row links (8 B a row), the per-op aggregates
    (28 B an admitted op, with containment), and the per-stream, per-name,
    gap, overlap, histogram and edge outputs."""
    flags = int(params.get("flags", 3))
    P, S, NN = int(params["n_procs"]), int(params["n_streams"]), int(params["n_names"])
    edges = params.get("edges")
    E = 0 if edges is None else len(edges)
    b = 37 * n + 8 * n
    if flags & 1:
        b += 28 * counters["n_admitted_cpu"]
    b += 16 * P * S + 32 * NN + 32 * int(params["n_op_names"]) + 64 * 8 + 25 * n_gaps + 8 * P + S + 112
    if flags & 2:
        b += 8 * (P * S * S + 12 * P)
    b += 36 * E  # each edge read (24 B) and its wait and status written
    if flags & 4:
        b += 8 * P + 16 * P * int(params["n_op_names"])  # GPU idle, op-name span and idle
    if flags & 8:  # each admitted op's counts read, its MFU, MBU and SOL written; per op name 5 sums and a reference
        b += 40 * counters["n_admitted_cpu"] + 48 * int(params["n_op_names"])
    if flags & 16:  # each admitted row's time charged and path flags written; per process 8 parts
        b += 9 * sum(counters[k] for k in ("n_admitted_cpu", "n_admitted_launch", "n_admitted_kernel")) + 64 * P
    return b


def sort_units(stats):
    """Key-passes the radix launches of the sort stage must make, and the
    number of those launches.  Pass p of a sort is its digit first + p, where
    first is 1 when the sort leaves its lowest digit to the refine pass (bit
    31 of its skipped-digit mask); a sort moves its keys once per pass whose
    digit is not skipped."""
    def first(skipped):
        return 1 if (skipped >> 31) & 1 else 0
    sorts = [s for s in (stats[0], stats[2]) if s[2] > 0]
    passes = max(nd - first(skipped) for _, skipped, nd in sorts)
    units = 0
    for nkeys, skipped, nd in sorts:
        f = first(skipped)
        units += nkeys * sum(1 for d in range(f, min(nd, f + passes)) if not (skipped >> d) & 1)
    return units, passes


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
            "cpu_model": cpu_model(), "host_cores": os.cpu_count(),
            "sample": f"the same {n}-row trace analyzed {calls} times by the single-threaded C oracle "
                      f"({dt:.1f} s, 1 of {os.cpu_count()} host cores used)"}


def make_trace(workload: str):
    from paper_2609_40247_amd import synth
    return {"config0": synth.config0, "config1": synth.config1, "config2": synth.config2,
            "config3": synth.config3}[workload]()


BATCH_OUTPUTS = ("name_count", "name_sum", "name_min", "name_max", "opname_count", "opname_sum", "opname_min",
                 "opname_max", "busy", "idle", "gap_pid", "gap_stream",
                 "gap_begin", "gap_end", "gap_flags", "lat_hist", "counters")


def run_config4(args) -> int:
    """One chunk of the 256-trace batch (traces 32c .. 32c+31, about 105M
    rows) through the batch entry point with the batch output set (per-name
    aggregates, busy / idle, gaps, latency histogram; the other outputs NULL),
    device-resident; then the same chunk streamed from pinned host memory
    through the chunked entry point (double-buffered uploads)."""
    import numpy as np
    from paper_2609_40247_amd import synth
    first = 32 * args.chunk
    ids = list(range(first, first + 32))
    def progress(done, total):
        print(f"generated {done}/{total} traces", file=sys.stderr, flush=True)

    gen = synth.config4_chunk(ids, progress=progress)  # spawned workers, before the GPU is touched
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
    outs = [H.HerschelOutputs(gap_capacity=a.gap_capacity,
                              **{k: (v.data_ptr() if k in BATCH_OUTPUTS else None) for k, v in a.o.items()})
            for a in ans]
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
    gaps, alg = 0, 0
    for t, a in enumerate(ans):
        c = {k: int(v) for k, v in zip(H.COUNTERS, a.o["counters"].cpu().tolist())}
        g = min(c["n_gaps_total"], a.gap_capacity)
        p = params_l[t]
        gaps += g
        # the batch set: every input column once, then busy / idle, the names,
        # the gap list, the histogram and the counters
        alg += 37 * ns[t] + 16 * p["n_procs"] * p["n_streams"] + 32 * p["n_names"] + 25 * g + 512 + 112

    # streamed: the same 32 traces from pinned host memory through the
    # library's chunked entry point, in chunks of 8 traces (two staging sets;
    # chunk c + 1 uploads on the library's copy stream while chunk c is analysed)
    host = {k: torch.from_numpy(np.ascontiguousarray(v)).pin_memory() for k, v in cols.items()}
    hev = H.HerschelEvents(**{k: v.data_ptr() for k, v in host.items()})
    per = 8
    srows = max(int(offs[min(c + per, 32)] - offs[c]) for c in range(0, 32, per))
    del dev, ev
    staging = [{k: torch.empty(srows, dtype=v.dtype, device="cuda") for k, v in host.items()} for _ in range(2)]
    sev = [H.events_struct(d) for d in staging]
    nbytes = sum(v.numel() * v.element_size() for v in host.values())
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in host:  # one chunk's upload alone, for the PCIe rate
        staging[0][k][:int(offs[per])].copy_(host[k][:int(offs[per])], non_blocking=True)
    torch.cuda.synchronize()
    h2d_s = (time.perf_counter() - t0) * nbytes / sum(v[:int(offs[per])].numel() * v.element_size()
                                                       for v in host.values())

    def call_chunked():
        code = H.herschel_trace_analyze_chunked(hev, offs, per, sev, srows, plist, outs)
        if code != 0:
            raise RuntimeError(f"chunked analysis failed: {H.herschel_strerror(code)}")

    call_chunked()
    reps = max(args.steps, 2)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        call_chunked()
    torch.cuda.synchronize()
    stream_ms = (time.perf_counter() - t0) * 1e3 / reps

    out = {
        "metric": METRIC, "value": round(n / (ms * 1e-3) / 1e6, 3), "unit": "M ev/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int64", "data": "synthetic",
        "config": {"workload": f"batch chunk {args.chunk} of the 256-trace set: traces {first}-{first + 31} "
                               "(decode-step traces of 200k-2M kernels, windows of ceil(L/1000) x 30 ms), "
                               "outputs: per-name aggregates, busy/idle, gaps, latency histogram",
                   "rows": n, "kernels": kernels, "traces": 32, "gaps": int(gaps),
                   "kernel_records_per_s_M": round(kernels / (ms * 1e-3) / 1e6, 3),
                   "est_ms_for_256_traces": round(ms * 8, 1)},
        "whole_call": {"algorithmic_bytes": alg, "algorithmic_GBps": round(alg / (ms * 1e-3) / 1e9, 1),
                       "frac": round(alg / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
        "streamed": {"value": round(n / (stream_ms * 1e-3) / 1e6, 3), "unit": "M ev/s", "ms_per_chunk":
                     round(stream_ms, 3), "traces_per_upload": per, "h2d_bytes_per_chunk": nbytes,
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
                               "kind": "oracle", "cpu_model": cpu_model(), "host_cores": os.cpu_count(),
                               "sample": f"the first {used} traces of the chunk ({done_rows} rows) analyzed once "
                                         f"each by the single-threaded C oracle ({dt:.1f} s)"}
    print(json.dumps(out), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-cold", action="store_true", help="skip the cold-cache timing")
    ap.add_argument("--stages", action="store_true", help="also print a per-stage breakdown to stderr")
    ap.add_argument("--copy-mb", type=int, default=0,
                    help="first copy a buffer of this many MiB on the device (a plain copy kernel of known "
                         "size, for scaling rocprofv3 byte counters)")
    ap.add_argument("--workload", choices=tuple(WORKLOADS) + ("config4",), default="config1",
                    help="config1: the decode-step trace (the headline line); config0, config2, config3: the "
                         "other single-window workloads; config4: one 32-trace chunk of the batch workload")
    ap.add_argument("--chunk", type=int, default=0, help="config4: which of the 8 chunks")
    ap.add_argument("--waits", action="store_true",
                    help="also compute the GPU idle coinciding with CPU ops, by op name")
    ap.add_argument("--crit", action="store_true", help="also compute the critical path")
    ap.add_argument("--sol", action="store_true",
                    help="also compute operator efficiency (MFU, MBU, SOL per op; per op name sums and hotness) "
                         "from synthetic per-op counts")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              "run it with --gpus 1", file=sys.stderr)
        return 2
    if args.workload == "config4":
        return run_config4(args)

    tr = make_trace(args.workload)  # generated before the GPU is touched
    import torch
    from paper_2609_40247_amd import herschel as H

    if args.copy_mb > 0:
        src = torch.empty(args.copy_mb << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    n = tr.n
    cols, params = tr.columns(), dict(tr.params)
    if args.waits:
        params["flags"] = int(params.get("flags", 3)) | H.OUT_WAITS
    if args.sol:
        from paper_2609_40247_amd import synth
        cols, params = synth.add_op_costs(cols, params, 7)
    if args.crit:
        params["flags"] = int(params.get("flags", 3)) | H.OUT_CRIT | H.OUT_CONTAIN
    an = H.Analyzer(params, n)
    dcols = H.device_columns(cols)
    ev = H.events_struct(dcols)
    torch.cuda.synchronize()

    def run():
        code = an.run(ev, n)
        if code != 0:
            raise RuntimeError(f"analysis failed: {H.herschel_strerror(code)}")

    for _ in range(args.warmup):
        run()
    res = an.results(n)
    c = res["counters"]
    units, launches = sort_units(H.herschel_sort_stats(an.params))

    # the timed region: K calls as a user makes them (each launches its
    # kernels directly: graph replay is the library's opt-in)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        run()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps

    # cold cache: before each call a 1 GiB fill evicts the caches (the 256 MB
    # last-level cache included); each call is timed on its own, and so are
    # warm calls the same way for comparison
    cold = None
    if not args.no_cold:
        flush = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        cold_ms, warm_ms = [], []
        for i in range(min(args.steps, 20)):
            flush.fill_(i & 0xFF)
            torch.cuda.synchronize()
            t = time.perf_counter()
            run()
            cold_ms.append((time.perf_counter() - t) * 1e3)
            t = time.perf_counter()
            run()
            warm_ms.append((time.perf_counter() - t) * 1e3)
        del flush
        cold = (statistics.median(cold_ms), statistics.median(warm_ms))

    # the roofline kernel: HIP events around the sort stage, recorded on the
    # stream its passes run on, over another K calls
    stage_id = H.STAGES.index(ROOFLINE_STAGE)
    pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    stream = torch.cuda.current_stream()
    for a, b in pairs:  # create the events
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    for a, b in pairs:
        H.herschel_time_stage(stage_id, a, b)
        run()
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
                torch.cuda.synchronize()  # the call returns before HIP marks its events complete
                tot += e0.elapsed_time(e1)
            H.herschel_time_stage(sid, None, None)
            print(f"stage {name:14s} {tot / 5 * 1e3:9.1f} us", file=sys.stderr)

    # per launch of k_radix_pass: the stage's bytes and time over its launches
    alg = BYTES_PER_KEY_PASS * units / launches
    launch_s = stage_ms * 1e-3 / launches
    achieved = alg / launch_s / 1e9
    prof = profile_fields(args.workload + ("_waits" if args.waits else "") + ("_sol" if args.sol else "") +
                          ("_crit" if args.crit else ""))
    gaps = min(c["n_gaps_total"], an.gap_capacity)
    call_bytes = algorithmic_bytes(n, c, params, gaps)
    whole = {"algorithmic_bytes": call_bytes, "algorithmic_GBps": round(call_bytes / (ms * 1e-3) / 1e9, 1),
             "frac": round(call_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
             "traffic_bytes": None, "kernel_us": None, "traffic_GBps": None, "traffic_frac": None}
    if cold is not None:
        whole.update({"cold_ms_per_call": round(cold[0], 4), "warm_ms_per_call_same_timing": round(cold[1], 4),
                      "cold_algorithmic_GBps": round(call_bytes / (cold[0] * 1e-3) / 1e9, 1)})
    if prof is not None:
        tb, ku = prof["hbm_bytes_per_call"], prof["kernel_us_per_call"]
        whole.update({"traffic_bytes": tb, "kernel_us": ku, "traffic_GBps": round(tb / (ku * 1e-6) / 1e9, 1),
                      "traffic_frac": round(tb / (ku * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)})
    out = {
        "metric": METRIC, "value": round(n / (ms * 1e-3) / 1e6, 3), "unit": "M ev/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int64", "data": "synthetic",
        "config": {"workload": WORKLOADS[args.workload], "rows": n, "kernels": c["n_admitted_kernel"],
                   "launches": c["n_admitted_launch"], "cpu_ops": c["n_admitted_cpu"],
                   "outputs": "all" + (", with the idle coincidence by op name" if args.waits else "") +
                              (", with operator efficiency" if args.sol else "") +
                              (", with the critical path" if args.crit else "")},
        "roofline": {"kernel": ROOFLINE_KERNEL, "bound": "hbm", "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": None if prof is None else prof["radix_hbm_bytes_per_launch"],
                     "algorithmic_bytes": round(alg), "launch_us": round(launch_s * 1e6, 2),
                     "launches_per_step": launches, "key_passes_per_step": units},
        "whole_call": whole,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(cols, params, n)
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
