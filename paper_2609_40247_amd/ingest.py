"""Real traces into the analyzer's input columns.

The profiler of the paper reads vendor tracing libraries through adapters
(Section 5.2, "Heterogeneous Devices Beyond NVIDIA": the AMD backend uses the
ROCm tracer).  This module is such an adapter for the CSV output of ROCm's
`rocprofv3` (`--kernel-trace --hip-runtime-trace --marker-trace
--output-format csv`):

* every kernel dispatch becomes a KERNEL record, located by its process and
  stream, named by its kernel name, carrying its correlation id;
* every HIP runtime call becomes a LAUNCH record (a host API interval with
  its correlation id), named by its function;
* every ROCTX range becomes a CPU_OP record (a named host range of its
  thread), named by its message.

Process, stream and thread ids are mapped to dense indices per process;
names are interned into three tables.  A kernel whose call is
`hipGraphLaunch` belongs to a graph replay, and its graph node is its rank by
start time among the replay's kernels (the replayed layer sequence); other
kernels get node -1.  The window covers every record.  Timestamps are the
profiler's nanoseconds on one host clock, so no clock offsets are needed.
"""
from __future__ import annotations

import csv
import dataclasses
import glob
import os

import numpy as np

CPU_OP, LAUNCH, KERNEL = 0, 1, 2
GRAPH_LAUNCH_CALLS = ("hipGraphLaunch",)
# a dependency edge record (the layout of herschel_edge); a trace has none
EDGE_DTYPE = np.dtype([("prod_pid", "<i4"), ("cons_pid", "<i4"), ("prod_corr", "<i8"), ("cons_corr", "<i8")],
                      align=True)


@dataclasses.dataclass
class Ingested:
    columns: dict          # ts, te, corr, pid, lane, name, kind, graph_node
    params: dict           # window, sizes, flags, n_graph_nodes
    kernel_names: list
    api_names: list
    op_names: list
    process_ids: list      # the trace's process ids, by dense index
    streams: dict          # (process id, stream id) -> dense stream index
    threads: dict          # (process id, thread id) -> dense thread index


def _find(path: str, suffix: str):
    if os.path.isdir(path):
        hits = sorted(glob.glob(os.path.join(path, "**", f"*{suffix}"), recursive=True))
    else:
        hits = [path + suffix] if os.path.exists(path + suffix) else []
    return hits[0] if hits else None


def _rows(path):
    if path is None:
        return []
    with open(path, newline="") as fh:
        return list(csv.DictReader(fh))


class _Interner:
    def __init__(self):
        self.ids = {}
        self.names = []

    def __call__(self, name: str) -> int:
        i = self.ids.get(name)
        if i is None:
            i = self.ids[name] = len(self.names)
            self.names.append(name)
        return i


def read_rocprofv3(path: str, flags: int = 1 | 2, gap_threshold: int = 0) -> Ingested:
    """Reads `<prefix>_kernel_trace.csv`, `<prefix>_hip_api_trace.csv` and
    `<prefix>_marker_api_trace.csv` (path is the prefix or a directory that
    holds them) into input columns and parameters for one window."""
    kern = _rows(_find(path, "_kernel_trace.csv"))
    api = _rows(_find(path, "_hip_api_trace.csv"))
    mark = _rows(_find(path, "_marker_api_trace.csv"))
    if not kern and not api and not mark:
        raise FileNotFoundError(f"no rocprofv3 CSV traces at {path}")

    # processes: the host records name them; a kernel takes the process of
    # its call (same correlation id), else the only process there is
    call_of = {int(a["Correlation_Id"]): a for a in api}
    pids = sorted({int(r["Process_Id"]) for r in api + mark})
    if not pids:
        pids = [0]
    pidx = {p: i for i, p in enumerate(pids)}

    def kernel_pid(k):
        a = call_of.get(int(k["Correlation_Id"]))
        if a is not None:
            return int(a["Process_Id"])
        if len(pids) == 1:
            return pids[0]
        raise ValueError(f"kernel with correlation id {k['Correlation_Id']} has no call to name its process")

    streams, threads = {}, {}
    per_proc_streams, per_proc_threads = {}, {}

    def stream_of(p, s):
        key = (p, s)
        if key not in streams:
            streams[key] = per_proc_streams.get(p, 0)
            per_proc_streams[p] = streams[key] + 1
        return streams[key]

    def thread_of(p, t):
        key = (p, t)
        if key not in threads:
            threads[key] = per_proc_threads.get(p, 0)
            per_proc_threads[p] = threads[key] + 1
        return threads[key]

    kn, an, on = _Interner(), _Interner(), _Interner()
    recs = []  # kind, pid index, lane, ts, te, corr, name, node
    # graph replays: the kernels of each hipGraphLaunch call, by start time
    replay = {}
    for k in kern:
        c = int(k["Correlation_Id"])
        a = call_of.get(c)
        if a is not None and a["Function"] in GRAPH_LAUNCH_CALLS:
            replay.setdefault(c, []).append(k)
    node_of = {}
    for c, ks in replay.items():
        for rank, k in enumerate(sorted(ks, key=lambda k: (int(k["Start_Timestamp"]), int(k["Dispatch_Id"])))):
            node_of[(c, int(k["Dispatch_Id"]))] = rank
    for k in kern:
        p = kernel_pid(k)
        sid = k.get("Stream_Id", k.get("Queue_Id", "0"))
        c = int(k["Correlation_Id"])
        recs.append((KERNEL, pidx[p], stream_of(p, int(sid)), int(k["Start_Timestamp"]), int(k["End_Timestamp"]), c,
                     kn(k["Kernel_Name"]), node_of.get((c, int(k["Dispatch_Id"])), -1)))
    for a in api:
        p = int(a["Process_Id"])
        recs.append((LAUNCH, pidx[p], thread_of(p, int(a["Thread_Id"])), int(a["Start_Timestamp"]),
                     int(a["End_Timestamp"]), int(a["Correlation_Id"]), an(a["Function"]), -1))
    for m in mark:
        p = int(m["Process_Id"])
        recs.append((CPU_OP, pidx[p], thread_of(p, int(m["Thread_Id"])), int(m["Start_Timestamp"]),
                     int(m["End_Timestamp"]), 0, on(m["Function"]), -1))
    a = np.array(recs, dtype=np.int64).reshape(-1, 8)
    cols = dict(kind=a[:, 0].astype(np.uint8), pid=a[:, 1].astype(np.int32), lane=a[:, 2].astype(np.int32),
                ts=a[:, 3].copy(), te=a[:, 4].copy(), corr=a[:, 5].copy(), name=a[:, 6].astype(np.int32),
                graph_node=a[:, 7].astype(np.int32))
    w0 = int(cols["ts"].min()) if len(a) else 0
    w1 = int(max(cols["te"].max(), cols["ts"].max())) + 1 if len(a) else 1
    n_graph = max((len(ks) for ks in replay.values()), default=0)
    params = dict(window_begin=w0, window_end=w1, gap_threshold=int(gap_threshold), n_procs=len(pids),
                  n_streams=max(max(per_proc_streams.values(), default=1), 1),
                  n_threads=max(max(per_proc_threads.values(), default=1), 1),
                  n_names=max(len(kn.names), 1), n_op_names=max(len(on.names), 1), clock_offset=None,
                  stream_class=None, edges=np.zeros(0, EDGE_DTYPE),
                  flags=int(flags) | (32 if n_graph and flags & 1 else 0), n_graph_nodes=max(n_graph, 1))
    return Ingested(columns=cols, params=params, kernel_names=kn.names, api_names=an.names, op_names=on.names,
                    process_ids=pids, streams=streams, threads=threads)
