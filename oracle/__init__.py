"""TEST INFRASTRUCTURE ONLY: ctypes wrapper of the CPU oracle.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product library never calls it.
The oracle (``herschel_oracle.c``) is a plain single-threaded C program that
computes the trace reconstruction of the Herschel analyzer (Section 6.1) from
its definitions; these bindings are written separately from the product's.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "herschel_oracle.c")
_SO = os.path.join(_HERE, "libherschel_oracle.so")

# Values the oracle leaves in rows it does not write (tests compare whole arrays).
UNWRITTEN_I32 = -3
UNWRITTEN_I64 = -3
UNWRITTEN_U8 = 0xFD


def build() -> str:
    """Compile the oracle with the host C compiler (no GPU code)."""
    cmd = ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC", "-o", _SO + ".tmp", _SRC]
    subprocess.run(cmd, check=True, cwd=_HERE)
    os.replace(_SO + ".tmp", _SO)
    return _SO


_lib = None


def load_library(path: str):
    """Open an oracle shared library (the default one, or a test variant)."""
    lib = ctypes.CDLL(path)
    lib.herschel_oracle_analyze.restype = ctypes.c_int
    lib.herschel_oracle_analyze.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO) or os.path.getmtime(_SO) < os.path.getmtime(_SRC):
            build()
        _lib = load_library(_SO)
    return _lib


_P = ctypes.c_void_p


class _Events(ctypes.Structure):
    _fields_ = [(k, _P) for k in ("ts", "te", "corr", "pid", "lane", "name", "kind", "flops", "bytes",
                                  "graph_node")]


class _Params(ctypes.Structure):
    _fields_ = [("w0", ctypes.c_int64), ("w1", ctypes.c_int64), ("thr", ctypes.c_int64),
                ("n_procs", ctypes.c_int32), ("n_streams", ctypes.c_int32),
                ("n_threads", ctypes.c_int32), ("n_names", ctypes.c_int32),
                ("n_op_names", ctypes.c_int32), ("clock_offset", _P), ("stream_class", _P),
                ("edges", _P), ("n_edges", ctypes.c_int64), ("flags", ctypes.c_uint32),
                ("peak_flops", ctypes.c_int64), ("peak_bytes", ctypes.c_int64), ("ref_sol_ppm", _P),
                ("n_graph_nodes", ctypes.c_int32)]


COUNTER_NAMES = ("n_admitted_cpu", "n_admitted_launch", "n_admitted_kernel", "n_outside_window",
                 "n_matched", "n_unmatched_kernels", "n_unmatched_launches", "n_dup_launch_corr",
                 "n_unattributed_kernels", "n_improper_nesting", "n_negative_latency",
                 "n_gaps_total", "first_invalid", "device_status")


class _Outputs(ctypes.Structure):
    _fields_ = [("link", _P), ("aux", _P), ("op_nkern", _P), ("op_first", _P), ("op_last", _P),
                ("op_ksum", _P), ("busy", _P), ("idle", _P), ("pair_overlap", _P),
                ("class_busy", _P), ("class_overlap", _P), ("any_busy", _P), ("name_count", _P),
                ("name_sum", _P), ("name_min", _P), ("name_max", _P), ("lat_hist", _P),
                ("edge_wait", _P), ("edge_status", _P), ("gap_capacity", ctypes.c_int64),
                ("gap_pid", _P), ("gap_stream", _P), ("gap_begin", _P), ("gap_end", _P),
                ("gap_flags", _P), ("counters", _P), ("dev_idle", _P), ("op_span", _P), ("op_idle", _P),
                ("op_mfu", _P), ("op_mbu", _P), ("op_sol", _P), ("opn_flops", _P), ("opn_bytes", _P),
                ("opn_time", _P), ("opn_sol", _P), ("opn_hot", _P), ("crit_time", _P), ("crit_flags", _P),
                ("crit_proc", _P), ("launch_first", _P), ("launch_last", _P), ("gn_count", _P), ("gn_sum", _P),
                ("gn_min", _P), ("gn_max", _P), ("gn_offset", _P), ("opname_count", _P), ("opname_sum", _P),
                ("opname_min", _P), ("opname_max", _P)]


def _ptr(a):
    return None if a is None else a.ctypes.data


def analyze(cols: dict, params: dict, gap_capacity: int | None = None, lib=None):
    """Run the oracle on host arrays.

    ``cols`` holds ts, te, corr (int64), pid, lane, name (int32), kind (uint8);
    ``params`` the window, threshold, sizes, optional clock_offset,
    stream_class and edges (structured array with prod_pid, cons_pid,
    prod_corr, cons_corr) and flags.  Returns (code, outputs dict)."""
    lib = lib or _load()
    c = {k: np.ascontiguousarray(cols[k], dtype=dt) for k, dt in
         (("ts", np.int64), ("te", np.int64), ("corr", np.int64), ("pid", np.int32),
          ("lane", np.int32), ("name", np.int32), ("kind", np.uint8))}
    n = int(c["ts"].shape[0])
    for k in ("flops", "bytes"):  # per-op operation counts and logical bytes (SOL outputs)
        if cols.get(k) is not None:
            c[k] = np.ascontiguousarray(cols[k], dtype=np.int64)
    if cols.get("graph_node") is not None:  # per-kernel graph nodes (graph replay outputs)
        c["graph_node"] = np.ascontiguousarray(cols["graph_node"], dtype=np.int32)
    P, S = int(params["n_procs"]), int(params["n_streams"])
    edges = params.get("edges")
    n_edges = 0 if edges is None else int(len(edges))
    off = params.get("clock_offset")
    off = None if off is None else np.ascontiguousarray(off, dtype=np.int64)
    cls = params.get("stream_class")
    cls = None if cls is None else np.ascontiguousarray(cls, dtype=np.uint8)
    ref = params.get("ref_sol_ppm")
    ref = None if ref is None else np.ascontiguousarray(ref, dtype=np.int64)
    edges = None if n_edges == 0 else np.ascontiguousarray(edges)
    if gap_capacity is None:
        gap_capacity = int(np.count_nonzero(c["kind"] == 2)) + P * S
    o = dict(
        link=np.full(n, UNWRITTEN_I32, np.int32), aux=np.full(n, UNWRITTEN_I32, np.int32),
        op_nkern=np.full(n, UNWRITTEN_I32, np.int32), op_first=np.full(n, UNWRITTEN_I64, np.int64),
        op_last=np.full(n, UNWRITTEN_I64, np.int64), op_ksum=np.full(n, UNWRITTEN_I64, np.int64),
        busy=np.zeros(P * S, np.int64), idle=np.zeros(P * S, np.int64),
        pair_overlap=np.zeros(P * S * S, np.int64), class_busy=np.zeros(P * 3, np.int64),
        class_overlap=np.zeros(P * 9, np.int64), any_busy=np.zeros(P, np.int64),
        name_count=np.zeros(params["n_names"], np.int64), name_sum=np.zeros(params["n_names"], np.int64),
        name_min=np.zeros(params["n_names"], np.int64), name_max=np.zeros(params["n_names"], np.int64),
        lat_hist=np.zeros(64, np.int64), edge_wait=np.zeros(n_edges, np.int64),
        edge_status=np.zeros(n_edges, np.int32),
        gap_pid=np.zeros(max(gap_capacity, 1), np.int32), gap_stream=np.zeros(max(gap_capacity, 1), np.int32),
        gap_begin=np.zeros(max(gap_capacity, 1), np.int64), gap_end=np.zeros(max(gap_capacity, 1), np.int64),
        gap_flags=np.zeros(max(gap_capacity, 1), np.uint8),
        dev_idle=np.zeros(P, np.int64), op_span=np.zeros(P * int(params["n_op_names"]), np.int64),
        op_idle=np.zeros(P * int(params["n_op_names"]), np.int64),
        op_mfu=np.full(n, UNWRITTEN_I64, np.int64), op_mbu=np.full(n, UNWRITTEN_I64, np.int64),
        op_sol=np.full(n, UNWRITTEN_I64, np.int64),
        **{k: np.zeros(int(params["n_op_names"]), np.int64)
           for k in ("opn_flops", "opn_bytes", "opn_time", "opn_sol", "opn_hot")},
        crit_time=np.full(n, UNWRITTEN_I64, np.int64), crit_flags=np.full(n, UNWRITTEN_U8, np.uint8),
        crit_proc=np.zeros(P * 8, np.int64),
        launch_first=np.full(n, UNWRITTEN_I64, np.int64), launch_last=np.full(n, UNWRITTEN_I64, np.int64),
        **{k: np.zeros(max(int(params.get("n_graph_nodes", 1)), 1), np.int64)
           for k in ("gn_count", "gn_sum", "gn_min", "gn_max", "gn_offset")},
        **{k: np.zeros(int(params["n_op_names"]), np.int64)
           for k in ("opname_count", "opname_sum", "opname_min", "opname_max")},
    )
    counters = np.zeros(len(COUNTER_NAMES), np.int64)
    ev = _Events(**{k: _ptr(v) for k, v in c.items()})
    pr = _Params(w0=int(params["window_begin"]), w1=int(params["window_end"]),
                 thr=int(params["gap_threshold"]), n_procs=P, n_streams=S,
                 n_threads=int(params["n_threads"]), n_names=int(params["n_names"]),
                 n_op_names=int(params["n_op_names"]), clock_offset=_ptr(off), stream_class=_ptr(cls),
                 edges=_ptr(edges), n_edges=n_edges, flags=int(params.get("flags", 3)),
                 peak_flops=int(params.get("peak_flops", 0)), peak_bytes=int(params.get("peak_bytes", 0)),
                 ref_sol_ppm=_ptr(ref), n_graph_nodes=int(params.get("n_graph_nodes", 0)))
    out = _Outputs(gap_capacity=gap_capacity, counters=counters.ctypes.data,
                   **{k: v.ctypes.data for k, v in o.items()})
    code = lib.herschel_oracle_analyze(ctypes.byref(ev), n, ctypes.byref(pr), ctypes.byref(out))
    o["counters"] = dict(zip(COUNTER_NAMES, (int(x) for x in counters)))
    ng = min(o["counters"]["n_gaps_total"], gap_capacity)
    for k in ("gap_pid", "gap_stream", "gap_begin", "gap_end", "gap_flags"):
        o[k] = o[k][:ng]
    return code, o
