"""ctypes binding of libherschel (argument marshalling only).

The names follow the C ABI in ``include/herschel.h``:
``herschel_workspace_size``, ``herschel_trace_analyze``,
``herschel_trace_analyze_batch``, ``herschel_trace_analyze_chunked`` and
``herschel_strerror``.  Every step of the
analysis runs in the HIP library; PyTorch only provides device memory and the
stream.  There is no CPU fallback: without the built library (or a GPU) the
calls raise.

``Analyzer`` keeps the workspace and output tensors of one problem size so
that repeated calls allocate nothing.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIBS = {"release": "libherschel.so", "checked": "libherschel_checked.so"}

CPU_OP, LAUNCH, KERNEL = 0, 1, 2
OK, EINVAL, EEVENT, ECAPACITY, EWORKSPACE, EDEVICE, ETOOBIG = 0, -1, -2, -3, -4, -5, -6
STATIC_SCRATCH_BYTES = 64 << 20  # HERSCHEL_STATIC_SCRATCH_BYTES
OUT_CONTAIN, OUT_OVERLAP, OUT_WAITS, OUT_SOL, OUT_CRIT, OUT_GRAPH = 0x1, 0x2, 0x4, 0x8, 0x10, 0x20
REPLAY = 0x100  # not an output: repeated equal calls replay a captured HIP graph

_P = ctypes.c_void_p


class HerschelEvents(ctypes.Structure):
    _fields_ = [(k, _P) for k in ("ts", "te", "corr", "pid", "lane", "name", "kind", "flops", "bytes",
                                  "graph_node")]


class HerschelParams(ctypes.Structure):
    _fields_ = [("window_begin", ctypes.c_int64), ("window_end", ctypes.c_int64),
                ("gap_threshold", ctypes.c_int64), ("n_procs", ctypes.c_int32),
                ("n_streams", ctypes.c_int32), ("n_threads", ctypes.c_int32),
                ("n_names", ctypes.c_int32), ("n_op_names", ctypes.c_int32),
                ("clock_offset", _P), ("stream_class", _P), ("edges", _P),
                ("n_edges", ctypes.c_int64), ("flags", ctypes.c_uint32), ("hip_stream", _P),
                ("workspace", _P), ("workspace_bytes", ctypes.c_size_t),
                ("peak_flops", ctypes.c_int64), ("peak_bytes", ctypes.c_int64), ("ref_sol_ppm", _P),
                ("n_graph_nodes", ctypes.c_int32)]


COUNTERS = ("n_admitted_cpu", "n_admitted_launch", "n_admitted_kernel", "n_outside_window", "n_matched",
            "n_unmatched_kernels", "n_unmatched_launches", "n_dup_launch_corr", "n_unattributed_kernels",
            "n_improper_nesting", "n_negative_latency", "n_gaps_total", "first_invalid", "device_status")


class HerschelOutputs(ctypes.Structure):
    _fields_ = [(k, _P) for k in ("link", "aux", "op_nkern", "op_first", "op_last", "op_ksum", "busy", "idle",
                                  "pair_overlap", "class_busy", "class_overlap", "any_busy", "name_count",
                                  "name_sum", "name_min", "name_max", "lat_hist", "edge_wait", "edge_status")] + [
        ("gap_capacity", ctypes.c_int64)] + [(k, _P) for k in ("gap_pid", "gap_stream", "gap_begin", "gap_end",
                                                               "gap_flags", "counters", "dev_idle", "op_span",
                                                               "op_idle", "op_mfu", "op_mbu", "op_sol",
                                                               "opn_flops", "opn_bytes", "opn_time", "opn_sol",
                                                               "opn_hot", "crit_time", "crit_flags", "crit_proc",
                                                               "launch_first", "launch_last", "gn_count", "gn_sum",
                                                               "gn_min", "gn_max", "gn_offset", "opname_count",
                                                               "opname_sum", "opname_min", "opname_max")]
OPNAME_OUTPUTS = ("opname_count", "opname_sum", "opname_min", "opname_max")
GRAPH_NODE_OUTPUTS = ("gn_count", "gn_sum", "gn_min", "gn_max", "gn_offset")
SOL_ROW_OUTPUTS = ("op_mfu", "op_mbu", "op_sol")
SOL_NAME_OUTPUTS = ("opn_flops", "opn_bytes", "opn_time", "opn_sol", "opn_hot")


_lib = {}


def library_path(variant: str | None = None) -> str:
    """``variant`` (or $HERSCHEL_LIB): "release", "checked", or a path to a
    library built elsewhere."""
    variant = variant or os.environ.get("HERSCHEL_LIB", "release")
    if variant.endswith(".so"):
        return os.path.abspath(variant)
    return os.path.join(_HERE, _LIBS[variant])


def load(variant: str | None = None) -> ctypes.CDLL:
    """Open the HIP library; raises if it has not been built."""
    path = library_path(variant)
    if path not in _lib:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is missing: build it with python -m paper_2609_40247_amd.build")
        lib = ctypes.CDLL(path)
        lib.herschel_workspace_size.restype = ctypes.c_int
        lib.herschel_workspace_size.argtypes = [ctypes.c_int64, ctypes.POINTER(HerschelParams),
                                                ctypes.POINTER(ctypes.c_size_t)]
        lib.herschel_trace_analyze.restype = ctypes.c_int
        lib.herschel_trace_analyze.argtypes = [ctypes.POINTER(HerschelEvents), ctypes.c_int64,
                                               ctypes.POINTER(HerschelParams), ctypes.POINTER(HerschelOutputs)]
        lib.herschel_trace_analyze_static.restype = ctypes.c_int
        lib.herschel_trace_analyze_static.argtypes = [ctypes.POINTER(HerschelEvents), ctypes.c_int64,
                                                      ctypes.POINTER(HerschelParams), ctypes.POINTER(HerschelOutputs)]
        lib.herschel_trace_analyze_batch.restype = ctypes.c_int
        lib.herschel_trace_analyze_batch.argtypes = [ctypes.POINTER(HerschelEvents), ctypes.POINTER(ctypes.c_int64),
                                                     ctypes.c_int32, ctypes.POINTER(HerschelParams),
                                                     ctypes.POINTER(HerschelOutputs)]
        lib.herschel_trace_analyze_chunked.restype = ctypes.c_int
        lib.herschel_trace_analyze_chunked.argtypes = [ctypes.POINTER(HerschelEvents), ctypes.POINTER(ctypes.c_int64),
                                                       ctypes.c_int32, ctypes.c_int32,
                                                       ctypes.POINTER(HerschelEvents), ctypes.c_int64,
                                                       ctypes.POINTER(HerschelParams),
                                                       ctypes.POINTER(HerschelOutputs)]
        lib.herschel_strerror.restype = ctypes.c_char_p
        lib.herschel_strerror.argtypes = [ctypes.c_int]
        lib.herschel_time_stage.restype = ctypes.c_int
        lib.herschel_time_stage.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p]
        lib.herschel_sort_stats.restype = ctypes.c_int
        lib.herschel_sort_stats.argtypes = [ctypes.POINTER(HerschelParams), ctypes.POINTER(ctypes.c_int32)]
        _lib[path] = lib
    return _lib[path]


# ------------------------------------------------------------ thin wrappers
def herschel_workspace_size(n: int, params: HerschelParams, lib=None) -> int:
    lib = lib or load()
    out = ctypes.c_size_t(0)
    code = lib.herschel_workspace_size(int(n), ctypes.byref(params), ctypes.byref(out))
    if code != OK:
        raise ValueError(f"herschel_workspace_size: {herschel_strerror(code, lib)}")
    return int(out.value)


def herschel_trace_analyze(events: HerschelEvents, n: int, params: HerschelParams, out: HerschelOutputs,
                           lib=None) -> int:
    lib = lib or load()
    return int(lib.herschel_trace_analyze(ctypes.byref(events), int(n), ctypes.byref(params), ctypes.byref(out)))


def herschel_trace_analyze_static(events: HerschelEvents, n: int, params: HerschelParams, out: HerschelOutputs,
                                  lib=None) -> int:
    """The entry point that allocates nothing: params' workspace is ignored
    and the library's static scratch is used instead."""
    lib = lib or load()
    return int(lib.herschel_trace_analyze_static(ctypes.byref(events), int(n), ctypes.byref(params),
                                                 ctypes.byref(out)))


def herschel_trace_analyze_batch(events: HerschelEvents, offsets: np.ndarray, params: list, outs: list,
                                 lib=None) -> int:
    lib = lib or load()
    T = len(params)
    offs = np.ascontiguousarray(offsets, dtype=np.int64)
    parr = (HerschelParams * T)(*params)
    oarr = (HerschelOutputs * T)(*outs)
    return int(lib.herschel_trace_analyze_batch(ctypes.byref(events),
                                                offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                                T, parr, oarr))


def herschel_trace_analyze_chunked(host: HerschelEvents, offsets: np.ndarray, chunk_traces: int, staging: list,
                                   staging_rows: int, params: list, outs: list, lib=None) -> int:
    """The batch over host-resident traces, uploaded chunk by chunk into two
    device staging sets (``staging``: two HerschelEvents of device pointers)."""
    lib = lib or load()
    T = len(params)
    offs = np.ascontiguousarray(offsets, dtype=np.int64)
    parr = (HerschelParams * T)(*params)
    oarr = (HerschelOutputs * T)(*outs)
    sarr = (HerschelEvents * 2)(*staging)
    return int(lib.herschel_trace_analyze_chunked(ctypes.byref(host),
                                                  offs.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                                  T, int(chunk_traces), sarr, int(staging_rows), parr, oarr))


STAGES = ("init", "prep", "hist", "names", "sort", "timeline", "overlap", "contain", "join", "opagg", "edges",
          "final", "waits", "sol", "crit", "graph")


def herschel_time_stage(stage: int, start_event, stop_event, lib=None) -> int:
    """Record two torch.cuda.Event objects around one stage of following
    calls (None, None stops)."""
    lib = lib or load()
    a = None if start_event is None else start_event.cuda_event
    b = None if stop_event is None else stop_event.cuda_event
    if (start_event is not None and not a) or (stop_event is not None and not b):
        raise ValueError("record the events once before handing them over (torch creates them lazily)")
    return int(lib.herschel_time_stage(int(stage), a, b))


def herschel_sort_stats(params: "HerschelParams", lib=None) -> list[tuple[int, int, int]]:
    """(keys, skipped-digit mask, digits) of the timeline, join and
    containment sorts of the last call made with params' workspace."""
    lib = lib or load()
    out = (ctypes.c_int32 * 9)()
    code = int(lib.herschel_sort_stats(ctypes.byref(params), out))
    if code != 0:
        raise RuntimeError(f"herschel_sort_stats: {code}")
    return [(int(out[3 * i]), int(out[3 * i + 1]) & 0xFFFFFFFF, int(out[3 * i + 2])) for i in range(3)]


def herschel_strerror(code: int, lib=None) -> str:
    lib = lib or load()
    return lib.herschel_strerror(int(code)).decode()


# ------------------------------------------------------------ marshalling
def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def device_columns(cols: dict, device="cuda") -> dict:
    """Host numpy columns -> contiguous device tensors of the ABI's types
    (flops and bytes only when the columns hold them)."""
    dt = dict(ts=np.int64, te=np.int64, corr=np.int64, pid=np.int32, lane=np.int32, name=np.int32, kind=np.uint8,
              flops=np.int64, bytes=np.int64, graph_node=np.int32)
    return {k: torch.from_numpy(np.ascontiguousarray(cols[k], dtype=dt[k])).to(device)
            for k in dt if cols.get(k) is not None}


def events_struct(dcols: dict, offset: int = 0) -> HerschelEvents:
    return HerschelEvents(**{k: dcols[k].data_ptr() + offset * dcols[k].element_size() for k in dcols})


class Analyzer:
    """Device buffers (params arrays, workspace, outputs) for one problem shape.

    ``params`` is a dict with window_begin, window_end, gap_threshold,
    n_procs, n_streams, n_threads, n_names, n_op_names, clock_offset,
    stream_class, edges (numpy structured array) and flags; ``n_max`` the
    largest row count this analyzer will be called with."""

    def __init__(self, params: dict, n_max: int, gap_capacity: int | None = None, device="cuda",
                 stream: torch.cuda.Stream | None = None, lib=None, op_fill: int = -3, workspace: bool = True):
        self.lib = lib or load()
        self.device = device
        self.p = dict(params)
        P, S, NN = int(params["n_procs"]), int(params["n_streams"]), int(params["n_names"])
        self.stream = stream
        off = params.get("clock_offset")
        cls = params.get("stream_class")
        edges = params.get("edges")
        self.n_edges = 0 if edges is None else len(edges)
        self.d_off = None if off is None else torch.from_numpy(np.ascontiguousarray(off, np.int64)).to(device)
        self.d_cls = None if cls is None else torch.from_numpy(np.ascontiguousarray(cls, np.uint8)).to(device)
        ref = params.get("ref_sol_ppm")
        self.d_ref = None if ref is None else torch.from_numpy(np.ascontiguousarray(ref, np.int64)).to(device)
        self.d_edges = None
        if self.n_edges:
            raw = np.ascontiguousarray(edges).view(np.uint8).reshape(-1)
            self.d_edges = torch.from_numpy(raw.copy()).to(device)
        self.n_max = int(n_max)
        if gap_capacity is None:
            gap_capacity = self.n_max + P * S
        self.gap_capacity = int(gap_capacity)
        self.op_fill = op_fill
        self.params = self._params_struct(None, 0)
        self.ws_bytes = herschel_workspace_size(self.n_max, self.params, self.lib)
        # outputs-only analyzers serve as the later traces of a batch call,
        # which runs in the first trace's workspace
        self.ws = torch.empty(max(self.ws_bytes, 256) if workspace else 256, dtype=torch.uint8, device=device)
        if not workspace:
            self.ws_bytes = 0
        n = max(self.n_max, 1)
        gc = max(self.gap_capacity, 1)
        z = lambda k, dt: torch.empty(k, dtype=dt, device=device)
        self.o = dict(
            link=z(n, torch.int32), aux=z(n, torch.int32), op_nkern=z(n, torch.int32),
            op_first=z(n, torch.int64), op_last=z(n, torch.int64), op_ksum=z(n, torch.int64),
            busy=z(P * S, torch.int64), idle=z(P * S, torch.int64), pair_overlap=z(P * S * S, torch.int64),
            class_busy=z(P * 3, torch.int64), class_overlap=z(P * 9, torch.int64), any_busy=z(P, torch.int64),
            name_count=z(NN, torch.int64), name_sum=z(NN, torch.int64), name_min=z(NN, torch.int64),
            name_max=z(NN, torch.int64), lat_hist=z(64, torch.int64),
            edge_wait=z(max(self.n_edges, 1), torch.int64), edge_status=z(max(self.n_edges, 1), torch.int32),
            gap_pid=z(gc, torch.int32), gap_stream=z(gc, torch.int32), gap_begin=z(gc, torch.int64),
            gap_end=z(gc, torch.int64), gap_flags=z(gc, torch.uint8), counters=z(len(COUNTERS), torch.int64),
            dev_idle=z(P, torch.int64), op_span=z(P * int(params["n_op_names"]), torch.int64),
            op_idle=z(P * int(params["n_op_names"]), torch.int64),
            **{k: z(n, torch.int64) for k in SOL_ROW_OUTPUTS},
            **{k: z(int(params["n_op_names"]), torch.int64) for k in SOL_NAME_OUTPUTS},
            crit_time=z(n, torch.int64), crit_flags=z(n, torch.uint8), crit_proc=z(P * 8, torch.int64),
            launch_first=z(n, torch.int64), launch_last=z(n, torch.int64),
            **{k: z(max(int(params.get("n_graph_nodes", 1)), 1), torch.int64) for k in GRAPH_NODE_OUTPUTS},
            **{k: z(int(params["n_op_names"]), torch.int64) for k in OPNAME_OUTPUTS},
        )
        self.params = self._params_struct(self.ws.data_ptr(), self.ws_bytes)
        self.outs = HerschelOutputs(gap_capacity=self.gap_capacity,
                                    **{k: v.data_ptr() for k, v in self.o.items()})

    def _params_struct(self, ws, ws_bytes) -> HerschelParams:
        p = self.p
        st = self.stream.cuda_stream if self.stream is not None else torch.cuda.current_stream().cuda_stream
        return HerschelParams(
            window_begin=int(p["window_begin"]), window_end=int(p["window_end"]),
            gap_threshold=int(p["gap_threshold"]), n_procs=int(p["n_procs"]), n_streams=int(p["n_streams"]),
            n_threads=int(p["n_threads"]), n_names=int(p["n_names"]), n_op_names=int(p["n_op_names"]),
            clock_offset=_ptr(self.d_off), stream_class=_ptr(self.d_cls), edges=_ptr(self.d_edges),
            n_edges=self.n_edges, flags=int(p.get("flags", 3)), hip_stream=st, workspace=ws,
            workspace_bytes=ws_bytes, peak_flops=int(p.get("peak_flops", 0)), peak_bytes=int(p.get("peak_bytes", 0)),
            ref_sol_ppm=_ptr(self.d_ref), n_graph_nodes=int(p.get("n_graph_nodes", 0)))

    def prefill(self) -> None:
        """Fill the op arrays with a marker so rows the library must not write
        can be checked."""
        for k in ("op_nkern", "op_first", "op_last", "op_ksum", "crit_time", "launch_first",
                  "launch_last") + SOL_ROW_OUTPUTS:
            self.o[k].fill_(self.op_fill)
        self.o["crit_flags"].fill_(0xFD)

    def run(self, events: HerschelEvents, n: int) -> int:
        if n > self.n_max:
            raise ValueError(f"n={n} exceeds this analyzer's n_max={self.n_max}")
        return herschel_trace_analyze(events, n, self.params, self.outs, self.lib)

    def results(self, n: int) -> dict:
        """Copy the outputs of the last call to host numpy (oracle layout)."""
        h = {k: v.cpu().numpy() for k, v in self.o.items()}
        c = dict(zip(COUNTERS, (int(x) for x in h.pop("counters"))))
        res = {k: h[k][:n] for k in ("link", "aux", "op_nkern", "op_first", "op_last", "op_ksum", "crit_time",
                                     "crit_flags", "launch_first", "launch_last") + SOL_ROW_OUTPUTS}
        for k in ("busy", "idle", "pair_overlap", "class_busy", "class_overlap", "any_busy", "name_count",
                  "name_sum", "name_min", "name_max", "lat_hist", "dev_idle", "op_span", "op_idle",
                  "crit_proc") + SOL_NAME_OUTPUTS + GRAPH_NODE_OUTPUTS + OPNAME_OUTPUTS:
            res[k] = h[k]
        res["edge_wait"] = h["edge_wait"][:self.n_edges]
        res["edge_status"] = h["edge_status"][:self.n_edges]
        ng = min(c["n_gaps_total"], self.gap_capacity)
        for k in ("gap_pid", "gap_stream", "gap_begin", "gap_end", "gap_flags"):
            res[k] = h[k][:ng]
        res["counters"] = c
        return res


def analyze(cols: dict, params: dict, gap_capacity: int | None = None, variant: str | None = None):
    """One call on host columns: copy to the GPU, analyze, copy back.
    Returns (code, outputs) in the same layout as the oracle's wrapper."""
    lib = load(variant)
    n = len(cols["ts"])
    if gap_capacity is None:
        gap_capacity = int(np.count_nonzero(np.asarray(cols["kind"]) == KERNEL)) + \
            int(params["n_procs"]) * int(params["n_streams"])
    an = Analyzer(params, n, gap_capacity=gap_capacity, lib=lib)
    an.prefill()
    d = device_columns(cols)
    code = an.run(events_struct(d), n)
    torch.cuda.synchronize()
    return code, an.results(n)
