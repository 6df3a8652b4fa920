"""Element-by-element comparison of two result sets (test code)."""
from __future__ import annotations

import numpy as np

COUNTERS = ("n_admitted_cpu", "n_admitted_launch", "n_admitted_kernel", "n_outside_window",
            "n_matched", "n_unmatched_kernels", "n_unmatched_launches", "n_dup_launch_corr",
            "n_unattributed_kernels", "n_improper_nesting", "n_negative_latency", "n_gaps_total",
            "first_invalid")


def _eq(name, a, b, ctx):
    a = np.asarray(a)
    b = np.asarray(b)
    if a.shape != b.shape:
        raise AssertionError(f"{ctx}: {name} shape {a.shape} != {b.shape}")
    bad = np.flatnonzero(a.reshape(-1) != b.reshape(-1))
    if len(bad):
        i = bad[:8]
        raise AssertionError(f"{ctx}: {name} differs at {len(bad)} of {a.size} entries; first {i.tolist()}: "
                             f"{a.reshape(-1)[i].tolist()} vs {b.reshape(-1)[i].tolist()}")


def assert_same(got: tuple, want: tuple, params: dict, ctx: str = "") -> None:
    """``got`` and ``want`` are (code, outputs) pairs in the layout of the
    oracle wrapper; every output that the flags select is compared."""
    gc, g = got
    wc, w = want
    if gc != wc:
        raise AssertionError(f"{ctx}: return code {gc} != {wc}")
    if wc == -2:
        assert g["counters"]["first_invalid"] == w["counters"]["first_invalid"], ctx
        return
    for k in COUNTERS:
        if g["counters"][k] != w["counters"][k]:
            raise AssertionError(f"{ctx}: counter {k}: {g['counters'][k]} != {w['counters'][k]}")
    keys = ["link", "aux", "busy", "idle", "lat_hist", "name_count", "name_sum", "name_min", "name_max",
            "opname_count", "opname_sum", "opname_min", "opname_max",
            "gap_pid", "gap_stream", "gap_begin", "gap_end", "gap_flags", "edge_wait", "edge_status"]
    if params.get("flags", 3) & 1:
        keys += ["op_nkern", "op_first", "op_last", "op_ksum"]
    if params.get("flags", 3) & 2:
        keys += ["pair_overlap", "class_busy", "class_overlap", "any_busy"]
    if params.get("flags", 3) & 4:
        keys += ["dev_idle", "op_span", "op_idle"]
    if params.get("flags", 3) & 8:
        keys += ["op_mfu", "op_mbu", "op_sol", "opn_flops", "opn_bytes", "opn_time", "opn_sol", "opn_hot"]
    if params.get("flags", 3) & 16:
        keys += ["crit_time", "crit_flags", "crit_proc"]
    if params.get("flags", 3) & 32:
        keys += ["launch_first", "launch_last", "gn_count", "gn_sum", "gn_min", "gn_max", "gn_offset"]
    for k in keys:
        _eq(k, g[k], w[k], ctx)
