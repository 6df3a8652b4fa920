"""Test inputs: golden fixtures and the seeded generators (no analysis arithmetic)."""
from __future__ import annotations

import json
import os

import numpy as np

from paper_2609_40247_amd import synth

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
I64_MAX = (1 << 63) - 1
I64_MIN = -(1 << 63)


def _val(x):
    return {"MAX": I64_MAX, "MIN": I64_MIN}.get(x, x) if isinstance(x, str) else x


def load_golden(name: str):
    with open(os.path.join(GOLDEN, name)) as f:
        g = json.load(f)
    rows = np.array(g["rows"], dtype=np.int64)
    f_ = g["row_fields"]
    col = {k: rows[:, f_.index(k)] for k in f_}
    cols = dict(ts=col["ts"].astype(np.int64), te=col["te"].astype(np.int64),
                corr=col["corr"].astype(np.int64), pid=col["pid"].astype(np.int32),
                lane=col["lane"].astype(np.int32), name=col["name"].astype(np.int32),
                kind=col["kind"].astype(np.uint8))
    p = dict(g["params"])
    e = np.zeros(len(p["edges"]), synth.EDGE_DTYPE)
    for i, (a, b, c, d) in enumerate(p["edges"]):
        e[i] = (a, b, c, d)
    p["edges"] = e
    if p["clock_offset"] is not None:
        p["clock_offset"] = np.array(p["clock_offset"], np.int64)
    if p["stream_class"] is not None:
        p["stream_class"] = np.array(p["stream_class"], np.uint8)
    exp = g["expect"]
    exp["edge_wait"] = [_val(x) for x in exp["edge_wait"]]
    exp["op"] = {int(k): [_val(x) for x in v] for k, v in exp["op"].items()}
    return cols, p, g


def load_golden_raw(name: str) -> dict:
    """A golden fixture's JSON as written (fixtures that are not row tables)."""
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)
