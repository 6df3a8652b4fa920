"""The rocprofv3 adapter on a real MI355X trace sample (CPU only): the
records it makes, and what the oracle finds in them."""
from __future__ import annotations

import csv
import os

import numpy as np

import oracle
from paper_2609_40247_amd import ingest

SAMPLE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "rocprof_sample")


def _csv(name):
    with open(os.path.join(SAMPLE, name), newline="") as fh:
        return list(csv.DictReader(fh))


def test_records_and_tables():
    t = ingest.read_rocprofv3(SAMPLE)
    c, p = t.columns, t.params
    kern, api, mark = _csv("sample_kernel_trace.csv"), _csv("sample_hip_api_trace.csv"), _csv(
        "sample_marker_api_trace.csv")
    assert [int((c["kind"] == k).sum()) for k in (0, 1, 2)] == [len(mark), len(api), len(kern)]
    assert t.op_names == ["layer1", "layer2", "sample", "decode_step", "graph_step"]
    assert "hipGraphLaunch" in t.api_names and "hipLaunchKernel" in t.api_names
    assert p["n_procs"] == 1 and p["n_threads"] == 1 and p["n_streams"] == len({k["Stream_Id"] for k in kern})
    assert p["window_begin"] == int(c["ts"].min()) and p["window_end"] > int(c["te"].max())
    # times and correlation ids are copied as recorded
    k0 = kern[0]
    i = int(np.flatnonzero((c["kind"] == 2) & (c["corr"] == int(k0["Correlation_Id"])))[0])
    assert (int(c["ts"][i]), int(c["te"][i])) == (int(k0["Start_Timestamp"]), int(k0["End_Timestamp"]))
    assert t.kernel_names[c["name"][i]] == k0["Kernel_Name"]


def test_graph_replays_get_node_ranks():
    t = ingest.read_rocprofv3(SAMPLE)
    c, p = t.columns, t.params
    graph_calls = [int(a["Correlation_Id"]) for a in _csv("sample_hip_api_trace.csv")
                   if a["Function"] == "hipGraphLaunch"]
    assert len(graph_calls) == 4 and p["flags"] & 32 and p["n_graph_nodes"] == 4
    for corr in graph_calls:
        m = (c["kind"] == 2) & (c["corr"] == corr)
        order = np.argsort(c["ts"][m], kind="stable")
        assert c["graph_node"][m][order].tolist() == [0, 1, 2, 3]
    assert (c["graph_node"][(c["kind"] == 2) & ~np.isin(c["corr"], graph_calls)] == -1).all()


def test_oracle_on_the_sample():
    """Every kernel joins its call; the layer ranges nest in their step; each
    graph node is seen once per replay with the same kernel name."""
    t = ingest.read_rocprofv3(SAMPLE)
    c, p = t.columns, dict(t.params, flags=t.params["flags"] | 4 | 16)
    code, o = oracle.analyze(c, p)
    assert code == 0
    cnt = o["counters"]
    assert cnt["n_matched"] == cnt["n_admitted_kernel"] == int((c["kind"] == 2).sum())
    assert cnt["n_improper_nesting"] == 0 and cnt["n_outside_window"] == 0
    names = t.op_names
    nested = {}
    for i in np.flatnonzero(c["kind"] == 0):
        parent = int(o["link"][i])
        key = (names[c["name"][i]], names[c["name"][parent]] if parent >= 0 else None)
        nested[key] = nested.get(key, 0) + 1
    # six eager steps; the warm-up and the capture run their layers outside
    # any step; every sample lies in its step
    assert nested[("layer1", "decode_step")] == nested[("layer2", "decode_step")] == 6
    assert nested[("sample", "decode_step")] == 6 and nested[("sample", "graph_step")] == 4
    assert nested[("layer1", None)] == 2
    assert o["gn_count"].tolist() == [4, 4, 4, 4]
    for q in range(4):
        ks = np.flatnonzero((c["kind"] == 2) & (c["graph_node"] == q))
        assert len({int(c["name"][k]) for k in ks}) == 1
    cp = o["crit_proc"]
    assert cp[0] == cp[1:].sum() > 0
