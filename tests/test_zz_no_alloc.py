"""The entry point that allocates nothing (herschel_trace_analyze_static)
against herschel_trace_analyze, through the C ABI: two calls in a row, the
second smaller than the first, every output compared element by element
(and with the oracle), plus the size limit of the static scratch."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from compare import assert_same
from paper_2609_40247_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def H():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_40247_amd import herschel
    herschel.load()
    return herschel


def _run_both(H, tr, label):
    cols, p = tr.columns(), tr.params
    n = tr.n
    cap = n + p["n_procs"] * p["n_streams"]
    ref = H.Analyzer(p, n, gap_capacity=cap)
    # outputs only: the static entry point ignores the workspace
    st = H.Analyzer(p, n, gap_capacity=cap, workspace=False)
    assert H.herschel_workspace_size(n, ref.params) <= H.STATIC_SCRATCH_BYTES, label
    ref.prefill()
    st.prefill()
    d = H.device_columns(cols)
    ev = H.events_struct(d)
    torch.cuda.synchronize()
    print(f"{label}: {n} rows, herschel_trace_analyze", flush=True)
    c_ref = H.herschel_trace_analyze(ev, n, ref.params, ref.outs)
    torch.cuda.synchronize()
    print(f"{label}: {n} rows, herschel_trace_analyze_static", flush=True)
    c_st = H.herschel_trace_analyze_static(ev, n, st.params, st.outs)
    torch.cuda.synchronize()
    r_ref, r_st = ref.results(n), st.results(n)
    assert c_st == c_ref == 0, (label, c_st, c_ref)
    assert r_st["counters"] == r_ref["counters"], label
    # outputs of flags this call does not set are never written
    flags = p.get("flags", 3)
    unwritten = (() if flags & 4 else ("dev_idle", "op_span", "op_idle")) + \
        (() if flags & 8 else H.SOL_ROW_OUTPUTS + H.SOL_NAME_OUTPUTS) + \
        (() if flags & 16 else ("crit_time", "crit_flags", "crit_proc")) + \
        (() if flags & 32 else ("launch_first", "launch_last") + H.GRAPH_NODE_OUTPUTS)
    for k in r_ref:
        if k != "counters" and k not in unwritten:
            assert np.array_equal(r_st[k], r_ref[k]), (label, k)
    assert_same((c_st, r_st), oracle.analyze(cols, p, gap_capacity=cap), p, label + " vs oracle")


def test_static_scratch_matches_workspace_entry(H):
    big = synth.config1(n_steps=70)
    small = synth.config0()
    assert small.n < big.n
    _run_both(H, big, "first call (decode-step trace, 70 steps)")
    _run_both(H, small, "second call (tiny trace, smaller)")


def test_static_scratch_rejects_larger_inputs(H):
    tr = synth.config1(n_steps=150)
    p = tr.params
    an = H.Analyzer(p, tr.n, workspace=False)
    assert H.herschel_workspace_size(tr.n, an.params) > H.STATIC_SCRATCH_BYTES
    d = H.device_columns(tr.columns())
    code = H.herschel_trace_analyze_static(H.events_struct(d), tr.n, an.params, an.outs)
    assert code == H.ETOOBIG
    assert "static scratch" in H.herschel_strerror(code)
