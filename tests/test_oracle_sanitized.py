"""The oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU).

The oracle is compiled a second time with ``-fsanitize=address,undefined``
(every report fatal) and run in a child process, with the sanitizer runtime
preloaded, over the tiny adversarial traces with every output flag, the
error paths (invalid rows, a gap list too short, bad parameters), the two
hand-worked timelines and the tiny workload trace.  Each call must finish
without a report and give the same results as the plain build.  Signed
overflow is not checked: the sums the outputs define wrap modulo 2^64 by
design, and the oracle computes them in unsigned arithmetic where it matters.
"""
from __future__ import annotations

import os
import subprocess
import sys
import textwrap

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _runtime(name: str) -> str | None:
    r = subprocess.run(["gcc", f"-print-file-name={name}"], capture_output=True, text=True)
    path = r.stdout.strip()
    return path if r.returncode == 0 and os.path.isabs(path) and os.path.exists(path) else None


@pytest.fixture(scope="module")
def sanitized_lib(tmp_path_factory):
    asan = _runtime("libasan.so")
    if asan is None:
        pytest.skip("gcc has no AddressSanitizer runtime here")
    out = str(tmp_path_factory.mktemp("asan") / "libherschel_oracle_asan.so")
    src = os.path.join(os.path.dirname(oracle.__file__), "herschel_oracle.c")
    cmd = ["gcc", "-O1", "-g", "-std=c11", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
           "-fno-sanitize=signed-integer-overflow", "-fno-sanitize-recover=all", "-shared", "-fPIC",
           "-o", out, src]
    subprocess.run(cmd, check=True)
    return out, asan


CHILD = textwrap.dedent(r"""
    import sys
    import numpy as np
    sys.path[:0] = [@ROOT@, @TESTS@]
    import oracle
    from paper_2609_40247_amd import synth
    from fixtures import load_golden

    san = oracle.load_library(@LIB@)
    plain = oracle._load()

    def same(cols, params, label, cap=None):
        a = oracle.analyze(cols, params, gap_capacity=cap, lib=san)
        b = oracle.analyze(cols, params, gap_capacity=cap, lib=plain)
        assert a[0] == b[0], (label, a[0], b[0])
        for k in b[1]:
            if k == "counters":
                assert a[1][k] == b[1][k], (label, k)
            else:
                assert np.array_equal(a[1][k], b[1][k]), (label, k)
        return a[0]

    calls = 0
    codes = set()
    for seed in range(60):
        tr = synth.random_small(seed=seed, flags=3 | 4 | 16 if seed % 2 else 3)
        cols = tr.columns()
        codes.add(same(cols, tr.params, tr.label)); calls += 1
        c2, p2 = synth.add_op_costs(cols, tr.params, seed, flops_median=1e7, bytes_median=3e4)
        codes.add(same(c2, p2, tr.label + " sol")); calls += 1
        if seed % 5 == 0:  # a gap list one entry short
            codes.add(same(cols, tr.params, tr.label + " capacity", cap=1)); calls += 1
        if seed % 7 == 0:  # invalid rows: a bad kind, a stream out of range, an end before the start
            bad = {k: np.array(v, copy=True) for k, v in cols.items()}
            bad["kind"][seed % len(bad["kind"])] = 3
            codes.add(same(bad, tr.params, tr.label + " bad kind")); calls += 1
            bad = {k: np.array(v, copy=True) for k, v in cols.items()}
            i = int(np.flatnonzero(bad["kind"] == 2)[0])
            bad["lane"][i] = tr.params["n_streams"]
            codes.add(same(bad, tr.params, tr.label + " bad stream")); calls += 1
            bad = {k: np.array(v, copy=True) for k, v in cols.items()}
            bad["te"][3] = bad["ts"][3] - 1
            codes.add(same(bad, tr.params, tr.label + " te < ts")); calls += 1
    tr = synth.random_small(seed=5)
    codes.add(same(tr.columns(), dict(tr.params, window_end=tr.params["window_begin"]), "empty window")); calls += 1
    codes.add(same(tr.columns(), dict(tr.params, n_streams=65), "65 streams")); calls += 1
    e = {k: np.array(v[:0], copy=True) for k, v in tr.columns().items()}
    codes.add(same(e, tr.params, "empty trace")); calls += 1
    cols, p = synth.graph_replay_trace(n_steps=12, n_nodes=60)
    codes.add(same(cols, dict(p, flags=p["flags"] | 16), "graph replays")); calls += 1
    for name in ("t1_worked_timeline.json", "t2_worked_timeline.json"):
        cols, p, _ = load_golden(name)
        codes.add(same(cols, p, name)); calls += 1
    tr = synth.config0()
    codes.add(same(tr.columns(), dict(tr.params, flags=3 | 4 | 16), "config0")); calls += 1
    print("ok", calls, sorted(codes))
""")


def test_oracle_clean_under_sanitizers(sanitized_lib):
    lib, asan = sanitized_lib
    code = (CHILD.replace("@ROOT@", repr(ROOT)).replace("@TESTS@", repr(os.path.dirname(os.path.abspath(__file__))))
            .replace("@LIB@", repr(lib)))
    env = dict(os.environ)
    env["LD_PRELOAD"] = asan
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1:allocator_may_return_null=0"
    env["UBSAN_OPTIONS"] = "halt_on_error=1:print_stacktrace=1"
    r = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True, timeout=900)
    assert r.returncode == 0, r.stdout[-4000:] + r.stderr[-8000:]
    last = r.stdout.strip().splitlines()[-1]
    assert last.startswith("ok "), r.stdout[-2000:]
    calls = int(last.split()[1])
    assert calls >= 150, last
    # the error paths were reached: success, bad parameters, invalid rows, gap capacity
    codes = {int(x) for x in last.split("[", 1)[1].rstrip("]").split(",")}
    assert {0, -1, -2, -3} <= codes, last
