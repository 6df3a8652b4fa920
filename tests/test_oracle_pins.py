"""Pins of the CPU oracle against values fixed independently of it.

* hand-built worked timelines (tests/golden, expected values derived by hand);
* the per-nanosecond brute force of tests/bruteforce.py on tiny adversarial
  traces (ties, zero-length kernels, duplicate ids, improper nesting, offsets);
* invariants that hold for any input;
* ground truth that the generator drew (latencies, drops, names, gaps);
* metamorphic relations (row permutation, time shift, clock offsets);
* the error paths of the boundary.
"""
from __future__ import annotations

import numpy as np
import pytest

import bruteforce
import oracle
from compare import COUNTERS, assert_same
from fixtures import I64_MAX, I64_MIN, load_golden, load_golden_raw
from paper_2609_40247_amd import synth

GOLDEN = ["t1_worked_timeline.json", "t2_worked_timeline.json"]


def _check_expect(o, cols, exp):
    for k, v in exp["counters"].items():
        assert o["counters"][k] == v, k
    assert o["link"].tolist() == exp["link"]
    assert o["aux"].tolist() == exp["aux"]
    for r, (nk, first, last, ksum) in exp["op"].items():
        assert (o["op_nkern"][r], o["op_first"][r], o["op_last"][r], o["op_ksum"][r]) == (nk, first, last, ksum), r
    # rows that are not admitted CPU ops are never written
    not_op = [i for i in range(len(cols["ts"])) if i not in exp["op"]]
    assert np.all(o["op_nkern"][not_op] == oracle.UNWRITTEN_I32)
    assert o["busy"].tolist() == exp["busy"] and o["idle"].tolist() == exp["idle"]
    gaps = list(zip(o["gap_pid"].tolist(), o["gap_stream"].tolist(), o["gap_begin"].tolist(),
                    o["gap_end"].tolist(), o["gap_flags"].tolist()))
    assert gaps == [tuple(g) for g in exp["gaps"]]
    hist = np.zeros(64, np.int64)
    for b, c in exp["lat_hist"].items():
        hist[int(b)] = c
    assert o["lat_hist"].tolist() == hist.tolist()
    for k in ("name_count", "name_sum", "name_min", "name_max", "pair_overlap", "any_busy", "class_busy",
              "class_overlap", "edge_wait", "edge_status"):
        assert o[k].tolist() == exp[k], k


@pytest.mark.parametrize("name", GOLDEN)
def test_worked_timeline(name):
    cols, p, g = load_golden(name)
    code, o = oracle.analyze(cols, p)
    assert code == g["expect"]["code"]
    _check_expect(o, cols, g["expect"])


def test_worked_timeline_all_compute():
    cols, p, g = load_golden("t1_worked_timeline.json")
    p["stream_class"] = None
    code, o = oracle.analyze(cols, p)
    assert o["class_busy"].tolist() == g["expect_all_compute"]["class_busy"]
    assert o["class_overlap"].tolist() == g["expect_all_compute"]["class_overlap"]


def test_worked_timeline_without_containment():
    cols, p, g = load_golden("t1_worked_timeline.json")
    p["flags"] = 0
    code, o = oracle.analyze(cols, p)
    kind = cols["kind"]
    exp_link = np.array(g["expect"]["link"])
    exp_aux = np.array(g["expect"]["aux"])
    adm = exp_link != -2
    # kernels keep their launch; launches keep their kernel count
    assert (o["link"][kind == 2] == exp_link[kind == 2]).all()
    assert (o["aux"][kind == 1] == exp_aux[kind == 1]).all()
    assert (o["link"][(kind != 2) & adm] == -1).all()
    assert (o["aux"][(kind != 1) & adm] == -1).all()
    assert (o["op_nkern"] == oracle.UNWRITTEN_I32).all()
    assert o["counters"]["n_unattributed_kernels"] == 0 and o["counters"]["n_improper_nesting"] == 0


# --------------------------------------------------------------------------- brute force

def _bf_compare(cols, p, o, b, ctx):
    bc = b["counters"]
    for k in COUNTERS:
        assert o["counters"][k] == bc[k], f"{ctx}: {k} {o['counters'][k]} != {bc[k]}"
    for k in ("link", "aux", "busy", "idle", "lat_hist", "name_count", "name_sum", "name_min", "name_max",
              "edge_wait", "edge_status"):
        assert o[k].tolist() == np.asarray(b[k]).tolist(), f"{ctx}: {k}"
    gaps = list(zip(o["gap_pid"].tolist(), o["gap_stream"].tolist(), o["gap_begin"].tolist(),
                    o["gap_end"].tolist(), o["gap_flags"].tolist()))
    assert gaps == [tuple(int(x) for x in g) for g in b["gaps"]], ctx
    for k, v in b["opname"].items():
        assert o[k].tolist() == v.tolist(), f"{ctx}: {k}"
    if p["flags"] & 1:
        for r, v in b["op"].items():
            assert (int(o["op_nkern"][r]), int(o["op_first"][r]), int(o["op_last"][r]), int(o["op_ksum"][r])) == v, \
                f"{ctx}: op {r}"
    if p["flags"] & 2:
        for k, v in b["overlap"].items():
            assert o[k].tolist() == v.tolist(), f"{ctx}: {k}"
    if p["flags"] & 4:
        for k, v in b["waits"].items():
            assert o[k].tolist() == v.tolist(), f"{ctx}: {k}"
    if p["flags"] & 8:
        for k in ("op_mfu", "op_mbu", "op_sol"):
            for r, v in b["sol"][k].items():
                assert int(o[k][r]) == v, f"{ctx}: {k} row {r}"
        for k in ("opn_flops", "opn_bytes", "opn_time", "opn_sol", "opn_hot"):
            assert o[k].tolist() == b["sol"][k].tolist(), f"{ctx}: {k}"
    if p["flags"] & 32:
        for k in ("launch_first", "launch_last"):
            for r, v in b["graph"][k].items():
                assert int(o[k][r]) == v, f"{ctx}: {k} row {r}"
        for k in ("gn_count", "gn_sum", "gn_min", "gn_max", "gn_offset"):
            assert o[k].tolist() == b["graph"][k].tolist(), f"{ctx}: {k}"
    if p["flags"] & 16:
        for r, v in b["crit"]["crit_time"].items():
            assert int(o["crit_time"][r]) == v, f"{ctx}: crit_time row {r}"
        for r, v in b["crit"]["crit_flags"].items():
            assert int(o["crit_flags"][r]) == v, f"{ctx}: crit_flags row {r}"
        assert o["crit_proc"].tolist() == b["crit"]["crit_proc"].tolist(), f"{ctx}: crit_proc"


BF_CASES = [dict(seed=s) for s in range(120)] + [
    dict(seed=1000 + s, n_rows=120, window=900, n_procs=3, n_streams=4, n_threads=3, corr_range=30) for s in range(30)
] + [dict(seed=2000 + s, n_rows=40, window=60, n_procs=1, n_streams=2, n_threads=1, corr_range=6, offsets=False)
     for s in range(30)] + [dict(seed=3000 + s, flags=s % 4) for s in range(16)] + [
    # many processes sharing few correlation ids: a join that forgets the
    # process would find another process's launch
    dict(seed=4000 + s, n_rows=30, window=200, n_procs=4, n_streams=2, n_threads=2, corr_range=3)
    for s in range(40)] + [
    # GPU idle coinciding with ops, with every other output and alone
    dict(seed=5000 + s, flags=7 if s % 2 else 4) for s in range(40)] + [
    dict(seed=5100 + s, n_rows=150, window=700, n_procs=2, n_streams=3, n_threads=3, n_op_names=3, flags=7)
    for s in range(20)] + [
    # the critical path, alone with containment and with every other output
    dict(seed=7000 + s, flags=17 if s % 2 else 23) for s in range(40)] + [
    dict(seed=7100 + s, n_rows=150, window=900, n_procs=3, n_streams=3, n_threads=2, corr_range=40, flags=17)
    for s in range(20)] + [
    # few distinct times: ties between releases everywhere
    dict(seed=7200 + s, n_rows=50, window=30, n_procs=1, n_streams=2, n_threads=1, corr_range=8, offsets=False,
         flags=17) for s in range(20)]


SOL_BF_SEEDS = list(range(40))


def sol_case(seed):
    """A tiny adversarial trace with per-op counts scaled to its nanosecond
    ops, so that SOL falls on both sides of the reference; every fourth case
    saturates the ppm at INT64_MAX with peaks of 1 /s."""
    tr = synth.random_small(seed=6000 + seed, n_rows=80 if seed % 2 else 40, window=500)
    tiny = seed % 4 == 3
    return synth.add_op_costs(tr.columns(), tr.params, seed, ref=seed % 3 != 0, flops_median=1e7,
                              bytes_median=3e4, peak_flops=1 if tiny else 2_500_000_000_000_000,
                              peak_bytes=1 if tiny else 8_000_000_000_000)


@pytest.mark.parametrize("seed", SOL_BF_SEEDS)
def test_bruteforce_sol(seed):
    """Operator efficiency against Python's exact integers on tiny traces."""
    cols, p = sol_case(seed)
    code, o = oracle.analyze(cols, p)
    bcode, b = bruteforce.analyze(cols, p)
    assert code == bcode
    if code == 0:
        _bf_compare(cols, p, o, b, f"sol seed {seed}")


@pytest.mark.parametrize("case", BF_CASES, ids=lambda c: f"seed{c['seed']}")
def test_bruteforce(case):
    tr = synth.random_small(**case)
    cols, p = tr.columns(), tr.params
    code, o = oracle.analyze(cols, p)
    bcode, b = bruteforce.analyze(cols, p)
    assert code == bcode
    if code == -2:
        assert o["counters"]["first_invalid"] == b["counters"]["first_invalid"]
        return
    _bf_compare(cols, p, o, b, tr.label)


def test_bruteforce_coverage_of_degenerate_cases():
    """The random tiny traces really contain the cases they are meant to."""
    seen = dict(dup=0, improper=0, neg=0, multi=0, unattributed=0, zero=0, outside=0)
    for case in BF_CASES[:150]:
        tr = synth.random_small(**case)
        code, o = oracle.analyze(tr.columns(), tr.params)
        c = o["counters"]
        seen["dup"] += c["n_dup_launch_corr"] > 0
        seen["improper"] += c["n_improper_nesting"] > 0
        seen["neg"] += c["n_negative_latency"] > 0
        seen["unattributed"] += c["n_unattributed_kernels"] > 0
        seen["outside"] += c["n_outside_window"] > 0
        seen["multi"] += bool((o["aux"][tr.kind == 1] > 1).any())
        seen["zero"] += bool(((tr.te == tr.ts) & (tr.kind == 2) & (o["link"] != -2)).any())
    assert all(v >= 5 for v in seen.values()), seen


# --------------------------------------------------------------------------- invariants

def _invariants(tr, o):
    p = tr.params
    c = o["counters"]
    n = tr.n
    W = p["window_end"] - p["window_begin"]
    kind = tr.kind
    adm = o["link"] != -2
    assert c["n_admitted_cpu"] + c["n_admitted_launch"] + c["n_admitted_kernel"] + c["n_outside_window"] == n
    assert (o["busy"] + o["idle"] == W).all() and (o["busy"] >= 0).all()
    kern = np.flatnonzero((kind == 2) & adm)
    lau = np.flatnonzero((kind == 1) & adm)
    assert c["n_matched"] + c["n_unmatched_kernels"] == len(kern)
    matched = kern[o["link"][kern] >= 0]
    assert len(matched) == c["n_matched"]
    L = o["link"][matched]
    assert (kind[L] == 1).all() and (tr.pid[L] == tr.pid[matched]).all() and (tr.corr[L] == tr.corr[matched]).all()
    assert o["aux"][lau].sum() == c["n_matched"]
    assert (o["aux"][lau] == 0).sum() == c["n_unmatched_launches"]
    assert o["lat_hist"].sum() == c["n_matched"]
    assert o["name_count"].sum() == len(kern)
    d = tr.te[kern] - tr.ts[kern]
    assert o["name_sum"].sum() == d.sum()
    if p["flags"] & 2:
        P, S = p["n_procs"], p["n_streams"]
        pair = o["pair_overlap"].reshape(P, S, S)
        assert (np.diagonal(pair, axis1=1, axis2=2).reshape(-1) == o["busy"]).all()
        assert (pair == pair.transpose(0, 2, 1)).all()
        co = o["class_overlap"].reshape(P, 3, 3)
        assert (np.diagonal(co, axis1=1, axis2=2) == o["class_busy"].reshape(P, 3)).all()
        assert (o["any_busy"] <= o["class_busy"].reshape(P, 3).sum(1)).all()
        assert (o["any_busy"] >= o["class_busy"].reshape(P, 3).max(1)).all()
        assert (o["any_busy"] <= W).all()
    if p["flags"] & 1:
        ops = np.flatnonzero((kind == 0) & adm)
        par = o["link"][ops]
        # op n_kernels(parent) = self + sum over children
        selfk = np.zeros(n, np.int64)
        ka = o["aux"][kern]
        np.add.at(selfk, ka[ka >= 0], 1)
        child = np.zeros(n, np.int64)
        np.add.at(child, par[par >= 0], o["op_nkern"][ops[par >= 0]])
        assert (o["op_nkern"][ops] == selfk[ops] + child[ops]).all()
        ne = ops[o["op_nkern"][ops] > 0]
        assert (o["op_last"][ne] >= o["op_first"][ne]).all()
        assert (o["aux"][ops[par >= 0]] == o["aux"][par[par >= 0]] + 1).all()
        assert (o["aux"][ops[par < 0]] == 0).all()


@pytest.fixture(scope="module")
def cfg0():
    tr = synth.config0()
    return tr, oracle.analyze(tr.columns(), tr.params)


def test_config0_invariants(cfg0):
    tr, (code, o) = cfg0
    assert code == 0
    _invariants(tr, o)
    c = o["counters"]
    assert int((tr.kind == 0).sum()) == 20_000 and int((tr.kind == 1).sum()) == 20_000
    assert 19_000 < c["n_admitted_kernel"] < 20_000 and c["n_admitted_cpu"] > 19_900
    assert c["n_outside_window"] > 0


@pytest.mark.parametrize("maker", [lambda: synth.config1(n_steps=40), lambda: synth.config2(scale=0.03),
                                   lambda: synth.config3(n_procs=3, n_steps=20, n_edges=500)],
                         ids=["config1-small", "config2-small", "config3-small"])
def test_small_config_invariants(maker):
    tr = maker()
    code, o = oracle.analyze(tr.columns(), tr.params)
    assert code == 0
    _invariants(tr, o)


def test_threshold_minus_one_gaps_sum_to_idle(cfg0):
    tr, _ = cfg0
    p = dict(tr.params, gap_threshold=-1)
    code, o = oracle.analyze(tr.columns(), p)
    S = p["n_streams"]
    tot = np.zeros(p["n_procs"] * S, np.int64)
    np.add.at(tot, o["gap_pid"] * S + o["gap_stream"], o["gap_end"] - o["gap_begin"])
    assert (tot == o["idle"]).all()
    # gaps tile the complement: begins after ends within a stream, sorted
    key = o["gap_pid"].astype(np.int64) * S + o["gap_stream"]
    assert (np.diff(key) >= 0).all()


# --------------------------------------------------------------------------- generator ground truth

def _truth_check(tr, o):
    pr = tr.truth["procs"][0]
    C, L, K = tr.truth["counts"][0]
    row_of = tr.truth["row_of"]
    p = tr.params
    W0, W1 = p["window_begin"], p["window_end"]
    kept = ~pr["dropped"]
    Kg = len(pr["start"])
    krow = np.full(Kg, -1, np.int64)
    krow[kept] = row_of[C + L + np.arange(K)]
    lrow = row_of[C + np.arange(Kg)]
    k_in = (pr["start"] >= W0) & (pr["start"] < W1)
    l_in = (pr["l_ts"] >= W0) & (pr["l_ts"] < W1)
    both = kept & k_in & l_in
    # every recorded kernel joins exactly its own launch, with the drawn latency
    assert (o["link"][krow[both]] == lrow[both]).all()
    x = pr["start"][both] - pr["l_ts"][both]
    assert (x == pr["lat"][both]).all()
    hist = np.zeros(64, np.int64)
    b = np.where(x <= 0, 0, np.floor(np.log2(np.maximum(x, 1))).astype(np.int64) + 1)
    np.add.at(hist, b, 1)
    assert (o["lat_hist"] == hist).all()
    # unmatched launches are those whose kernel was dropped or fell outside
    assert o["counters"]["n_unmatched_launches"] == int((l_in & ~(kept & k_in)).sum())
    assert o["counters"]["n_unmatched_kernels"] == int((kept & k_in & ~l_in).sum())
    # names of the recorded, admitted kernels
    cnt = np.bincount(pr["name"][kept & k_in], minlength=p["n_names"])
    assert (o["name_count"] == cnt).all()
    # each drawn gap between queue neighbours that were both recorded shows up
    gaps = set(zip(o["gap_stream"].tolist(), o["gap_begin"].tolist(), o["gap_end"].tolist()))
    st = np.argsort(pr["start"], kind="stable")
    ok = 0
    for s in range(p["n_streams"]):
        m = st[pr["stream"][st] == s]
        for a, c in zip(m[:-1], m[1:]):
            if pr["first_in_queue"][c] or not (kept[a] and kept[c]) or not (k_in[a] and k_in[c]):
                continue
            assert pr["start"][c] - pr["end"][a] == pr["gap"][c]
            if pr["gap"][c] > p["gap_threshold"] and pr["end"][a] < W1:
                assert (s, int(pr["end"][a]), int(pr["start"][c])) in gaps
                ok += 1
            elif pr["end"][a] < W1:
                assert (s, int(pr["end"][a]), int(pr["start"][c])) not in gaps
    assert ok > 0


def test_config0_ground_truth(cfg0):
    tr, (code, o) = cfg0
    _truth_check(tr, o)


def test_config1_ground_truth():
    tr = synth.config1(n_steps=60)
    code, o = oracle.analyze(tr.columns(), tr.params)
    _truth_check(tr, o)


# --------------------------------------------------------------------------- metamorphic

def test_row_permutation(cfg0):
    tr, (code, o) = cfg0
    rng = np.random.default_rng(7)
    perm = rng.permutation(tr.n)  # new row j holds old row perm[j]
    inv = np.empty_like(perm)
    inv[perm] = np.arange(tr.n)
    t2 = tr.take(perm)
    code2, o2 = oracle.analyze(t2.columns(), t2.params)
    assert code2 == code
    kind = tr.kind
    for k in ("link", "aux"):
        old = o[k][perm]
        is_row = (old >= 0) & ((k == "link") | ((kind[perm] == 2) & (k == "aux")))
        exp = np.where(is_row, inv[np.maximum(old, 0)], old)
        assert (o2[k] == exp).all(), k
    for k in ("op_nkern", "op_first", "op_last", "op_ksum"):
        assert (o2[k] == o[k][perm]).all(), k
    for k in ("busy", "idle", "lat_hist", "name_count", "name_sum", "name_min", "name_max", "gap_begin",
              "gap_end", "gap_flags", "pair_overlap", "class_busy", "class_overlap", "any_busy"):
        assert (o2[k] == o[k]).all(), k
    for k in COUNTERS:
        assert o2["counters"][k] == o["counters"][k]


def test_global_time_shift(cfg0):
    tr, (code, o) = cfg0
    d = -123_456_789_012
    cols = tr.columns()
    cols["ts"] = cols["ts"] + d
    cols["te"] = cols["te"] + d
    p = dict(tr.params, window_begin=tr.params["window_begin"] + d, window_end=tr.params["window_end"] + d)
    code2, o2 = oracle.analyze(cols, p)
    for k in ("link", "aux", "op_nkern", "op_ksum", "busy", "idle", "lat_hist", "name_count", "name_sum",
              "name_min", "name_max", "gap_flags", "pair_overlap", "any_busy"):
        assert (o2[k] == o[k]).all(), k
    ops = o["op_nkern"] > 0
    assert (o2["op_first"][ops] == o["op_first"][ops] + d).all()
    assert (o2["gap_begin"] == o["gap_begin"] + d).all() and (o2["gap_end"] == o["gap_end"] + d).all()


@pytest.fixture(scope="module")
def cfg3():
    tr = synth.config3(n_procs=3, n_steps=20, n_edges=400)
    return tr, oracle.analyze(tr.columns(), tr.params)


def test_clock_offset_shift_changes_nothing(cfg3):
    tr, (code, o) = cfg3
    rng = np.random.default_rng(3)
    delta = rng.integers(-10**6, 10**6, tr.params["n_procs"])
    cols = tr.columns()
    cols["ts"] = cols["ts"] + delta[tr.pid]
    cols["te"] = cols["te"] + delta[tr.pid]
    p = dict(tr.params, clock_offset=tr.params["clock_offset"] + delta)
    code2, o2 = oracle.analyze(cols, p)
    assert_same((code2, o2), (code, o), p, "offset shift")
    assert (o["edge_status"] == 0).mean() > 0.9


def test_clock_shift_without_offset_changes_waits(cfg3):
    """Negative control: moving one process's clock without telling the
    analyzer must change the cross-process waits."""
    tr, (code, o) = cfg3
    cols = tr.columns()
    sel = tr.pid == 1
    cols["ts"] = np.where(sel, cols["ts"] + 7_000, cols["ts"])
    cols["te"] = np.where(sel, cols["te"] + 7_000, cols["te"])
    code2, o2 = oracle.analyze(cols, tr.params)
    e = tr.params["edges"]
    touched = ((e["prod_pid"] == 1) | (e["cons_pid"] == 1)) & (o["edge_status"] == 0) & (o2["edge_status"] == 0)
    assert touched.sum() > 10
    assert (o2["edge_wait"][touched] != o["edge_wait"][touched]).all()


def test_config3_edges_nonnegative_waits(cfg3):
    """Consumers were drawn to start at or after their producer's end."""
    tr, (code, o) = cfg3
    ok = o["edge_status"] == 0
    assert (o["edge_wait"][ok] >= 0).all()


# --------------------------------------------------------------------------- errors

def _t1():
    cols, p, g = load_golden("t1_worked_timeline.json")
    return {k: v.copy() for k, v in cols.items()}, p


@pytest.mark.parametrize("field,row,value", [
    ("kind", 3, 3), ("pid", 5, 1), ("pid", 5, -1), ("lane", 12, 2), ("lane", 4, 1), ("name", 12, 3),
    ("name", 2, 4), ("name", 6, -1), ("te", 7, 12),
    ("ts", 0, -(1 << 62)), ("te", 0, 1 << 62),
])
def test_invalid_row(field, row, value):
    cols, p = _t1()
    if field == "ts":
        cols["te"][row] = value + 5
    cols[field][row] = value
    code, o = oracle.analyze(cols, p)
    assert code == -2 and o["counters"]["first_invalid"] == row
    b = bruteforce.analyze(cols, p)
    assert b[0] == -2 and b[1]["counters"]["first_invalid"] == row


def test_invalid_smallest_row_reported():
    cols, p = _t1()
    cols["kind"][14] = 9
    cols["pid"][6] = 4
    code, o = oracle.analyze(cols, p)
    assert code == -2 and o["counters"]["first_invalid"] == 6


def test_cpu_op_corr_is_not_validated():
    cols, p = _t1()
    cols["corr"][0] = -5
    code, o = oracle.analyze(cols, p)
    assert code == 0


def _remap_ids(cols, p, f):
    """Apply the id map f (numpy, elementwise) to every launch / kernel id
    and to both ids of every edge."""
    c = {k: v.copy() for k, v in cols.items()}
    jk = c["kind"] != 0
    c["corr"][jk] = f(c["corr"][jk])
    q = dict(p)
    if p.get("edges") is not None and len(p["edges"]):
        e = p["edges"].copy()
        e["prod_corr"] = f(e["prod_corr"])
        e["cons_corr"] = f(e["cons_corr"])
        q["edges"] = e
    return c, q


ID_MAPS = {
    "negate": lambda x: -x - 1,
    "extremes": lambda x: np.where(x % 2 == 0, np.int64(-(1 << 63)) + x, np.int64((1 << 63) - 1) - x),
    "spread": lambda x: (x * np.int64(1 << 40)) ^ np.int64(0x5555),
}


@pytest.mark.parametrize("name", sorted(ID_MAPS))
def test_any_int64_correlation_id(name):
    """The correlation id is an opaque per-process identifier (any int64,
    Section 5.2): a one-to-one map of the ids, applied to the rows and the
    edges alike, leaves every result unchanged (the join and the edges only
    compare ids), whether the ids come out negative, at the int64 limits or
    spread far apart."""
    for tr in (synth.random_small(seed=71, n_rows=400, window=3000, n_procs=3, n_streams=4, n_threads=3,
                                  corr_range=60, edges=20),
               synth.random_small(seed=72, n_rows=60, window=400, n_procs=2, n_streams=2, n_threads=2,
                                  corr_range=8, edges=6)):
        cols, p = tr.columns(), tr.params
        ref = oracle.analyze(cols, p)
        c2, p2 = _remap_ids(cols, p, ID_MAPS[name])
        assert len(np.unique(c2["corr"][c2["kind"] != 0])) == len(np.unique(cols["corr"][cols["kind"] != 0]))
        got = oracle.analyze(c2, p2)
        assert_same(got, ref, p, f"ids {name}")
        if tr.n <= 100:
            bcode, b = bruteforce.analyze(c2, p2)
            assert bcode == ref[0]
            _bf_compare(c2, p2, ref[1], b, f"brute force, ids {name}")


def test_thread_limit():
    """Up to 2048 threads per process are accepted (the containment key then
    fills 64 bits at the largest process count and window)."""
    cols, p = _t1()
    p["n_threads"] = 2048
    assert oracle.analyze(cols, p)[0] == 0


@pytest.mark.parametrize("change", [
    dict(window_end=0), dict(window_end=-5), dict(window_end=(1 << 40) + 1), dict(n_procs=0),
    dict(n_procs=4097), dict(n_streams=65), dict(n_streams=0), dict(n_threads=2049), dict(n_names=0),
    dict(n_op_names=0), dict(clock_offset=np.array([1 << 62])), dict(stream_class=np.array([0, 3], np.uint8)),
    dict(window_begin=-(1 << 62), window_end=-(1 << 62) + 100),
])
def test_invalid_params(change):
    cols, p = _t1()
    p.update(change)
    code, o = oracle.analyze(cols, p)
    assert code == -1


def test_gap_capacity():
    cols, p = _t1()
    code, full = oracle.analyze(cols, p)
    for cap in (0, 1, 2, 4):
        code2, o = oracle.analyze(cols, p, gap_capacity=cap)
        assert code2 == -3 and o["counters"]["n_gaps_total"] == 5
        for k in ("gap_pid", "gap_stream", "gap_begin", "gap_end", "gap_flags"):
            assert (o[k] == full[k][:cap]).all()
        assert (o["link"] == full["link"]).all() and (o["busy"] == full["busy"]).all()
    code3, o = oracle.analyze(cols, p, gap_capacity=5)
    assert code3 == 0


def test_empty_trace():
    p = synth.empty_params(n_procs=2, n_streams=3, gap_threshold=10, flags=3)
    cols = dict(ts=np.zeros(0, np.int64), te=np.zeros(0, np.int64), corr=np.zeros(0, np.int64),
                pid=np.zeros(0, np.int32), lane=np.zeros(0, np.int32), name=np.zeros(0, np.int32),
                kind=np.zeros(0, np.uint8))
    code, o = oracle.analyze(cols, p)
    W = p["window_end"] - p["window_begin"]
    assert code == 0 and (o["busy"] == 0).all() and (o["idle"] == W).all()
    assert o["counters"]["n_gaps_total"] == 6 and (o["gap_flags"] == 3).all()
    assert (o["name_min"] == I64_MAX).all() and (o["name_max"] == I64_MIN).all()
    assert (o["any_busy"] == 0).all() and o["lat_hist"].sum() == 0


# --------------------------------------------------------------------------- GPU idle x CPU ops

def test_t1_idle_coincidence():
    """Hand-worked values of GPU idle coinciding with op names on T1, and the
    strict threshold (an idle interval as long as the threshold is dropped)."""
    cols, p, g = load_golden("t1_worked_timeline.json")
    exp = g["expect_waits"]
    p["flags"] = exp["flags"]
    code, o = oracle.analyze(cols, p)
    assert code == 0
    for k in ("dev_idle", "op_span", "op_idle"):
        assert o[k].tolist() == exp[k], k
    p["gap_threshold"] = 10
    code, o = oracle.analyze(cols, p)
    for k in ("dev_idle", "op_span", "op_idle"):
        assert o[k].tolist() == exp["thr10"][k], k


@pytest.mark.parametrize("seed", range(8))
def test_idle_coincidence_invariants(seed):
    """op_idle <= op_span and <= dev_idle; with threshold -1 the GPU idle is
    the window minus the time any stream is busy; an op spanning the whole
    window of every process sees all of its GPU idle."""
    tr = synth.random_small(seed=5200 + seed, n_rows=400, window=3000, n_procs=3, n_streams=4, n_threads=3,
                            corr_range=60, flags=7)
    cols, p = tr.columns(), dict(tr.params)
    code, o = oracle.analyze(cols, p)
    nop = p["n_op_names"]
    span, idle = o["op_span"].reshape(-1, nop), o["op_idle"].reshape(-1, nop)
    assert (idle <= span).all() and (idle <= o["dev_idle"][:, None]).all()
    p["gap_threshold"] = -1
    code, o = oracle.analyze(cols, p)
    W = p["window_end"] - p["window_begin"]
    assert (o["dev_idle"] == W - o["any_busy"]).all()
    # one more op per process covering the window, with its own name
    P = p["n_procs"]
    off = p["clock_offset"] if p["clock_offset"] is not None else np.zeros(P, np.int64)
    extra = dict(kind=np.zeros(P, np.uint8), pid=np.arange(P, dtype=np.int32), lane=np.zeros(P, np.int32),
                 ts=(p["window_begin"] + off).astype(np.int64), te=(p["window_end"] + off).astype(np.int64),
                 corr=np.zeros(P, np.int64), name=np.full(P, nop, np.int32))
    c2 = {k: np.concatenate([cols[k], extra[k]]) for k in cols}
    p2 = dict(p, n_op_names=nop + 1, gap_threshold=int(tr.params["gap_threshold"]))
    code, o2 = oracle.analyze(c2, p2)
    whole = o2["op_idle"].reshape(-1, nop + 1)[:, nop]
    assert (whole == o2["dev_idle"]).all()
    assert (o2["op_span"].reshape(-1, nop + 1)[:, nop] == W).all()


def test_idle_coincidence_name_limit():
    cols, p = _t1()
    p["flags"] = 7
    p["n_op_names"] = 2048
    assert oracle.analyze(cols, p)[0] == 0
    p["n_op_names"] = 2049
    assert oracle.analyze(cols, p)[0] == -1


# --------------------------------------------------------------------------- operator efficiency

def pa_trace(T):
    """One op, one launch and one kernel of T ns: T_op = T."""
    g = load_golden_raw("pa_sol_case.json")
    rows = [(0, 0, 0, 0, T + 2000, 0, 0), (1, 0, 0, 100, 200, 7, 0), (2, 0, 0, 1000, 1000 + T, 7, 0)]
    a = np.array(rows, dtype=np.int64)
    cols = dict(kind=a[:, 0].astype(np.uint8), pid=a[:, 1].astype(np.int32), lane=a[:, 2].astype(np.int32),
                ts=a[:, 3], te=a[:, 4], corr=a[:, 5], name=a[:, 6].astype(np.int32),
                flops=np.array([g["flops"], 0, 0], np.int64), bytes=np.array([g["bytes"], 0, 0], np.int64))
    p = synth.empty_params(window_begin=0, window_end=2 * 10**9, gap_threshold=0, flags=1 | 8,
                           peak_flops=g["peak_flops"], peak_bytes=g["peak_bytes"],
                           ref_sol_ppm=np.array([g["ref_sol_ppm"]], np.int64))
    return cols, p, g


def test_pa_case_arithmetic():
    """The printed PagedAttention figures: SOL is the larger of MFU and MBU,
    it scales with 1/T_op (a 60.9% cut takes 7.32% to 18.7%, +155%), and the
    recoverable time against a 17% reference."""
    check_pa_case()


def check_pa_case(lib=None):
    res = {}
    for phase in ("before", "after"):
        cols, p, g = pa_trace(load_golden_raw("pa_sol_case.json")[phase]["T_op"])
        code, o = oracle.analyze(cols, p, lib=lib)
        assert code == 0
        e = g[phase]
        assert [int(o["op_mfu"][0]), int(o["op_mbu"][0]), int(o["op_sol"][0])] == [e["mfu"], e["mbu"], e["sol"]]
        assert int(o["opn_hot"][0]) == e["hot"] and int(o["opn_sol"][0]) == e["sol"]
        assert int(o["opn_time"][0]) == e["T_op"]
        assert o["op_sol"][1:].tolist() == [oracle.UNWRITTEN_I64] * 2  # launch and kernel rows
        res[phase] = e["sol"]
    assert round(res["before"] / 1e4, 1) == 7.3 and round(res["after"] / 1e4, 1) == 18.7
    assert int(100 * (res["after"] / res["before"] - 1)) == 155


def test_sol_unmeasured_and_invariants():
    """An op without kernels, or whose kernels span no time, is unmeasured
    (-1); SOL is the larger of MFU and MBU; per-name sums cover the measured
    ops only; Hotness never exceeds the measured time."""
    tr = synth.config0()
    cols, p = synth.add_op_costs(tr.columns(), tr.params, 3)
    code, o = oracle.analyze(cols, p)
    assert code == 0
    ops = np.flatnonzero((cols["kind"] == 0) & (o["link"] != -2))
    meas = ops[o["op_nkern"][ops] > 0]
    meas = meas[o["op_last"][meas] > o["op_first"][meas]]
    un = np.setdiff1d(ops, meas)
    assert len(un) and (o["op_sol"][un] == -1).all() and (o["op_mfu"][un] == -1).all()
    assert (o["op_sol"][meas] == np.maximum(o["op_mfu"][meas], o["op_mbu"][meas])).all()
    T = o["op_last"][meas] - o["op_first"][meas]
    nm = cols["name"][meas]
    assert (np.bincount(nm, weights=T, minlength=p["n_op_names"]).astype(np.int64) == o["opn_time"]).all()
    assert (o["opn_hot"] <= o["opn_time"]).all() and (o["opn_hot"] >= 0).all()


@pytest.mark.parametrize("change", ["no containment", "zero peak", "negative reference", "negative flops"])
def test_sol_errors(change):
    cols, p, g = pa_trace(10**9)
    if change == "no containment":
        p["flags"] = 8
    elif change == "zero peak":
        p["peak_bytes"] = 0
    elif change == "negative reference":
        p["ref_sol_ppm"] = np.array([-1], np.int64)
    else:
        cols["flops"][0] = -5
        code, o = oracle.analyze(cols, p)
        assert code == -2 and o["counters"]["first_invalid"] == 0
        return
    assert oracle.analyze(cols, p)[0] == -1


# --------------------------------------------------------------- critical path

def crit_golden_cases():
    g = load_golden_raw("crit_path_cases.json")
    out = []
    for c in g["cases"]:
        a = np.array(c["rows"], np.int64)
        cols = dict(kind=a[:, 0].astype(np.uint8), pid=a[:, 1].astype(np.int32), lane=a[:, 2].astype(np.int32),
                    ts=a[:, 3], te=a[:, 4], corr=a[:, 5], name=a[:, 6].astype(np.int32))
        out.append((c["name"], cols, synth.empty_params(**c["params"]), c["expect"]))
    return out


def check_crit_golden(lib=None):
    for name, cols, p, exp in crit_golden_cases():
        code, o = oracle.analyze(cols, p, lib=lib)
        assert code == 0, name
        for k in ("crit_time", "crit_flags", "crit_proc"):
            assert o[k].tolist() == exp[k], (name, k)


def test_crit_path_worked_cases():
    """Two hand-worked cases: the scenario of the paper's critical-path figure
    (a synchronizing call makes the kernel it waited for part of the path;
    the other stream's kernel is off it) and nested ops with a queued kernel,
    launch and queue gaps and an op's tail after its last child."""
    check_crit_golden()


def crit_invariants(tr, o):
    cols, p = tr.columns(), tr.params
    cp = o["crit_proc"].reshape(-1, 8)
    assert (cp >= 0).all()
    assert (cp[:, 0] == cp[:, 1:].sum(axis=1)).all(), "length = sum of the parts"
    adm = o["link"] != -2
    ct, cf = o["crit_time"], o["crit_flags"]
    assert (ct[adm] >= 0).all() and (cf[adm] <= 3).all()
    assert (ct[~adm] == oracle.UNWRITTEN_I64).all() and (cf[~adm] == oracle.UNWRITTEN_U8).all()
    pid = cols["pid"]
    for q in range(p["n_procs"]):
        m = adm & (pid == q)
        assert ct[m].sum() == cp[q, 1:5].sum(), "attributed time = kernel + api + sync + op"
        assert cp[q, 0] <= int(p["window_end"]) - int(p["window_begin"])
        # time is charged only to records on the path
        assert ((ct[m] == 0) | (cf[m] != 0)).all()
        # kernels are charged their whole run exactly when their end event is on the path
        ker = m & (cols["kind"] == 2)
        run = np.minimum(cols["te"] - _off(p, pid), int(p["window_end"])) - (cols["ts"] - _off(p, pid))
        assert (ct[ker & ((cf & 2) != 0)] == run[ker & ((cf & 2) != 0)]).all()
        assert (ct[ker & ((cf & 2) == 0)] == 0).all()


def _off(p, pid):
    off = p.get("clock_offset")
    return np.zeros(len(pid), np.int64) if off is None else np.asarray(off, np.int64)[pid]


@pytest.mark.parametrize("which", ["config0", "config1_short", "config3_small"])
def test_crit_path_invariants(which):
    tr = {"config0": lambda: synth.config0(), "config1_short": lambda: synth.config1(n_steps=20),
          "config3_small": lambda: synth.config3(n_procs=3, n_steps=10, n_edges=50)}[which]()
    tr.params["flags"] = 17
    code, o = oracle.analyze(tr.columns(), tr.params)
    assert code == 0
    crit_invariants(tr, o)
    # a decode step is GPU-bound: most of the path is kernel time
    cp = o["crit_proc"].reshape(-1, 8)
    assert cp[:, 0].min() > 0


def test_crit_path_time_shift():
    """A global shift of every time and of the window leaves the path and its
    parts unchanged."""
    tr = synth.config1(n_steps=10)
    tr.params["flags"] = 17
    code, a = oracle.analyze(tr.columns(), tr.params)
    cols = dict(tr.columns())
    d = 123_456_789
    cols["ts"] = cols["ts"] + d
    cols["te"] = cols["te"] + d
    q = dict(tr.params, window_begin=int(tr.params["window_begin"]) + d, window_end=int(tr.params["window_end"]) + d)
    code2, b = oracle.analyze(cols, q)
    assert code == code2 == 0
    for k in ("crit_time", "crit_flags", "crit_proc"):
        assert a[k].tolist() == b[k].tolist(), k


def test_crit_path_needs_containment():
    name, cols, p, _ = crit_golden_cases()[0]
    assert oracle.analyze(cols, dict(p, flags=16))[0] == -1


# --------------------------------------------------------------- graph replays

def graph_golden():
    g = load_golden_raw("graph_replay_case.json")
    a = np.array(g["rows"], np.int64)
    cols = dict(kind=a[:, 0].astype(np.uint8), pid=a[:, 1].astype(np.int32), lane=a[:, 2].astype(np.int32),
                ts=a[:, 3], te=a[:, 4], corr=a[:, 5], name=a[:, 6].astype(np.int32),
                graph_node=a[:, 7].astype(np.int32))
    return cols, synth.empty_params(**g["params"]), g["expect"]


def check_graph_golden(lib=None):
    cols, p, exp = graph_golden()
    code, o = oracle.analyze(cols, p, lib=lib)
    assert code == 0
    for k in ("launch_first", "launch_last"):
        for r, v in exp[k].items():
            assert int(o[k][int(r)]) == v, (k, r)
    for k in ("gn_count", "gn_sum", "gn_min", "gn_max", "gn_offset"):
        assert o[k].tolist() == exp[k], k


def test_graph_replay_worked_case():
    """Two replays of a three-node graph, an eager kernel and an unmatched
    node kernel, worked by hand."""
    check_graph_golden()


def graph_case(seed):
    """A tiny adversarial trace with graph nodes on its kernels (-1 for about
    a quarter of them); launches owning several kernels come from repeated
    correlation ids."""
    tr = synth.random_small(seed=8000 + seed, n_rows=80, window=600, corr_range=6 + seed % 5,
                            flags=33 if seed % 2 else 35)
    rng = np.random.default_rng(seed)
    cols = dict(tr.columns())
    ng = 1 + seed % 7
    cols["graph_node"] = np.where(rng.random(tr.n) < 0.25, -1, rng.integers(0, ng, tr.n)).astype(np.int32)
    return cols, dict(tr.params, n_graph_nodes=ng)


@pytest.mark.parametrize("seed", range(40))
def test_bruteforce_graph(seed):
    cols, p = graph_case(seed)
    code, o = oracle.analyze(cols, p)
    bcode, b = bruteforce.analyze(cols, p)
    assert code == bcode
    if code == 0:
        _bf_compare(cols, p, o, b, f"graph seed {seed}")


def test_graph_replay_invariants():
    cols, p = synth.graph_replay_trace(n_steps=30, n_nodes=200)
    code, o = oracle.analyze(cols, p)
    assert code == 0
    k = (cols["kind"] == 2) & (o["link"] >= 0)
    node = cols["graph_node"]
    assert o["gn_count"].sum() == int((k & (node >= 0)).sum())
    assert (o["gn_offset"] >= 0).all()
    # every node of the graph is seen about once per replay inside the window
    assert o["gn_count"].min() >= 25
    # each joined kernel lies inside its launch's span
    L = o["link"][k]
    assert (o["launch_first"][L] <= cols["ts"][k]).all() and (o["launch_last"][L] >= cols["te"][k]).all()


@pytest.mark.parametrize("change", ["no containment", "no nodes", "node out of range"])
def test_graph_replay_errors(change):
    cols, p, _ = graph_golden()
    if change == "no containment":
        assert oracle.analyze(cols, dict(p, flags=32))[0] == -1
    elif change == "no nodes":
        assert oracle.analyze(cols, dict(p, n_graph_nodes=0))[0] == -1
    else:
        cols["graph_node"][5] = 3
        code, o = oracle.analyze(cols, p)
        assert code == -2 and o["counters"]["first_invalid"] == 5



def test_op_name_aggregates_worked():
    """Per op name, over admitted ops, of the unclipped duration: the worked
    critical-path cases hold one op of each name (prep 90 and use 80; step
    600 and layer 290)."""
    cases = crit_golden_cases()
    for (name, cols, p, _), exp in zip(cases[:2], ([90, 80], [600, 290])):
        code, o = oracle.analyze(cols, p)
        assert code == 0
        assert o["opname_count"].tolist() == [1, 1], name
        for k in ("opname_sum", "opname_min", "opname_max"):
            assert o[k].tolist() == exp, (name, k)
    # an op crossing W1 keeps its whole duration; an op outside the window is not counted
    cols, p, _ = pa_trace(10**9)
    p = dict(p, window_end=500)
    code, o = oracle.analyze(cols, p)
    assert code == 0 and o["opname_sum"].tolist() == [10**9 + 2000]
