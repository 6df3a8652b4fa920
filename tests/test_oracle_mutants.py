"""Strength of the oracle's pins: each plausible mistake planted in a copy of
the oracle (a dropped term, a wrong sign, an off-by-one bound, a transposed
operand) must make at least one pin fail.  Runs on the CPU only; the mutated
copies are compiled into a temporary directory."""
from __future__ import annotations

import os
import subprocess

import numpy as np
import pytest

import bruteforce
import oracle
import test_oracle_pins as pins
from fixtures import load_golden
from paper_2609_40247_amd import synth

SRC = os.path.join(os.path.dirname(oracle.__file__), "herschel_oracle.c")

MUTANTS = [
    ("admit end inclusive", "adm[i] = (ts[i] >= W0 && ts[i] < W1);", "adm[i] = (ts[i] >= W0 && ts[i] <= W1);"),
    ("admit begin exclusive", "adm[i] = (ts[i] >= W0 && ts[i] < W1);", "adm[i] = (ts[i] > W0 && ts[i] < W1);"),
    ("no clip at W1", "kr[w].c = te[i] < W1 ? te[i] : W1;", "kr[w].c = te[i];"),
    # (keeping touching runs apart would be an equivalent mutant: the gap
    # between them is empty and never emitted)
    ("overlapping runs kept apart", "if (r > 0 && v[i].s <= v[r - 1].e) {", "if (r > 0 && v[i].s == v[r - 1].e) {"),
    ("run end not extended", "if (v[i].e > v[r - 1].e) v[r - 1].e = v[i].e;", ";"),
    ("empty kernels cover", "if (kr[q].c > kr[q].b) {", "if (kr[q].c >= kr[q].b) {"),
    ("threshold inclusive", "if (ge - gb > p->thr) {", "if (ge - gb >= p->thr) {"),
    ("gap flags swapped", "(uint8_t)((gb == W0 ? 1 : 0) | (ge == W1 ? 2 : 0))",
     "(uint8_t)((gb == W0 ? 2 : 0) | (ge == W1 ? 1 : 0))"),
    ("trailing gap dropped", "for (int64_t q = 0; q <= r; ++q) {", "for (int64_t q = 0; q < r; ++q) {"),
    ("idle sign", "out->idle[ps] = W - b;", "out->idle[ps] = b - W;"),
    ("offset sign", "ts[i] = ev->ts[i] - off;", "ts[i] = ev->ts[i] + off;"),
    ("offset on start only", "te[i] = ev->te[i] - off;", "te[i] = ev->te[i];"),
    ("zero-length rows invalid", "if (ev->te[i] < ev->ts[i]) return 0;", "if (ev->te[i] <= ev->ts[i]) return 0;"),
    ("row tie-break reversed", "if (u->row != v->row) return u->row < v->row ? -1 : 1;",
     "if (u->row != v->row) return u->row > v->row ? -1 : 1;"),
    ("idle threshold inclusive", "if (ge > gb && ge - gb > p->thr) {", "if (ge > gb && ge - gb >= p->thr) {"),
    ("GPU idle from one stream", "union_of(runs + (int64_t)pp * S, nruns + (int64_t)pp * S, S, &all);",
     "union_of(runs + (int64_t)pp * S, nruns + (int64_t)pp * S, 1, &all);"),
    ("op ranges unclipped", "int64_t e = te[i] < W1 ? te[i] : W1;", "int64_t e = te[i];"),
    ("op time intersected with busy", "runs_intersection(u, r, idle, ni);", "runs_intersection(u, r, all, nall);"),
    ("op ranges not merged", "int64_t r = merge_runs(u, w);\n        out->op_span", "int64_t r = w;\n        out->op_span"),
    ("join ignores pid", "if (lo < nl && lr[lo].a == ev->pid[i] && lr[lo].b == ev->corr[i]) {",
     "if (lo < nl && lr[lo].b == ev->corr[i]) {"),
    ("latency sign", "int64_t x = ts[i] - ts[l];", "int64_t x = ts[l] - ts[i];"),
    ("latency from launch end", "int64_t x = ts[i] - ts[l];", "int64_t x = ts[i] - te[l];"),
    ("latency bin off by one", "  return b;\n}", "  return b > 0 ? b - 1 : 0;\n}"),
    ("zero latency negative", "if (x < 0) c->n_negative_latency++;", "if (x <= 0) c->n_negative_latency++;"),
    ("duplicates not counted", "c->n_dup_launch_corr++;", ";"),
    ("unmatched launches", "if (out->aux[lr[q].row] == 0) c->n_unmatched_launches++;",
     "if (out->aux[lr[q].row] <= 1) c->n_unmatched_launches++;"),
    ("op order te ascending", "cr[w].c = -te[i];", "cr[w].c = te[i];"),
    ("parent end inclusive", "while (j >= segstart[q] && -cr[j].c <= cr[q].b) j = par[j];",
     "while (j >= segstart[q] && -cr[j].c < cr[q].b) j = par[j];"),
    ("launch excludes ops starting with it",
     "if (cr[mid].a < seg || (cr[mid].a == seg && cr[mid].b <= t))",
     "if (cr[mid].a < seg || (cr[mid].a == seg && cr[mid].b < t))"),
    ("launch end inclusive", "while (j >= 0 && -cr[j].c <= t) j = par[j];", "while (j >= 0 && -cr[j].c < t) j = par[j];"),
    ("depth not incremented", "out->aux[row] = out->aux[cr[j].row] + 1;", "out->aux[row] = out->aux[cr[j].row];"),
    ("improper inclusive", "if (te[row] > te[cr[j].row]) c->n_improper_nesting++;",
     "if (te[row] >= te[cr[j].row]) c->n_improper_nesting++;"),
    ("kernel op is launch row", "out->aux[i] = out->link[l];", "out->aux[i] = (int32_t)l;"),
    ("aggregates not inclusive", "        r = out->link[r];\n", "        r = -1;\n"),
    ("op_last from start", "if (te[i] > out->op_last[r]) out->op_last[r] = te[i];",
     "if (ts[i] > out->op_last[r]) out->op_last[r] = ts[i];"),
    ("op_last clipped", "if (te[i] > out->op_last[r]) out->op_last[r] = te[i];",
     "if ((te[i] < W1 ? te[i] : W1) > out->op_last[r]) out->op_last[r] = te[i] < W1 ? te[i] : W1;"),
    ("ksum wrong term", "out->op_ksum[r] = wrap_add(out->op_ksum[r], te[i] - ts[i]);",
     "out->op_ksum[r] = wrap_add(out->op_ksum[r], te[i] - out->op_first[r]);"),
    ("name min as max", "if (d < out->name_min[q]) out->name_min[q] = d;", "if (d > out->name_min[q]) out->name_min[q] = d;"),
    ("name duration clipped", "    int64_t d = te[i] - ts[i];\n    out->name_count",
     "    int64_t d = (te[i] < W1 ? te[i] : W1) - ts[i];\n    out->name_count"),
    ("intersection advance swapped", "if (a[i].e < b[j].e) ++i; else ++j;", "if (a[i].e < b[j].e) ++j; else ++i;"),
    ("class of wrong stream", "int sc = p->stream_class ? p->stream_class[s] : 0;",
     "int sc = p->stream_class ? p->stream_class[S - 1 - s] : 0;"),
    ("any_busy one stream", "int64_t nall = union_of(L, N, S, &all);", "int64_t nall = union_of(L, N, 1, &all);"),
    ("producer by start", "if (side == 0 && te[r] > prod_end) prod_end = te[r];",
     "if (side == 0 && ts[r] > prod_end) prod_end = ts[r];"),
    ("consumer latest", "if (side == 1 && ts[r] < cons_start) cons_start = ts[r];",
     "if (side == 1 && (cons_start == I64_MAX || ts[r] > cons_start)) cons_start = ts[r];"),
    ("wait sign", "wrap_sub(cons_start, prod_end)", "wrap_sub(prod_end, cons_start)"),
    ("SOL as the smaller", "out->op_sol[i] = out->op_mfu[i] > out->op_mbu[i]",
     "out->op_sol[i] = out->op_mfu[i] < out->op_mbu[i]"),
    ("MBU over the compute peak", "out->op_mbu[i] = ppm_of((uint64_t)ev->bytes[i], (uint64_t)T, (uint64_t)p->peak_bytes);",
     "out->op_mbu[i] = ppm_of((uint64_t)ev->bytes[i], (uint64_t)T, (uint64_t)p->peak_flops);"),
    ("T_op as kernel time", "int64_t T = out->op_nkern[i] > 0 ? wrap_sub(out->op_last[i], out->op_first[i]) : 0;",
     "int64_t T = out->op_nkern[i] > 0 ? out->op_ksum[i] : 0;"),
    ("ppm scale off by ten", "(unsigned __int128)x * 1000000000000000ull;", "(unsigned __int128)x * 100000000000000ull;"),
    ("ppm not saturated", "return q > (unsigned __int128)I64_MAX ? I64_MAX : (int64_t)q;", "return (int64_t)q;"),
    ("hotness at or above reference", "if (ref > 0 && out->op_sol[i] < ref) {", "if (ref > 0) {"),
    ("hotness over SOL", "(int64_t)(uint64_t)(x / (uint64_t)ref)", "(int64_t)(uint64_t)(x / (uint64_t)out->op_sol[i])"),
    ("name MFU dropped", "int64_t f = ppm_of((uint64_t)out->opn_flops[o], t, (uint64_t)p->peak_flops);",
     "int64_t f = 0;"),
    ("hotness overwritten", "out->opn_hot[o] = wrap_add(out->opn_hot[o], (int64_t)(uint64_t)(x / (uint64_t)ref));",
     "out->opn_hot[o] = (int64_t)(uint64_t)(x / (uint64_t)ref);"),
    ("kernel tie to the stream", "if (tE[l] <= t && tE[l] >= rel) y = l, ys = 1, rel = tE[l], cat = 5, who = -1;",
     "if (tE[l] <= t && tE[l] > rel) y = l, ys = 1, rel = tE[l], cat = 5, who = -1;"),
    ("sync gate ignored", "if (k == K_LAUNCH && gate[x] >= 0 && tE[gate[x]] < tE[x]) {",
     "if (0 && k == K_LAUNCH && gate[x] >= 0 && tE[gate[x]] < tE[x]) {"),
    ("first child as last", "if (par >= 0) lastc[par] = x; /* later children overwrite earlier */",
     "if (par >= 0 && lastc[par] < 0) lastc[par] = x;"),
    ("path ends unclipped", "tE[i] = te[i] < W1 ? te[i] : W1;", "tE[i] = te[i];"),
    ("last record by smallest row", "if (z < 0 || tE[i] > tE[z] || (tE[i] == tE[z] && i > z)) zrow[ev->pid[i]] = i;",
     "if (z < 0 || tE[i] > tE[z] || (tE[i] == tE[z] && i < z)) zrow[ev->pid[i]] = i;"),
    ("launch gap as queue gap", "y = l, ys = 1, rel = tE[l], cat = 5, who = -1;", "y = l, ys = 1, rel = tE[l], cat = 6, who = -1;"),
    ("parent released at its end", "if (par >= 0) y = par, ys = 0, rel = tS[par], cat = 4, who = par;",
     "if (par >= 0) y = par, ys = 0, rel = tE[par], cat = 4, who = par;"),
    ("api charged to the kernel", "y = l, ys = 0, rel = tS[l], cat = 2, who = l;", "y = l, ys = 0, rel = tS[l], cat = 2, who = x;"),
    ("op tail charged to the child", "y = lastc[x], ys = 1, cat = 4, who = x;", "y = lastc[x], ys = 1, cat = 4, who = lastc[x];"),
    ("replay offset from the launch", "ts[i] - out->launch_first[out->link[i]]);",
     "ts[i] - ts[out->link[i]]);"),
    ("unmatched node kernels counted",
     "if (!adm[i] || ev->kind[i] != K_KERNEL || out->link[i] < 0 || ev->graph_node[i] < 0) continue;",
     "if (!adm[i] || ev->kind[i] != K_KERNEL || ev->graph_node[i] < 0) continue;"),
    ("replay end from the start", "if (te[i] > out->launch_last[l]) out->launch_last[l] = te[i];",
     "if (ts[i] > out->launch_last[l]) out->launch_last[l] = ts[i];"),
    ("node minimum as maximum", "if (d < out->gn_min[q]) out->gn_min[q] = d;", "if (d > out->gn_min[q]) out->gn_min[q] = d;"),
    ("op-name duration clipped", "    int64_t d = te[i] - ts[i];\n    if (out->opname_count)",
     "    int64_t d = (te[i] < W1 ? te[i] : W1) - ts[i];\n    if (out->opname_count)"),
    ("op-name maximum as minimum", "if (out->opname_max && d > out->opname_max[q]) out->opname_max[q] = d;",
     "if (out->opname_max && d < out->opname_max[q]) out->opname_max[q] = d;"),
    ("edge status bits swapped", "(found[0] ? 0 : 1) | (found[1] ? 0 : 2)", "(found[0] ? 0 : 2) | (found[1] ? 0 : 1)"),
]


def _battery(lib) -> None:
    """All pins, against the library ``lib``; raises on the first failure."""
    for name in pins.GOLDEN:
        cols, p, g = load_golden(name)
        code, o = oracle.analyze(cols, p, lib=lib)
        assert code == g["expect"]["code"]
        pins._check_expect(o, cols, g["expect"])
    many_procs = [c for c in pins.BF_CASES if 4000 <= c["seed"] < 4100]
    waits = [c for c in pins.BF_CASES if c["seed"] >= 5000][::2]
    for case in pins.BF_CASES[::4] + many_procs + waits:
        tr = synth.random_small(**case)
        code, o = oracle.analyze(tr.columns(), tr.params, lib=lib)
        bcode, b = bruteforce.analyze(tr.columns(), tr.params)
        assert code == bcode
        if code == 0:
            pins._bf_compare(tr.columns(), tr.params, o, b, tr.label)
    tr = synth.config1(n_steps=12)
    code, o = oracle.analyze(tr.columns(), tr.params, lib=lib)
    pins._invariants(tr, o)
    pins._truth_check(tr, o)
    cols, p, g = load_golden("t1_worked_timeline.json")
    exp = g["expect_waits"]
    p["flags"] = exp["flags"]
    code, o = oracle.analyze(cols, p, lib=lib)
    for k in ("dev_idle", "op_span", "op_idle"):
        assert o[k].tolist() == exp[k], k
    pins.check_pa_case(lib)
    pins.check_crit_golden(lib)
    pins.check_graph_golden(lib)
    for seed in range(0, 40, 3):
        cols, p = pins.graph_case(seed)
        code, o = oracle.analyze(cols, p, lib=lib)
        bcode, b = bruteforce.analyze(cols, p)
        assert code == bcode
        if code == 0:
            pins._bf_compare(cols, p, o, b, f"graph seed {seed}")
    for case in [c for c in pins.BF_CASES if c.get("flags", 3) & 16][::3]:
        tr = synth.random_small(**case)
        code, o = oracle.analyze(tr.columns(), tr.params, lib=lib)
        bcode, b = bruteforce.analyze(tr.columns(), tr.params)
        assert code == bcode
        if code == 0:
            pins._bf_compare(tr.columns(), tr.params, o, b, tr.label)
    tr = synth.config1(n_steps=12)
    tr.params["flags"] = 17
    code, o = oracle.analyze(tr.columns(), tr.params, lib=lib)
    pins.crit_invariants(tr, o)
    for seed in pins.SOL_BF_SEEDS[::3] + [4, 5, 29]:  # 4, 5, 29: two ops of one name below its reference
        cols, p = pins.sol_case(seed)
        code, o = oracle.analyze(cols, p, lib=lib)
        bcode, b = bruteforce.analyze(cols, p)
        assert code == bcode
        if code == 0:
            pins._bf_compare(cols, p, o, b, f"sol seed {seed}")


@pytest.fixture(scope="module")
def src():
    with open(SRC) as f:
        return f.read()


def test_pristine_oracle_passes_battery():
    _battery(oracle._load())


def test_parent_scan_skip_is_exact(src, tmp_path):
    """The oracle's backward scan for the enclosing op jumps from a failing
    candidate to that candidate's parent; a literal one-by-one scan must give
    identical results (equivalent variant, not a mutant)."""
    old = "while (j >= segstart[q] && -cr[j].c <= cr[q].b) j = par[j];"
    lit = src.replace(old, "while (j >= segstart[q] && -cr[j].c <= cr[q].b) j = j - 1;", 1)
    assert lit != src
    c = tmp_path / "literal.c"
    c.write_text(lit)
    so = tmp_path / "libliteral.so"
    subprocess.run(["gcc", "-O1", "-std=c11", "-shared", "-fPIC", "-I", os.path.dirname(SRC), "-o", str(so),
                    str(c)], check=True)
    lib = oracle.load_library(str(so))
    tr = synth.config0()
    a = oracle.analyze(tr.columns(), tr.params, lib=lib)
    b = oracle.analyze(tr.columns(), tr.params)
    assert (a[1]["link"] == b[1]["link"]).all() and (a[1]["aux"] == b[1]["aux"]).all()
    for case in pins.BF_CASES[:60]:
        t = synth.random_small(**case)
        a = oracle.analyze(t.columns(), t.params, lib=lib)
        b = oracle.analyze(t.columns(), t.params)
        if a[0] == 0:
            assert (a[1]["link"] == b[1]["link"]).all() and (a[1]["aux"] == b[1]["aux"]).all()


@pytest.mark.parametrize("label,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(label, old, new, src, tmp_path):
    assert src.count(old) >= 1, f"mutation site not found: {label}"
    mutated = src.replace(old, new, 1)
    c = tmp_path / "mutant.c"
    c.write_text(mutated)
    so = tmp_path / "libmutant.so"
    hdr = os.path.dirname(SRC)
    subprocess.run(["gcc", "-O1", "-std=c11", "-shared", "-fPIC", "-I", hdr, "-o", str(so), str(c)], check=True)
    lib = oracle.load_library(str(so))
    with pytest.raises((AssertionError, IndexError, ValueError)):
        _battery(lib)
