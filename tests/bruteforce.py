"""Brute-force reference for tiny traces (test code).

An independent, deliberately naive restatement of the trace reconstruction
(Section 6.1 of the paper) used to pin the oracle: coverage is a boolean
array with one cell per nanosecond of the window, joins and containment are
all-pairs loops, and the nearest enclosing op is found by a literal backward
scan with no shortcuts.  It shares no code with the oracle or the library and
is only fast enough for windows of a few thousand ns and ~100 rows.
"""
from __future__ import annotations

import numpy as np

I64_MAX = (1 << 63) - 1
I64_MIN = -(1 << 63)
ABS = 1 << 62


def _wrap(x: int) -> int:
    x &= (1 << 64) - 1
    return x - (1 << 64) if x >= (1 << 63) else x


def _valid(k, pid, lane, name, ts, te, corr, p, flops=0, nbytes=0) -> bool:
    if k not in (0, 1, 2):
        return False
    if not 0 <= pid < p["n_procs"]:
        return False
    if k == 2:
        if not (0 <= lane < p["n_streams"] and 0 <= name < p["n_names"]):
            return False
    else:
        if not 0 <= lane < p["n_threads"]:
            return False
        if k == 0 and not 0 <= name < p["n_op_names"]:
            return False
        if k == 1 and name < 0:
            return False
        if k == 0 and p["flags"] & 8 and (flops < 0 or nbytes < 0):
            return False
    if not (-ABS < ts < ABS and -ABS < te < ABS):
        return False
    return te >= ts


def _runs(mask: np.ndarray):
    """Maximal runs of True as (start, end) index pairs."""
    out = []
    i, n = 0, len(mask)
    while i < n:
        if mask[i]:
            j = i
            while j < n and mask[j]:
                j += 1
            out.append((i, j))
            i = j
        else:
            i += 1
    return out


def analyze(cols: dict, p: dict):
    n = len(cols["ts"])
    W0, W1 = int(p["window_begin"]), int(p["window_end"])
    W = W1 - W0
    P, S, T = p["n_procs"], p["n_streams"], p["n_threads"]
    contain, overlap = bool(p["flags"] & 1), bool(p["flags"] & 2)
    rows = [dict(kind=int(cols["kind"][i]), pid=int(cols["pid"][i]), lane=int(cols["lane"][i]),
                 name=int(cols["name"][i]), ts=int(cols["ts"][i]), te=int(cols["te"][i]),
                 corr=int(cols["corr"][i])) for i in range(n)]
    for i, r in enumerate(rows):
        fb = (int(cols["flops"][i]), int(cols["bytes"][i])) if p["flags"] & 8 else (0, 0)
        bad_node = bool(p["flags"] & 32) and r["kind"] == 2 and \
            not -1 <= int(cols["graph_node"][i]) < int(p["n_graph_nodes"])
        if bad_node or not _valid(r["kind"], r["pid"], r["lane"], r["name"], r["ts"], r["te"], r["corr"], p, *fb):
            return -2, dict(counters=dict(first_invalid=i))
    off = p.get("clock_offset")
    for r in rows:
        o = 0 if off is None else int(off[r["pid"]])
        r["t0"] = r["ts"] - o
        r["t1"] = r["te"] - o
        r["in"] = W0 <= r["t0"] < W1
    cnt = dict(n_admitted_cpu=0, n_admitted_launch=0, n_admitted_kernel=0, n_outside_window=0,
               n_matched=0, n_unmatched_kernels=0, n_unmatched_launches=0, n_dup_launch_corr=0,
               n_unattributed_kernels=0, n_improper_nesting=0, n_negative_latency=0,
               n_gaps_total=0, first_invalid=-1)
    kname = ("n_admitted_cpu", "n_admitted_launch", "n_admitted_kernel")
    for r in rows:
        if r["in"]:
            cnt[kname[r["kind"]]] += 1
        else:
            cnt["n_outside_window"] += 1
    link = [-2 if not r["in"] else -1 for r in rows]
    aux = [-2 if not r["in"] else -1 for r in rows]
    ker = [i for i, r in enumerate(rows) if r["in"] and r["kind"] == 2]
    lau = [i for i, r in enumerate(rows) if r["in"] and r["kind"] == 1]
    ops = [i for i, r in enumerate(rows) if r["in"] and r["kind"] == 0]

    # coverage bitmaps, one cell per ns of [W0, W1)
    cov = np.zeros((P, S, W), bool)
    for i in ker:
        r = rows[i]
        a, b = r["t0"] - W0, min(r["t1"], W1) - W0
        if b > a:
            cov[r["pid"], r["lane"], a:b] = True
    busy = cov.sum(axis=2).reshape(-1).astype(np.int64)
    idle = W - busy
    gaps = []
    for q in range(P):
        for s in range(S):
            for a, b in _runs(~cov[q, s]):
                if b - a > p["gap_threshold"]:
                    gaps.append((q, s, W0 + a, W0 + b, (1 if a == 0 else 0) | (2 if b == W else 0)))
    cnt["n_gaps_total"] = len(gaps)

    # join: all pairs
    for l in lau:
        aux[l] = 0
    for idx, l in enumerate(lau):
        if any(rows[m]["pid"] == rows[l]["pid"] and rows[m]["corr"] == rows[l]["corr"] for m in lau[:idx]):
            cnt["n_dup_launch_corr"] += 1
    hist = [0] * 64
    for k in ker:
        cands = [l for l in lau if rows[l]["pid"] == rows[k]["pid"] and rows[l]["corr"] == rows[k]["corr"]]
        if cands:
            l = min(cands)
            link[k] = l
            aux[l] += 1
            cnt["n_matched"] += 1
            x = rows[k]["t0"] - rows[l]["t0"]
            if x < 0:
                cnt["n_negative_latency"] += 1
            hist[0 if x <= 0 else x.bit_length()] += 1
        else:
            cnt["n_unmatched_kernels"] += 1
    cnt["n_unmatched_launches"] = sum(1 for l in lau if aux[l] == 0)

    op_arrays = None
    if contain:
        order = sorted(ops, key=lambda i: (rows[i]["pid"], rows[i]["lane"], rows[i]["t0"], -rows[i]["t1"], i))
        for pos, i in enumerate(order):
            par = -1
            for j in reversed(order[:pos]):  # literal backward scan
                if (rows[j]["pid"], rows[j]["lane"]) != (rows[i]["pid"], rows[i]["lane"]):
                    break
                if rows[j]["t1"] > rows[i]["t0"]:
                    par = j
                    break
            link[i] = par
        for i in order:  # parents precede children in this order
            aux[i] = 0 if link[i] < 0 else aux[link[i]] + 1
            if link[i] >= 0 and rows[i]["t1"] > rows[link[i]]["t1"]:
                cnt["n_improper_nesting"] += 1
        for l in lau:
            t = rows[l]["t0"]
            best = -1
            for j in order:  # the last op in the order with ts' <= t and te' > t
                if (rows[j]["pid"], rows[j]["lane"]) == (rows[l]["pid"], rows[l]["lane"]) \
                        and rows[j]["t0"] <= t and rows[j]["t1"] > t:
                    best = j
            link[l] = best
        for k in ker:
            if link[k] >= 0:
                aux[k] = link[link[k]]
                if aux[k] < 0:
                    cnt["n_unattributed_kernels"] += 1
        op_arrays = {}
        for i in ops:
            sub = [k for k in ker if link[k] >= 0]
            mine = []
            for k in sub:
                a = aux[k]
                while a >= 0:
                    if a == i:
                        mine.append(k)
                        break
                    a = link[a]
            op_arrays[i] = (len(mine),
                            min((rows[k]["t0"] for k in mine), default=I64_MAX),
                            max((rows[k]["t1"] for k in mine), default=I64_MIN),
                            _wrap(sum(rows[k]["t1"] - rows[k]["t0"] for k in mine)))

    nn = p["n_names"]
    ncount = [0] * nn
    nsum = [0] * nn
    nmin = [I64_MAX] * nn
    nmax = [I64_MIN] * nn
    for k in ker:
        q = rows[k]["name"]
        d = rows[k]["t1"] - rows[k]["t0"]
        ncount[q] += 1
        nsum[q] = _wrap(nsum[q] + d)
        nmin[q] = min(nmin[q], d)
        nmax[q] = max(nmax[q], d)
    # the same over admitted ops, by op name, as lists of their durations
    opd = {q: [] for q in range(p["n_op_names"])}
    for i in ops:
        opd[rows[i]["name"]].append(rows[i]["t1"] - rows[i]["t0"])
    opname = dict(opname_count=np.array([len(v) for v in opd.values()], np.int64),
                  opname_sum=np.array([_wrap(sum(v)) for v in opd.values()], np.int64),
                  opname_min=np.array([min(v, default=I64_MAX) for v in opd.values()], np.int64),
                  opname_max=np.array([max(v, default=I64_MIN) for v in opd.values()], np.int64))

    ov = None
    if overlap:
        cls = p.get("stream_class")
        cls = [0] * S if cls is None else [int(x) for x in cls]
        pair = np.zeros((P, S, S), np.int64)
        cb = np.zeros((P, 3), np.int64)
        co = np.zeros((P, 3, 3), np.int64)
        anyb = np.zeros(P, np.int64)
        for q in range(P):
            for i in range(S):
                for j in range(S):
                    pair[q, i, j] = np.count_nonzero(cov[q, i] & cov[q, j])
            cm = [np.zeros(W, bool) for _ in range(3)]
            for s in range(S):
                cm[cls[s]] |= cov[q, s]
            for c1 in range(3):
                cb[q, c1] = cm[c1].sum()
                for c2 in range(3):
                    co[q, c1, c2] = np.count_nonzero(cm[c1] & cm[c2])
            anyb[q] = cov[q].any(axis=0).sum()
        ov = dict(pair_overlap=pair.reshape(-1), class_busy=cb.reshape(-1),
                  class_overlap=co.reshape(-1), any_busy=anyb)

    waits = None
    if p["flags"] & 4:
        # GPU idle: no stream of the process covers the ns; runs of idle ns
        # longer than the threshold count; per op name, the ns covered by any
        # of its admitted ops (clipped at W1)
        nop = p["n_op_names"]
        dev_idle = np.zeros(P, np.int64)
        span = np.zeros((P, nop), np.int64)
        oidle = np.zeros((P, nop), np.int64)
        for q in range(P):
            idle_ns = np.zeros(W, bool)
            for a, b in _runs(~cov[q].any(axis=0)):
                if b - a > p["gap_threshold"]:
                    idle_ns[a:b] = True
            dev_idle[q] = idle_ns.sum()
            for o in range(nop):
                m = np.zeros(W, bool)
                for i in ops:
                    r = rows[i]
                    if r["pid"] == q and r["name"] == o:
                        m[r["t0"] - W0:min(r["t1"], W1) - W0] = True
                span[q, o] = m.sum()
                oidle[q, o] = np.count_nonzero(m & idle_ns)
        waits = dict(dev_idle=dev_idle, op_span=span.reshape(-1), op_idle=oidle.reshape(-1))

    sol = None
    if p["flags"] & 8:
        # operator efficiency in parts per million with Python's exact
        # integers: 10^15 * count / (T_op * peak), T_op from the op's
        # inclusive kernel span; per op name over the measured ops
        nop = p["n_op_names"]
        PF, PB = int(p["peak_flops"]), int(p["peak_bytes"])
        ref = p.get("ref_sol_ppm")
        mfu, mbu, so = {}, {}, {}
        nf, nb, nt, nh = [0] * nop, [0] * nop, [0] * nop, [0] * nop
        for i in ops:
            nk, first, last, _ = op_arrays[i]
            T = last - first if nk > 0 else 0
            if T <= 0:
                mfu[i] = mbu[i] = so[i] = -1
                continue
            F, B = int(cols["flops"][i]), int(cols["bytes"][i])
            mfu[i] = min(10**15 * F // (T * PF), I64_MAX)
            mbu[i] = min(10**15 * B // (T * PB), I64_MAX)
            so[i] = max(mfu[i], mbu[i])
            o = rows[i]["name"]
            nf[o] += F
            nb[o] += B
            nt[o] += T
            r = 0 if ref is None else int(ref[o])
            if r > 0 and so[i] < r:
                nh[o] += T * (r - so[i]) // r
        nsol = []
        for o in range(nop):
            t = nt[o] % (1 << 64)
            if t == 0:
                nsol.append(-1)
            else:
                f, b2 = nf[o] % (1 << 64), nb[o] % (1 << 64)
                nsol.append(max(min(10**15 * f // (t * PF), I64_MAX), min(10**15 * b2 // (t * PB), I64_MAX)))
        sol = dict(op_mfu=mfu, op_mbu=mbu, op_sol=so, opn_flops=np.array([_wrap(x) for x in nf], np.int64),
                   opn_bytes=np.array([_wrap(x) for x in nb], np.int64),
                   opn_time=np.array([_wrap(x) for x in nt], np.int64), opn_sol=np.array(nsol, np.int64),
                   opn_hot=np.array([_wrap(x) for x in nh], np.int64))

    edges = p.get("edges")
    ew, es = [], []
    for e in ([] if edges is None else edges):
        prod = [k for k in ker if rows[k]["pid"] == int(e["prod_pid"]) and rows[k]["corr"] == int(e["prod_corr"])]
        cons = [k for k in ker if rows[k]["pid"] == int(e["cons_pid"]) and rows[k]["corr"] == int(e["cons_corr"])]
        st = (0 if prod else 1) | (0 if cons else 2)
        es.append(st)
        if st:
            ew.append(I64_MIN)
        else:
            ew.append(_wrap(min(rows[k]["t0"] for k in cons) - max(rows[k]["t1"] for k in prod)))

    crit = None
    if p["flags"] & 16 and contain:
        # critical path: every release candidate of every event is an explicit
        # edge (release time, priority, target event, category, charged row);
        # the released-by edge is the maximum by (release, priority); the
        # structures come from all-pairs scans over this brute force's own
        # join and containment
        adm = [i for i, r in enumerate(rows) if r["in"]]
        tS = {i: rows[i]["t0"] for i in adm}
        tE = {i: min(rows[i]["t1"], W1) for i in adm}

        def hkey(i):  # containment order within a thread
            r = rows[i]
            return (r["t0"], 0 if r["kind"] == 0 else 1, -r["t1"] if r["kind"] == 0 else 0, i)

        host = [i for i in adm if rows[i]["kind"] != 2]
        cands = {}
        for i in adm:
            r = rows[i]
            ce, cs = [], []
            if r["kind"] == 2:
                ce.append((tS[i], 0, (i, 0), 1, i))
                prev = [j for j in ker if rows[j]["pid"] == r["pid"] and rows[j]["lane"] == r["lane"]
                        and (rows[j]["t0"], j) < (r["t0"], i)]
                if prev:
                    j = max(prev, key=lambda j: (rows[j]["t0"], j))
                    if tE[j] <= tS[i]:
                        cs.append((tE[j], 0, (j, 1), 6, -1))
                L = link[i]
                if L >= 0:
                    if tE[L] <= tS[i]:
                        cs.append((tE[L], 1, (L, 1), 5, -1))
                    elif tS[L] <= tS[i]:
                        cs.append((tS[L], 1, (L, 0), 2, L))
            else:
                same = [j for j in host if (rows[j]["pid"], rows[j]["lane"]) == (r["pid"], r["lane"])
                        and link[j] == link[i]]
                before = [j for j in same if hkey(j) < hkey(i)]
                if r["kind"] == 1:
                    g = [k for k in ker if rows[k]["pid"] == r["pid"] and tS[i] < tE[k] < tE[i]]
                    if aux[i] == 0 and g:
                        k = max(g, key=lambda k: (tE[k], k))
                        ce.append((tE[k], 1, (k, 1), 3, i))
                    ce.append((tS[i], 0, (i, 0), 2, i))
                else:
                    kids = [j for j in host if link[j] == i]
                    if kids:
                        c = max(kids, key=hkey)
                        if tE[c] <= tE[i]:
                            ce.append((tE[c], 1, (c, 1), 4, i))
                    ce.append((tS[i], 0, (i, 0), 4, i))
                if before:
                    j = max(before, key=hkey)
                    if tE[j] <= tS[i]:
                        cs.append((tE[j], 1, (j, 1), 7, -1))
                if link[i] >= 0:
                    cs.append((tS[link[i]], 0, (link[i], 0), 4, link[i]))
            # an end event prefers its priority-1 edge when it has one
            cands[(i, 1)] = max(ce, key=lambda c: (c[1], c[0])) if ce else None
            cands[(i, 0)] = max(cs, key=lambda c: (c[0], c[1])) if cs else None
        ctime = {i: 0 for i in adm}
        cflag = {i: 0 for i in adm}
        cproc = np.zeros((P, 8), np.int64)
        for q in range(P):
            mine = [i for i in adm if rows[i]["pid"] == q]
            if not mine:
                continue
            z = max(mine, key=lambda i: (tE[i], i))
            ev_, seen = (z, 1), set()
            while True:
                assert ev_ not in seen, "a cycle"
                seen.add(ev_)
                cflag[ev_[0]] |= 2 if ev_[1] else 1
                t = tE[ev_[0]] if ev_[1] else tS[ev_[0]]
                c = cands[ev_]
                if c is None:
                    cproc[q, 0] = tE[z] - t
                    break
                tgt = c[2]
                d = t - (tE[tgt[0]] if tgt[1] else tS[tgt[0]])
                assert d >= 0
                cproc[q, c[3]] += d
                if c[4] >= 0:
                    ctime[c[4]] += d
                ev_ = tgt
        crit = dict(crit_time=ctime, crit_flags=cflag, crit_proc=cproc.reshape(-1))

    graph = None
    if p["flags"] & 32 and contain:
        # graph replays: every launch's joined kernels, all pairs
        NG = int(p["n_graph_nodes"])
        lf, ll = {}, {}
        for l in lau:
            mine = [k for k in ker if link[k] == l]
            lf[l] = min((rows[k]["t0"] for k in mine), default=I64_MAX)
            ll[l] = max((rows[k]["t1"] for k in mine), default=I64_MIN)
        gn = {k: [] for k in range(NG)}
        for k in ker:
            q = int(cols["graph_node"][k])
            if q >= 0 and link[k] >= 0:
                gn[q].append((rows[k]["t1"] - rows[k]["t0"], rows[k]["t0"] - lf[link[k]]))
        graph = dict(launch_first=lf, launch_last=ll,
                     gn_count=np.array([len(gn[q]) for q in range(NG)], np.int64),
                     gn_sum=np.array([_wrap(sum(d for d, _ in gn[q])) for q in range(NG)], np.int64),
                     gn_min=np.array([min((d for d, _ in gn[q]), default=I64_MAX) for q in range(NG)], np.int64),
                     gn_max=np.array([max((d for d, _ in gn[q]), default=I64_MIN) for q in range(NG)], np.int64),
                     gn_offset=np.array([_wrap(sum(o for _, o in gn[q])) for q in range(NG)], np.int64))

    out = dict(counters=cnt, link=np.array(link, np.int32), aux=np.array(aux, np.int32),
               busy=busy, idle=idle, gaps=gaps, lat_hist=np.array(hist, np.int64),
               name_count=np.array(ncount, np.int64), name_sum=np.array(nsum, np.int64),
               name_min=np.array(nmin, np.int64), name_max=np.array(nmax, np.int64),
               op=op_arrays, overlap=ov, waits=waits, sol=sol, crit=crit, graph=graph, opname=opname,
               edge_wait=np.array(ew, np.int64),
               edge_status=np.array(es, np.int32))
    return 0, out
