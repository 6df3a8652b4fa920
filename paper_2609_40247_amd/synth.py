"""Seeded synthetic profiling windows (inputs only; no analysis arithmetic).

The paper's workloads are production inference services whose traces are not
available.  These generators stand in for them with the record kinds of
Section 5.2 (CPU operator ranges, launch-API intervals, kernel records linked
by correlation id) at the scale of the paper's collection windows
(Section 5.3, "Bounded collection window": typically 30 s, hundreds of
inference steps).

The recipe is kernel-timeline first, so that the drawn quantities are known
exactly (``Trace.truth``):

* per (step, stream) queue: ``start = previous end + rint(Exp(gap_mean))``,
  plus, with probability ``stall_p``, a stall drawn uniformly from
  ``stall_ns``; ``dur = max(1, rint(LogNormal(ln median, sigma)))``;
* steps begin every ``period`` ns, or when the previous step ends if later;
* each kernel's launch starts ``rint(Exp(lat_mean))`` before the kernel and
  lasts U[1000, 4000] ns; correlation ids increase in launch order per process;
* kernel names follow a Zipf law over ``n_names`` ids;
* kernel records are dropped independently after the truth is recorded;
* CPU operators form a properly nested forest over each thread's sorted
  launch start points: one root per step (or per block of launches), contiguous
  child groups below it, boundaries placed strictly between neighbouring launch
  points, about 2% of launches outside every op, and extra leaf ops that launch
  nothing to reach the requested operator count;
* rows are emitted in "delivery order": per (process, kind) sorted by end
  time, cut into blocks of 4096 rows, blocks ordered by their last end time.

All draws come from ``numpy.random.Generator(PCG64(seed))``.
"""
from __future__ import annotations

import dataclasses
import math

import os

import numpy as np

CPU_OP, LAUNCH, KERNEL = 0, 1, 2
US = 1_000
MS = 1_000_000
S = 1_000_000_000
EPOCH = 1_765_000_000 * S  # window base: an epoch-like int64 ns timestamp

EDGE_DTYPE = np.dtype(
    [("prod_pid", "<i4"), ("cons_pid", "<i4"), ("prod_corr", "<i8"), ("cons_corr", "<i8")],
    align=True,
)
assert EDGE_DTYPE.itemsize == 24


@dataclasses.dataclass
class Trace:
    ts: np.ndarray
    te: np.ndarray
    corr: np.ndarray
    pid: np.ndarray
    lane: np.ndarray
    name: np.ndarray
    kind: np.ndarray
    params: dict
    truth: dict = dataclasses.field(default_factory=dict)
    label: str = ""

    @property
    def n(self) -> int:
        return int(self.ts.shape[0])

    def columns(self) -> dict:
        return {k: getattr(self, k) for k in ("ts", "te", "corr", "pid", "lane", "name", "kind")}

    def take(self, order: np.ndarray) -> "Trace":
        """The same records in another row order (metamorphic tests)."""
        cols = {k: v[order] for k, v in self.columns().items()}
        return Trace(params=dict(self.params), truth={}, label=self.label + "/perm", **cols)


def empty_params(**kw) -> dict:
    p = dict(
        window_begin=EPOCH, window_end=EPOCH + 10 * S, gap_threshold=0,
        n_procs=1, n_streams=1, n_threads=1, n_names=1, n_op_names=1,
        clock_offset=None, stream_class=None, edges=np.zeros(0, EDGE_DTYPE), flags=3,
    )
    p.update(kw)
    return p


def _zipf(rng, n_names: int, s: float, size: int) -> np.ndarray:
    k = np.arange(1, n_names + 1, dtype=np.float64)
    cdf = np.cumsum(k ** -s)
    cdf /= cdf[-1]
    return np.minimum(np.searchsorted(cdf, rng.random(size), side="right"), n_names - 1).astype(np.int32)


def _lognormal_ns(rng, median_ns: float, sigma: float, size: int) -> np.ndarray:
    return np.maximum(1, np.rint(rng.lognormal(math.log(median_ns), sigma, size))).astype(np.int64)


def _gaps(rng, size: int, gap_mean: float, stall_p: float, stall_ns) -> tuple[np.ndarray, np.ndarray]:
    g = np.rint(rng.exponential(gap_mean, size)).astype(np.int64)
    stall = rng.random(size) < stall_p
    g[stall] += rng.integers(stall_ns[0], stall_ns[1] + 1, int(stall.sum()))
    return g, stall


def _group_cumsum(values: np.ndarray, group: np.ndarray) -> np.ndarray:
    """Inclusive cumulative sum restarting at every change of ``group``
    (``group`` must be sorted)."""
    cs = np.cumsum(values)
    starts = np.flatnonzero(np.r_[True, group[1:] != group[:-1]])
    base = np.repeat(cs[starts] - values[starts], np.diff(np.r_[starts, len(values)]))
    return cs - base


def _phase_kernels(rng, *, kernels_per_step, period, t0, streams, stream_p, median, sigma,
                   gap_mean, stall_p, stall_ns) -> dict:
    """Kernel timeline of one phase (a sequence of steps) on its streams."""
    kps = np.asarray(kernels_per_step, dtype=np.int64)
    n_steps = len(kps)
    k = int(kps.sum())
    step = np.repeat(np.arange(n_steps, dtype=np.int64), kps)
    stream = rng.choice(np.asarray(streams, dtype=np.int32), size=k, p=stream_p)
    dur = _lognormal_ns(rng, median, sigma, k)
    gap, stall = _gaps(rng, k, gap_mean, stall_p, stall_ns)
    # queue order within (step, stream): the draw order
    order = np.lexsort((np.arange(k), stream, step))
    grp = step[order] * 1024 + stream[order]
    rel_end_sorted = _group_cumsum(gap[order] + dur[order], grp)
    rel_end = np.empty(k, np.int64)
    rel_end[order] = rel_end_sorted
    rel_start = rel_end - dur
    step_len = np.zeros(n_steps, np.int64)
    np.maximum.at(step_len, step, rel_end)
    # s_i = max(t0 + i*period, s_{i-1} + len_{i-1})
    d = np.r_[0, np.cumsum(step_len)[:-1]]
    s = np.maximum.accumulate(t0 + np.arange(n_steps, dtype=np.int64) * period - d) + d
    start = s[step] + rel_start
    first_in_queue = np.zeros(k, bool)
    first_in_queue[order[np.r_[True, grp[1:] != grp[:-1]]]] = True
    return dict(start=start, end=start + dur, stream=stream, step=step, gap=gap, stall=stall,
                dur=dur, first_in_queue=first_in_queue)


def _op_forest(rng, points: np.ndarray, root_cut: np.ndarray, *, depth: int, level_p,
               orphan_frac: float, n_ops_target: int | None, min_sep: int = 8):
    """CPU operator ranges over sorted launch start points.

    ``root_cut[i]`` marks a root boundary between point i and i+1.  Returns
    (ts, te, depth) of the ops.  Nesting is proper: parents' margins are
    wider than their children's, siblings are separated between points."""
    L = len(points)
    if L == 0:
        return np.zeros(0, np.int64), np.zeros(0, np.int64), np.zeros(0, np.int32)
    gapr = np.r_[np.diff(points), 10_000].astype(np.int64)  # gap to the right of point i
    gapl = np.r_[10_000, np.diff(points)].astype(np.int64)
    lam = np.full(L - 1, depth, np.int64)  # level of the cut between i and i+1 (depth = none)
    u = rng.random(L - 1)
    cum = np.cumsum(level_p)  # P(lambda <= d) for d = 1..depth-1
    for d in range(depth - 1, 0, -1):
        lam[u < cum[d - 1]] = d
    lam[gapr[:-1] < min_sep] = depth
    lam[root_cut[:-1]] = 0
    # orphans: the first orphan_frac of each root group lies outside every op
    roots = np.flatnonzero(np.r_[True, lam == 0])
    root_len = np.diff(np.r_[roots, L])
    n_orph = np.floor(root_len * orphan_frac + rng.random(len(roots))).astype(np.int64)
    n_orph = np.minimum(n_orph, root_len - 1)
    orphan = np.zeros(L, bool)
    for a, m in zip(roots[n_orph > 0], n_orph[n_orph > 0]):
        orphan[a:a + m] = True
        lam[a + m - 1] = 0
    ts_l, te_l, dep_l = [], [], []
    for d in range(depth):
        f = 0.4 * (depth - d) / depth
        cuts = np.flatnonzero(lam <= d)
        a = np.r_[0, cuts + 1]
        b = np.r_[cuts, L - 1]
        keep = ~orphan[a]
        a, b = a[keep], b[keep]
        ts_l.append(points[a] - np.floor(gapl[a] * f).astype(np.int64))
        te_l.append(points[b] + 1 + np.floor((gapr[b] - 1) * f).astype(np.int64))
        dep_l.append(np.full(len(a), d, np.int32))
    ts = np.concatenate(ts_l)
    te = np.concatenate(te_l)
    dep = np.concatenate(dep_l)
    if n_ops_target is not None and n_ops_target > len(ts):
        # leaf ops that launch nothing, in the middle of a gap between two
        # launch points of the same root group (clear of every op boundary)
        ok = np.flatnonzero((lam > 0) & (gapr[:-1] >= 40) & ~orphan[:-1] & ~orphan[1:])
        m = min(n_ops_target - len(ts), len(ok))
        pick = np.sort(rng.choice(ok, size=m, replace=False))
        g = gapr[pick]
        ts = np.r_[ts, points[pick] + np.ceil(g * 0.42).astype(np.int64)]
        te = np.r_[te, points[pick] + np.floor(g * 0.58).astype(np.int64)]
        dep = np.r_[dep, np.full(m, depth, np.int32)]
    return ts, te, dep


def _delivery_order(rng, te: np.ndarray, stream_key: np.ndarray, block: int = 4096) -> np.ndarray:
    """Rows per stream_key (process, kind) sorted by end time, cut into blocks,
    blocks ordered by their last end time."""
    order = np.lexsort((te, stream_key))
    key_sorted = stream_key[order]
    heads = np.flatnonzero(np.r_[True, key_sorted[1:] != key_sorted[:-1]])
    pos_in_key = np.arange(len(order)) - np.repeat(heads, np.diff(np.r_[heads, len(order)]))
    blk_id = np.cumsum(np.r_[True, (key_sorted[1:] != key_sorted[:-1]) | (pos_in_key[1:] % block == 0)]) - 1
    blk_last_te = np.zeros(blk_id[-1] + 1 if len(blk_id) else 0, np.int64)
    if len(order):
        np.maximum.at(blk_last_te, blk_id, te[order])
    blk_rank = np.argsort(blk_last_te, kind="stable")
    rank_of = np.empty_like(blk_rank)
    rank_of[blk_rank] = np.arange(len(blk_rank))
    final = np.lexsort((np.arange(len(order)), rank_of[blk_id]))
    return order[final]


def _process(rng, *, phases, n_threads, drop_p, lat_mean, n_names, zipf_s, n_op_names,
             depth, level_p, orphan_frac, ops_per_launch, corr_base, block_roots=None):
    """One process: kernels of all phases, their launches, CPU ops."""
    ks = [ph["kern"] for ph in phases]
    start = np.concatenate([k["start"] for k in ks])
    end = np.concatenate([k["end"] for k in ks])
    stream = np.concatenate([k["stream"] for k in ks])
    thread = np.concatenate([np.full(len(k["start"]), ph["thread"], np.int32) for k, ph in zip(ks, phases)])
    step = np.concatenate([k["step"] + 10_000_000 * i for i, k in enumerate(ks)])
    gap = np.concatenate([k["gap"] for k in ks])
    first_q = np.concatenate([k["first_in_queue"] for k in ks])
    K = len(start)
    name = _zipf(rng, n_names, zipf_s, K)
    lat = np.rint(rng.exponential(lat_mean, K)).astype(np.int64)
    l_ts = start - lat
    l_te = l_ts + rng.integers(1000, 4001, K)
    # correlation ids increase in launch order (ties by draw order)
    lorder = np.lexsort((np.arange(K), l_ts))
    corr = np.empty(K, np.int64)
    corr[lorder] = corr_base + np.cumsum(rng.integers(1, 4, K))
    dropped = rng.random(K) < drop_p
    api = np.where(rng.random(K) < 0.05, 1, 0).astype(np.int32)
    # CPU ops per thread over the thread's sorted launch points
    o_ts, o_te, o_thr, o_dep = [], [], [], []
    for t in range(n_threads):
        sel = np.flatnonzero(thread == t)
        if len(sel) == 0:
            continue
        srt = sel[np.lexsort((sel, l_ts[sel]))]
        pts = l_ts[srt]
        if block_roots:
            root_cut = (np.arange(len(srt)) % block_roots) == block_roots - 1
        else:
            root_cut = np.r_[step[srt][1:] != step[srt][:-1], True]
        target = int(round(len(srt) * ops_per_launch)) if ops_per_launch else None
        a, b, dd = _op_forest(rng, pts, root_cut, depth=depth, level_p=level_p,
                              orphan_frac=orphan_frac, n_ops_target=target)
        o_ts.append(a); o_te.append(b); o_dep.append(dd)
        o_thr.append(np.full(len(a), t, np.int32))
    o_ts = np.concatenate(o_ts) if o_ts else np.zeros(0, np.int64)
    o_te = np.concatenate(o_te) if o_te else np.zeros(0, np.int64)
    o_thr = np.concatenate(o_thr) if o_thr else np.zeros(0, np.int32)
    o_name = _zipf(rng, n_op_names, 1.1, len(o_ts))
    return dict(start=start, end=end, stream=stream, thread=thread, name=name, lat=lat,
                l_ts=l_ts, l_te=l_te, corr=corr, dropped=dropped, api=api, gap=gap,
                first_in_queue=first_q, o_ts=o_ts, o_te=o_te, o_thr=o_thr, o_name=o_name)


def _assemble(rng, procs, offsets, params, label, shuffle=False) -> Trace:
    cols = {k: [] for k in ("ts", "te", "corr", "pid", "lane", "name", "kind")}
    truth_rows = []
    for p, (pr, off) in enumerate(zip(procs, offsets)):
        keep = ~pr["dropped"]
        K = int(keep.sum())
        L = len(pr["l_ts"])
        C = len(pr["o_ts"])
        cols["ts"] += [pr["o_ts"] + off, pr["l_ts"] + off, pr["start"][keep] + off]
        cols["te"] += [pr["o_te"] + off, pr["l_te"] + off, pr["end"][keep] + off]
        cols["corr"] += [np.zeros(C, np.int64), pr["corr"], pr["corr"][keep]]
        cols["pid"] += [np.full(C + L + K, p, np.int32)]
        cols["lane"] += [pr["o_thr"], pr["thread"], pr["stream"][keep]]
        cols["name"] += [pr["o_name"], pr["api"], pr["name"][keep]]
        cols["kind"] += [np.full(C, CPU_OP, np.uint8), np.full(L, LAUNCH, np.uint8),
                         np.full(K, KERNEL, np.uint8)]
        truth_rows.append((C, L, K))
    arr = {k: np.concatenate(v) for k, v in cols.items()}
    arr["ts"] = arr["ts"].astype(np.int64)
    arr["te"] = arr["te"].astype(np.int64)
    arr["lane"] = arr["lane"].astype(np.int32)
    arr["name"] = arr["name"].astype(np.int32)
    n = len(arr["ts"])
    if shuffle:
        order = rng.permutation(n)
    else:
        key = arr["pid"].astype(np.int64) * 3 + arr["kind"]
        order = _delivery_order(rng, arr["te"], key)
    arr = {k: np.ascontiguousarray(v[order]) for k, v in arr.items()}
    inv = np.empty(n, np.int64)
    inv[order] = np.arange(n)
    return Trace(params=params, label=label, truth=dict(procs=procs, offsets=offsets,
                 counts=truth_rows, row_of=inv), **arr)


DECODE_LEVELS_4 = (1 / 50, 1 / 6 - 1 / 50, 1 / 1.5 - 1 / 6)  # P(cut at level 1, 2, 3)
LEVELS_3 = (1 / 10, 1 / 1.5 - 1 / 10)


def _decode_process(rng, *, n_steps_kernels, period, t0, n_streams, corr_base, drop_p,
                    n_names=2000, median=6 * US, sigma=1.2):
    kern = _phase_kernels(rng, kernels_per_step=n_steps_kernels, period=period, t0=t0,
                          streams=list(range(n_streams)), stream_p=None, median=median, sigma=sigma,
                          gap_mean=3 * US, stall_p=0.01, stall_ns=(200 * US, 5 * MS))
    return _process(rng, phases=[dict(kern=kern, thread=0)], n_threads=1, drop_p=drop_p,
                    lat_mean=5 * US, n_names=n_names, zipf_s=1.1, n_op_names=100, depth=4,
                    level_p=DECODE_LEVELS_4, orphan_frac=0.02, ops_per_launch=1.0,
                    corr_base=corr_base)


def config0(seed: int = 0, shuffle: bool = False) -> Trace:
    """Tiny trace: 1 process, 2 streams, 10 s window, 20k kernels (2% dropped),
    20k launches, exactly 20k CPU ops nested up to depth 3, 200 Zipf(1.1)
    names, durations LogNormal(median 8 us, sigma 1.0), threshold 50 us."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w0 = EPOCH
    kern = _phase_kernels(rng, kernels_per_step=[20_000], period=10 * S, t0=w0 - 100 * US,
                          streams=[0, 1], stream_p=None, median=8 * US, sigma=1.0,
                          gap_mean=3 * US, stall_p=0.01, stall_ns=(200 * US, 5 * MS))
    pr = _process(rng, phases=[dict(kern=kern, thread=0)], n_threads=1, drop_p=0.02,
                  lat_mean=5 * US, n_names=200, zipf_s=1.1, n_op_names=100, depth=3,
                  level_p=LEVELS_3, orphan_frac=0.02, ops_per_launch=1.0,
                  corr_base=rng.integers(0, 1 << 20), block_roots=100)
    params = empty_params(window_begin=w0, window_end=w0 + 10 * S, gap_threshold=50 * US,
                          n_procs=1, n_streams=2, n_threads=1, n_names=200, n_op_names=100)
    return _assemble(rng, [pr], [0], params, "config0", shuffle)


def config1(seed: int = 1, shuffle: bool = False, n_steps: int = 1000, clock_offset: int = 0) -> Trace:
    """Decode-step trace: 1 process, 4 streams, 30 s window, steps of 30 ms
    with 1,000 kernels each (about 1M kernel records), matching launches and
    CPU ops nested up to depth 4, 2,000 Zipf(1.1) names, LogNormal(6 us, 1.2),
    1% dropped, threshold 20 us.  One extra step straddles W0 and the last one
    crosses W1, so both window edges are exercised."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w0 = EPOCH
    period = 30 * MS
    W = n_steps * period
    pr = _decode_process(rng, n_steps_kernels=[1000] * (n_steps + 1), period=period,
                         t0=w0 - 5 * MS, n_streams=4, corr_base=int(rng.integers(0, 1 << 20)),
                         drop_p=0.01)
    params = empty_params(window_begin=w0, window_end=w0 + W, gap_threshold=20 * US, n_procs=1,
                          n_streams=4, n_threads=1, n_names=2000, n_op_names=100)
    tr = _assemble(rng, [pr], [clock_offset], params, "config1", shuffle)
    if clock_offset:
        tr.params["clock_offset"] = np.array([clock_offset], np.int64)
    return tr


def config2(seed: int = 2, shuffle: bool = False, scale: float = 1.0) -> Trace:
    """Mixed prefill/decode trace: 1 process, 8 streams (0-1 decode compute,
    2-3 prefill compute, 4-5 comm, 6-7 copy), 30 s window, prefill steps of
    200 ms with about 3,459 kernels (LogNormal(40 us, 1.5)) running alongside
    decode steps of 30 ms with about 1,153 kernels, 30% of kernels on comm/copy
    streams, each placed to overlap a running compute kernel with probability
    0.6.  5.0M rows at scale 1."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w0 = EPOCH
    f = 1.153
    n_dec = max(1, int(round(1000 * scale)))
    n_pre = max(1, int(round(150 * scale)))
    W = 30 * S if scale == 1.0 else n_dec * 30 * MS
    kps_dec = [int(round(1000 * f))] * (n_dec + 1)
    kps_pre = [int(round(3000 * f))] * (n_pre + 1)
    phases = []
    for kps, period, comp, med, sig, thread in ((kps_dec, 30 * MS, [0, 1], 6 * US, 1.2, 0),
                                                (kps_pre, 200 * MS, [2, 3], 40 * US, 1.5, 1)):
        kern = _phase_kernels(rng, kernels_per_step=kps, period=period, t0=w0 - 5 * MS,
                              streams=comp + [4, 5, 6, 7],
                              stream_p=[0.35, 0.35, 0.075, 0.075, 0.075, 0.075],
                              median=med, sigma=sig, gap_mean=3 * US, stall_p=0.01,
                              stall_ns=(200 * US, 5 * MS))
        # comm/copy kernels: with probability 0.6 moved to start inside the
        # nearest preceding compute kernel of the same step
        side = kern["stream"] >= 4
        comp_idx = np.flatnonzero(~side)
        cs = kern["start"][comp_idx]
        cord = np.argsort(cs, kind="stable")
        sidx = np.flatnonzero(side & (rng.random(len(side)) < 0.6))
        pos = np.searchsorted(cs[cord], kern["start"][sidx], side="right") - 1
        ok = pos >= 0
        host = comp_idx[cord[pos[ok]]]
        sidx = sidx[ok]
        same = kern["step"][host] == kern["step"][sidx]
        sidx, host = sidx[same], host[same]
        kern["start"][sidx] = kern["start"][host] + np.floor(
            rng.random(len(sidx)) * kern["dur"][host]).astype(np.int64)
        # keep each side stream a queue: a kernel never starts before the
        # previous kernel on its stream ends
        order = np.lexsort((kern["start"], kern["stream"]))
        st = kern["stream"][order]
        s0 = kern["start"][order]
        d0 = kern["dur"][order]
        newst = s0.copy()
        for sid in (4, 5, 6, 7):
            m = np.flatnonzero(st == sid)
            if len(m) == 0:
                continue
            a = s0[m]
            dd = d0[m]
            # start_i = max(a_i, start_{i-1} + d_{i-1}) via the max-plus prefix form
            D = np.r_[0, np.cumsum(dd)[:-1]]
            newst[m] = np.maximum.accumulate(a - D) + D
        kern["start"][order] = newst
        kern["end"] = kern["start"] + kern["dur"]
        phases.append(dict(kern=kern, thread=thread))
    pr = _process(rng, phases=phases, n_threads=2, drop_p=0.01, lat_mean=5 * US, n_names=2000,
                  zipf_s=1.1, n_op_names=100, depth=4, level_p=DECODE_LEVELS_4,
                  orphan_frac=0.02, ops_per_launch=1.0, corr_base=int(rng.integers(0, 1 << 20)))
    params = empty_params(window_begin=w0, window_end=w0 + W, gap_threshold=20 * US, n_procs=1,
                          n_streams=8, n_threads=2, n_names=2000, n_op_names=100,
                          stream_class=np.array([0, 0, 0, 0, 1, 1, 2, 2], np.uint8))
    return _assemble(rng, [pr], [0], params, "config2", shuffle)


def config3(seed: int = 1000, shuffle: bool = False, n_procs: int = 8, n_steps: int = 1000,
            n_edges: int = 20_000) -> Trace:
    """Node-level trace: n_procs processes, each as config 1 with its own seed
    and a clock offset uniform in +-50 us added to all its raw timestamps
    (supplied in params), plus n_edges dependency edges: producer = a random
    kernel of process p, consumer = the first kernel of another process q that
    starts at or after the producer's end (corrected clock)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w0 = EPOCH
    period = 30 * MS
    procs, offs = [], []
    for p in range(n_procs):
        prng = np.random.Generator(np.random.PCG64(seed + 1 + p))
        procs.append(_decode_process(prng, n_steps_kernels=[1000] * (n_steps + 1), period=period,
                                     t0=w0 - 5 * MS, n_streams=4,
                                     corr_base=(p << 40) + int(prng.integers(0, 1 << 20)),
                                     drop_p=0.01))
        offs.append(int(rng.integers(-50 * US, 50 * US + 1)))
    edges = np.zeros(n_edges, EDGE_DTYPE)
    pp = rng.integers(0, n_procs, n_edges)
    qq = (pp + rng.integers(1, n_procs, n_edges)) % n_procs
    for q in range(n_procs):
        order = np.argsort(procs[q]["start"], kind="stable")
        procs[q]["_sorted_start"] = procs[q]["start"][order]
        procs[q]["_sorted_idx"] = order
    for e in range(n_edges):
        P = procs[pp[e]]
        k = int(rng.integers(0, len(P["start"])))
        Q = procs[qq[e]]
        j = int(np.searchsorted(Q["_sorted_start"], P["end"][k], side="left"))
        j = min(j, len(Q["_sorted_start"]) - 1)
        c = Q["_sorted_idx"][j]
        edges[e] = (pp[e], qq[e], P["corr"][k], Q["corr"][c])
    for P in procs:
        del P["_sorted_start"], P["_sorted_idx"]
    params = empty_params(window_begin=w0, window_end=w0 + n_steps * period, gap_threshold=20 * US,
                          n_procs=n_procs, n_streams=4, n_threads=1, n_names=2000, n_op_names=100,
                          clock_offset=np.array(offs, np.int64), edges=edges)
    return _assemble(rng, procs, offs, params, "config3", shuffle)


def config4_trace(t: int, kernels: int | None = None) -> Trace:
    """Trace t of the 256-trace batch: config 1 with L_t ~ U_int[200k, 2M]
    kernel records and a window of ceil(L_t / 1000) * 30 ms (2M kernels cannot
    fit in 30 s of 30 ms steps)."""
    rng = np.random.Generator(np.random.PCG64(4000 + t))
    L = int(rng.integers(200_000, 2_000_001)) if kernels is None else int(kernels)
    n_steps = -(-L // 1000)
    kps = [1000] * (n_steps - 1) + [L - 1000 * (n_steps - 1)]
    w0 = EPOCH
    period = 30 * MS
    pr = _decode_process(rng, n_steps_kernels=kps, period=period, t0=w0 - 5 * MS, n_streams=4,
                         corr_base=int(rng.integers(0, 1 << 20)), drop_p=0.01)
    params = empty_params(window_begin=w0, window_end=w0 + n_steps * period, gap_threshold=20 * US,
                          n_procs=1, n_streams=4, n_threads=1, n_names=2000, n_op_names=100, flags=0)
    return _assemble(rng, [pr], [0], params, f"config4[{t}]")


def _config4_columns(t: int):
    tr = config4_trace(t)
    return tr.columns(), tr.params


def config4_chunk(ids, workers: int = 16, progress=None):
    """Columns and params of the batch traces `ids`, generated by a pool of
    fresh worker processes (spawned, so that a parent that already uses the
    GPU forks nothing); `progress(done, total)` is called as traces finish."""
    import multiprocessing as mp
    ids = [int(t) for t in ids]
    workers = max(1, min(workers, len(ids), os.cpu_count() or 1))
    out = []
    if workers == 1:
        for t in ids:
            out.append(_config4_columns(t))
            if progress:
                progress(len(out), len(ids))
        return out
    with mp.get_context("spawn").Pool(workers) as pool:
        for r in pool.imap(_config4_columns, ids):
            out.append(r)
            if progress:
                progress(len(out), len(ids))
    return out


def add_op_costs(cols: dict, params: dict, seed: int, ref: bool = True, flops_median: float = 2e9,
                 bytes_median: float = 5e8, peak_flops: int = 2_500_000_000_000_000,
                 peak_bytes: int = 8_000_000_000_000):
    """Columns of per-op operation counts and logical bytes (the shapes an
    analyzer recovers from Python object fields), device peaks and a
    reference SOL per op name, for the operator-efficiency outputs.  Counts
    are LogNormal (sigma 1.5) around 2 GFLOP and 0.5 GB per op by default,
    peaks those of a device of 2.5 PFLOP/s and 8 TB/s; rows other than ops
    get zeros."""
    rng = np.random.Generator(np.random.PCG64(seed))
    n = len(cols["ts"])
    ops = np.asarray(cols["kind"]) == CPU_OP
    flops = np.where(ops, np.rint(rng.lognormal(np.log(flops_median), 1.5, n)), 0).astype(np.int64)
    nbytes = np.where(ops, np.rint(rng.lognormal(np.log(bytes_median), 1.5, n)), 0).astype(np.int64)
    c = dict(cols, flops=flops, bytes=nbytes)
    q = dict(params, peak_flops=int(peak_flops), peak_bytes=int(peak_bytes),
             flags=int(params.get("flags", 3)) | 8 | 1)
    q["ref_sol_ppm"] = rng.integers(0, 400_000, int(params["n_op_names"])).astype(np.int64) if ref else None
    return c, q


def graph_replay_trace(seed: int = 21, n_steps: int = 200, n_nodes: int = 1000, n_streams: int = 2,
                       drop_p: float = 0.01, eager: int = 3, period: int = 30 * MS):
    """Decode steps replayed from one captured graph (the case where graph
    replay hides the operator calls): per step a CPU op holds one graph
    launch whose n_nodes kernels carry their node id (node i runs on stream
    i % n_streams, back to back per stream after the launch, each node with
    its own LogNormal median around 6 us and 20% spread per replay), and
    `eager` kernels launched one by one (graph node -1) under ops of their
    own.  Graph kernels are dropped with probability drop_p.  One process,
    one thread; the window cuts the first and the last step.  Returns
    (columns with graph_node, params)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w0 = EPOCH
    med = _lognormal_ns(rng, 6 * US, 1.0, n_nodes)
    node_name = _zipf(rng, 2000, 1.1, n_nodes)
    rows = []  # kind, lane, ts, te, corr, name, node
    corr = int(rng.integers(0, 1 << 20))
    for s_ in range(-1, n_steps + 1):
        t = w0 + s_ * period + int(rng.integers(0, 200 * US))
        step_rows = []
        lat = int(rng.integers(3 * US, 9 * US))
        l_end = t + int(rng.integers(10 * US, 20 * US))
        step_rows.append((1, 0, t, l_end, corr, 1, -1))
        ends = [t + lat] * n_streams
        dur = np.maximum(1, np.rint(med * rng.lognormal(0.0, 0.2, n_nodes))).astype(np.int64)
        keep = rng.random(n_nodes) >= drop_p
        for i in range(n_nodes):
            st = i % n_streams
            a = ends[st] + int(rng.integers(0, 2 * US))
            b = a + int(dur[i])
            ends[st] = b
            if keep[i]:
                step_rows.append((2, st, a, b, corr, int(node_name[i]), i))
        corr += 1
        g_end = max(ends)
        # eager kernels after the graph, each under its own op
        te_ = g_end + int(rng.integers(2 * US, 10 * US))
        for e in range(eager):
            o0 = te_
            l0 = o0 + int(rng.integers(1 * US, 3 * US))
            l1 = l0 + int(rng.integers(3 * US, 8 * US))
            k0 = max(l1, ends[0]) + int(rng.integers(1 * US, 5 * US))
            k1 = k0 + int(rng.integers(2 * US, 20 * US))
            ends[0] = k1
            step_rows.append((1, 0, l0, l1, corr, 0, -1))
            step_rows.append((2, 0, k0, k1, corr, int(rng.integers(0, 2000)), -1))
            step_rows.append((0, 0, o0, l1 + int(rng.integers(1 * US, 3 * US)), 0, 1 + e, -1))
            corr += 1
            te_ = l1 + int(rng.integers(4 * US, 8 * US))
        step_rows.append((0, 0, t - int(rng.integers(20 * US, 60 * US)), te_ + 5 * US, 0, 0, -1))
        rows.extend(step_rows)
    a = np.array(rows, np.int64)
    order = rng.permutation(len(a))
    a = a[order]
    cols = dict(kind=a[:, 0].astype(np.uint8), pid=np.zeros(len(a), np.int32), lane=a[:, 1].astype(np.int32),
                ts=a[:, 2], te=a[:, 3], corr=a[:, 4], name=a[:, 5].astype(np.int32),
                graph_node=a[:, 6].astype(np.int32))
    params = empty_params(window_begin=w0, window_end=w0 + n_steps * period, gap_threshold=20 * US,
                          n_procs=1, n_streams=n_streams, n_threads=1, n_names=2000, n_op_names=1 + eager,
                          flags=1 | 32, n_graph_nodes=n_nodes)
    return cols, params


def config4_lengths(n_traces: int = 256) -> np.ndarray:
    return np.array([int(np.random.Generator(np.random.PCG64(4000 + t)).integers(200_000, 2_000_001))
                     for t in range(n_traces)], np.int64)


def random_small(seed: int, *, n_rows: int = 60, window: int = 400, n_procs: int = 2,
                 n_streams: int = 3, n_threads: int = 2, n_names: int = 5, n_op_names: int = 4,
                 corr_range: int = 12, offsets: bool = True, edges: int = 6,
                 flags: int = 3) -> Trace:
    """Tiny adversarial traces for brute-force checks: ties, zero-length and
    same-stream-overlapping kernels, duplicate correlation ids, one launch with
    several kernels, improper nesting, rows outside the window."""
    rng = np.random.Generator(np.random.PCG64(seed))
    w0 = int(rng.integers(-10_000, 10_000))
    n = n_rows
    kind = rng.integers(0, 3, n).astype(np.uint8)
    pid = rng.integers(0, n_procs, n).astype(np.int32)
    off = rng.integers(-30, 31, n_procs).astype(np.int64) if offsets else np.zeros(n_procs, np.int64)
    ts = w0 - 40 + rng.integers(0, window + 80, n)
    # coarse grid for some rows -> many exact ties
    coarse = rng.random(n) < 0.4
    ts[coarse] = w0 + (ts[coarse] - w0) // 25 * 25
    dur = np.where(rng.random(n) < 0.15, 0, rng.integers(1, window // 3 + 2, n))
    te = ts + dur
    ts = (ts + off[pid]).astype(np.int64)
    te = (te + off[pid]).astype(np.int64)
    lane = np.where(kind == KERNEL, rng.integers(0, n_streams, n), rng.integers(0, n_threads, n)).astype(np.int32)
    name = np.where(kind == KERNEL, rng.integers(0, n_names, n),
                    np.where(kind == CPU_OP, rng.integers(0, n_op_names, n), rng.integers(0, 3, n))).astype(np.int32)
    corr = np.where(kind == CPU_OP, 0, rng.integers(0, corr_range, n)).astype(np.int64)
    e = np.zeros(edges, EDGE_DTYPE)
    e["prod_pid"] = rng.integers(0, n_procs + 1, edges)
    e["cons_pid"] = rng.integers(0, n_procs, edges)
    e["prod_corr"] = rng.integers(0, corr_range + 2, edges)
    e["cons_corr"] = rng.integers(0, corr_range + 2, edges)
    cls = rng.integers(0, 3, n_streams).astype(np.uint8)
    params = empty_params(window_begin=w0, window_end=w0 + window, gap_threshold=int(rng.integers(-1, 30)),
                          n_procs=n_procs, n_streams=n_streams, n_threads=n_threads, n_names=n_names,
                          n_op_names=n_op_names, clock_offset=off if offsets else None,
                          stream_class=cls if rng.random() < 0.7 else None, edges=e, flags=flags)
    return Trace(ts=ts, te=te, corr=corr, pid=pid, lane=lane, name=name, kind=kind, params=params,
                 label=f"random_small[{seed}]")


CONFIGS = {0: config0, 1: config1, 2: config2, 3: config3}
