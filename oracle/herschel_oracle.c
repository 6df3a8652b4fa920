/*
 * herschel_oracle.c -- TEST INFRASTRUCTURE ONLY: the CPU oracle.
 *
 * A plain, slow, single-threaded C implementation of the trace
 * reconstruction that the Herschel analyzer performs on one bounded
 * profiling window (Section 6.1, "Deriving Performance Observations", and
 * Figure "Key performance observations").  Only the tests, the smoke check
 * and the benchmark's CPU-baseline leg call it.  It shares no code with the
 * HIP library.
 *
 * The paper states the analysis in prose only; every result here is a plain
 * definition, written out step by step in the order below.  Readings of the
 * prose that the paper leaves open are marked READING.
 *
 *   1. validate rows                      (record schema, Section 5.2)
 *   2. correct clocks, 3. admit by start   (session transitions, Section 5.2)
 *   4-6. per-stream coverage, busy/idle, gaps (idle intervals, Section 9.1)
 *   7-8. launch/kernel join by correlation id, launch latency
 *        (call-to-kernel links, Section 6.1; the submission-time and
 *        "correlation id" in panel "Operator execution and efficiency")
 *   9-12. op nesting, launch -> op, kernel -> op, inclusive T_op aggregates
 *        (kernel composition and T_op, Section 6.1; nested calls, Section 5.2)
 *   13. per kernel-name aggregates
 *   14. cross-stream overlap as interval coverage (panel "Overlap and exposed
 *       work"; Section 6.1 "Execution progress and state")
 *   15. cross-process dependency waits (panel "Cross-process blocking")
 *   16. GPU idle coinciding with CPU ops, by op name (Section 9.1)
 *   17. operator MFU, MBU and SOL, per op name and Hotness (Section 6.1,
 *       "Operator execution and efficiency"; Section 6.2)
 *
 * Sorting uses the C library's qsort with comparators that end in the row
 * index, so every order is total and the result does not depend on qsort's
 * stability.  Sums use unsigned arithmetic and wrap modulo 2^64.
 *
 * Parity: pinned in the tests against the hand-built worked timeline, a
 * per-nanosecond brute force on tiny traces, invariants and the trace
 * generator's ground truth.  No output is "parity unpinned".
 */
#include "herschel_oracle.h"

#include <stdlib.h>
#include <string.h>

#define K_CPU 0
#define K_LAUNCH 1
#define K_KERNEL 2
#define I64_MAX ((int64_t)0x7fffffffffffffffLL)
#define I64_MIN ((int64_t)(-0x7fffffffffffffffLL - 1))
#define ABS_LIMIT (1LL << 62)

static int64_t wrap_add(int64_t a, int64_t b) { return (int64_t)((uint64_t)a + (uint64_t)b); }
static int64_t wrap_sub(int64_t a, int64_t b) { return (int64_t)((uint64_t)a - (uint64_t)b); }
static int in_abs(int64_t x) { return x > -ABS_LIMIT && x < ABS_LIMIT; }

/* ---- step 1: row validity (record schema of Section 5.2) ---------------- */
static int row_is_valid(const hro_events *ev, int64_t i, const hro_params *p) {
  int k = ev->kind[i];
  if (k != K_CPU && k != K_LAUNCH && k != K_KERNEL) return 0;
  if (ev->pid[i] < 0 || ev->pid[i] >= p->n_procs) return 0;
  if (k == K_KERNEL) {
    if (ev->lane[i] < 0 || ev->lane[i] >= p->n_streams) return 0;
    if (ev->name[i] < 0 || ev->name[i] >= p->n_names) return 0;
  } else {
    if (ev->lane[i] < 0 || ev->lane[i] >= p->n_threads) return 0;
    if (k == K_CPU && (ev->name[i] < 0 || ev->name[i] >= p->n_op_names)) return 0;
    if (k == K_LAUNCH && ev->name[i] < 0) return 0;
  }
  if (!in_abs(ev->ts[i]) || !in_abs(ev->te[i])) return 0;
  if (ev->te[i] < ev->ts[i]) return 0;
  /* with the SOL outputs, an op's operation count and logical bytes */
  if ((p->flags & 8u) != 0 && k == K_CPU && (ev->flops[i] < 0 || ev->bytes[i] < 0)) return 0;
  /* with graph replay separation, a kernel's graph node */
  if ((p->flags & 32u) != 0 && k == K_KERNEL && (ev->graph_node[i] < -1 || ev->graph_node[i] >= p->n_graph_nodes))
    return 0;
  return 1;
}

static int params_ok(int64_t n, const hro_params *p) {
  if (n < 0 || n >= (1LL << 30)) return 0;
  if (!in_abs(p->w0) || !in_abs(p->w1) || p->w1 <= p->w0) return 0;
  if (p->w1 - p->w0 > (1LL << 40)) return 0;
  if (p->n_procs < 1 || p->n_procs > 4096) return 0;
  if (p->n_streams < 1 || p->n_streams > 64) return 0;
  if (p->n_threads < 1 || p->n_threads > 2048) return 0;
  if (p->n_names < 1 || p->n_names > (1 << 24)) return 0;
  if (p->n_op_names < 1) return 0;
  if (p->n_edges < 0 || (p->n_edges > 0 && !p->edges)) return 0;
  /* implementation limit shared with the library, for error parity: with
   * the idle-coincidence outputs, at most 2048 op names */
  if ((p->flags & 4u) != 0 && p->n_op_names > 2048) return 0;
  /* SOL needs T_op (containment), positive peaks */
  if ((p->flags & 8u) != 0) {
    if ((p->flags & 1u) == 0 || p->peak_flops <= 0 || p->peak_bytes <= 0) return 0;
    if (p->ref_sol_ppm)
      for (int o = 0; o < p->n_op_names; ++o)
        if (p->ref_sol_ppm[o] < 0) return 0;
  }
  /* the critical path walks the host nesting (containment) */
  if ((p->flags & 16u) != 0 && (p->flags & 1u) == 0) return 0;
  /* graph replay separation uses the per-launch kernel spans of containment */
  if ((p->flags & 32u) != 0 && ((p->flags & 1u) == 0 || p->n_graph_nodes < 1)) return 0;
  if (p->clock_offset)
    for (int q = 0; q < p->n_procs; ++q)
      if (!in_abs(p->clock_offset[q])) return 0;
  if (p->stream_class)
    for (int s = 0; s < p->n_streams; ++s)
      if (p->stream_class[s] > 2) return 0;
  return 1;
}

/* ---- generic sort records --------------------------------------------- */
typedef struct {
  int64_t a, b, c; /* sort fields, compared in order */
  int64_t row;
} rec4;

static int cmp_rec4(const void *x, const void *y) {
  const rec4 *u = (const rec4 *)x, *v = (const rec4 *)y;
  if (u->a != v->a) return u->a < v->a ? -1 : 1;
  if (u->b != v->b) return u->b < v->b ? -1 : 1;
  if (u->c != v->c) return u->c < v->c ? -1 : 1;
  if (u->row != v->row) return u->row < v->row ? -1 : 1;
  return 0;
}

typedef struct {
  int64_t s, e;
} ival;

static int cmp_ival(const void *x, const void *y) {
  const ival *u = (const ival *)x, *v = (const ival *)y;
  if (u->s != v->s) return u->s < v->s ? -1 : 1;
  if (u->e != v->e) return u->e < v->e ? -1 : 1;
  return 0;
}

/* Merge a start-sorted list of half-open intervals into maximal disjoint runs.
 * Touching intervals merge; empty intervals are never passed in (step 4). */
static int64_t merge_runs(ival *v, int64_t m) {
  int64_t r = 0;
  for (int64_t i = 0; i < m; ++i) {
    if (r > 0 && v[i].s <= v[r - 1].e) {
      if (v[i].e > v[r - 1].e) v[r - 1].e = v[i].e;
    } else {
      v[r++] = v[i];
    }
  }
  return r;
}

static int64_t runs_length(const ival *v, int64_t m) {
  int64_t t = 0;
  for (int64_t i = 0; i < m; ++i) t += v[i].e - v[i].s;
  return t;
}

/* |A intersect B| for two sorted lists of disjoint runs. */
static int64_t runs_intersection(const ival *a, int64_t na, const ival *b, int64_t nb) {
  int64_t i = 0, j = 0, t = 0;
  while (i < na && j < nb) {
    int64_t lo = a[i].s > b[j].s ? a[i].s : b[j].s;
    int64_t hi = a[i].e < b[j].e ? a[i].e : b[j].e;
    if (hi > lo) t += hi - lo;
    if (a[i].e < b[j].e) ++i; else ++j;
  }
  return t;
}

/* Union of several run lists: concatenate, sort by start, merge. */
static int64_t union_of(ival *const *lists, const int64_t *lens, int nl, ival **outp) {
  int64_t tot = 0;
  for (int k = 0; k < nl; ++k) tot += lens[k];
  ival *u = (ival *)malloc(sizeof(ival) * (size_t)(tot > 0 ? tot : 1));
  int64_t w = 0;
  for (int k = 0; k < nl; ++k) {
    memcpy(u + w, lists[k], sizeof(ival) * (size_t)lens[k]);
    w += lens[k];
  }
  qsort(u, (size_t)tot, sizeof(ival), cmp_ival);
  int64_t r = merge_runs(u, tot);
  *outp = u;
  return r;
}

/* floor(10^15 x / (t peak)) in parts per million: x per t ns against a peak
 * per second (step 17), exact in 128 bits; saturates at INT64_MAX. */
static int64_t ppm_of(uint64_t x, uint64_t t, uint64_t peak) {
  unsigned __int128 num = (unsigned __int128)x * 1000000000000000ull;
  unsigned __int128 den = (unsigned __int128)t * peak;
  unsigned __int128 q = num / den;
  return q > (unsigned __int128)I64_MAX ? I64_MAX : (int64_t)q;
}

/* floor(log2 x) + 1 for x > 0, 0 otherwise (step 8's histogram bin). */
static int latency_bin(int64_t x) {
  int b = 0;
  while (x > 0) {
    ++b;
    x >>= 1;
  }
  return b;
}

int herschel_oracle_analyze(const hro_events *ev, int64_t n, const hro_params *p,
                            hro_outputs *out) {
  if (!ev || !p || !out || !out->counters) return -1;
  if (!params_ok(n, p)) return -1;
  if ((p->flags & 8u) != 0 && n > 0 && (!ev->flops || !ev->bytes)) return -1;
  if ((p->flags & 32u) != 0 && n > 0 && !ev->graph_node) return -1;
  const int P = p->n_procs, S = p->n_streams;
  const int64_t W0 = p->w0, W1 = p->w1, W = W1 - W0;
  const int contain = (p->flags & 1u) != 0, overlap = (p->flags & 2u) != 0;
  hro_counters *c = out->counters;
  memset(c, 0, sizeof(*c));
  c->first_invalid = -1;

  /* 1. Validate every row; the smallest bad index is reported. */
  for (int64_t i = 0; i < n; ++i)
    if (!row_is_valid(ev, i, p)) {
      c->first_invalid = i;
      return -2;
    }

  /* 2. Correct each row onto the common clock: corrected = raw - offset[pid].
   *    READING: the paper does not discuss clock alignment; offsets are given. */
  int64_t *ts = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
  int64_t *te = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
  unsigned char *adm = (unsigned char *)calloc((size_t)(n > 0 ? n : 1), 1);
  for (int64_t i = 0; i < n; ++i) {
    int64_t off = p->clock_offset ? p->clock_offset[ev->pid[i]] : 0;
    ts[i] = ev->ts[i] - off;
    te[i] = ev->te[i] - off;
  }

  /* 3. Admit a row iff its corrected start lies in [W0, W1) (start-time
   *    filtering, Section 5.2).  Rows outside get link = aux = -2. */
  for (int64_t i = 0; i < n; ++i) {
    adm[i] = (ts[i] >= W0 && ts[i] < W1);
    if (adm[i]) {
      c->n_admitted[ev->kind[i]]++;
      out->link[i] = -1;
      out->aux[i] = -1;
    } else {
      c->n_outside_window++;
      out->link[i] = -2;
      out->aux[i] = -2;
    }
  }

  /* 4-6. Per (process, stream): coverage of the admitted kernels, each
   * covering [ts', min(te', W1)); empty intervals cover nothing; touching
   * intervals merge.  busy = |union|, idle = W - busy.  Gaps are the maximal
   * uncovered sub-intervals of [W0, W1), emitted in (p, s, begin) order when
   * longer than the threshold.  (Idle intervals of GPU activity, Section 9.1.) */
  int64_t nk = 0;
  for (int64_t i = 0; i < n; ++i)
    if (adm[i] && ev->kind[i] == K_KERNEL) ++nk;
  rec4 *kr = (rec4 *)malloc(sizeof(rec4) * (size_t)(nk > 0 ? nk : 1));
  {
    int64_t w = 0;
    for (int64_t i = 0; i < n; ++i)
      if (adm[i] && ev->kind[i] == K_KERNEL) {
        kr[w].a = (int64_t)ev->pid[i] * S + ev->lane[i];
        kr[w].b = ts[i];
        kr[w].c = te[i] < W1 ? te[i] : W1;
        kr[w].row = i;
        ++w;
      }
    qsort(kr, (size_t)nk, sizeof(rec4), cmp_rec4);
  }
  ival **runs = (ival **)calloc((size_t)P * S, sizeof(ival *));
  int64_t *nruns = (int64_t *)calloc((size_t)P * S, sizeof(int64_t));
  int64_t gw = 0;
  {
    int64_t at = 0;
    for (int64_t ps = 0; ps < (int64_t)P * S; ++ps) {
      int64_t begin = at;
      while (at < nk && kr[at].a == ps) ++at;
      ival *v = (ival *)malloc(sizeof(ival) * (size_t)(at - begin + 1));
      int64_t m = 0;
      for (int64_t q = begin; q < at; ++q)
        if (kr[q].c > kr[q].b) { /* non-empty after clipping */
          v[m].s = kr[q].b;
          v[m].e = kr[q].c;
          ++m;
        }
      int64_t r = merge_runs(v, m);
      runs[ps] = v;
      nruns[ps] = r;
      int64_t b = runs_length(v, r);
      out->busy[ps] = b;
      out->idle[ps] = W - b;
      int64_t prev = W0;
      for (int64_t q = 0; q <= r; ++q) {
        int64_t gb = prev, ge = (q < r) ? v[q].s : W1;
        if (ge > gb) {
          if (ge - gb > p->thr) {
            if (gw < out->gap_capacity) {
              out->gap_pid[gw] = (int32_t)(ps / S);
              out->gap_stream[gw] = (int32_t)(ps % S);
              out->gap_begin[gw] = gb;
              out->gap_end[gw] = ge;
              out->gap_flags[gw] = (uint8_t)((gb == W0 ? 1 : 0) | (ge == W1 ? 2 : 0));
            }
            ++gw;
          }
        }
        if (q < r) prev = v[q].e;
      }
    }
  }
  c->n_gaps_total = gw;

  /* 7. Join each admitted kernel to the admitted launch with the same
   *    (process, correlation id) (call-to-kernel links, Section 6.1).  Several
   *    launches with one id: the smallest row wins, the others are counted as
   *    duplicates.  One launch may own several kernels (graph replay). */
  int64_t nl = 0;
  for (int64_t i = 0; i < n; ++i)
    if (adm[i] && ev->kind[i] == K_LAUNCH) ++nl;
  rec4 *lr = (rec4 *)malloc(sizeof(rec4) * (size_t)(nl > 0 ? nl : 1));
  {
    int64_t w = 0;
    for (int64_t i = 0; i < n; ++i)
      if (adm[i] && ev->kind[i] == K_LAUNCH) {
        lr[w].a = ev->pid[i];
        lr[w].b = ev->corr[i];
        lr[w].c = 0;
        lr[w].row = i;
        ++w;
      }
    qsort(lr, (size_t)nl, sizeof(rec4), cmp_rec4);
    for (int64_t q = 1; q < nl; ++q)
      if (lr[q].a == lr[q - 1].a && lr[q].b == lr[q - 1].b) c->n_dup_launch_corr++;
    for (int64_t q = 0; q < nl; ++q) out->aux[lr[q].row] = 0;
  }
  for (int64_t i = 0; i < n; ++i) {
    if (!adm[i] || ev->kind[i] != K_KERNEL) continue;
    /* lower bound of (pid, corr) among sorted launches */
    int64_t lo = 0, hi = nl;
    while (lo < hi) {
      int64_t mid = lo + (hi - lo) / 2;
      if (lr[mid].a < ev->pid[i] || (lr[mid].a == ev->pid[i] && lr[mid].b < ev->corr[i]))
        lo = mid + 1;
      else
        hi = mid;
    }
    if (lo < nl && lr[lo].a == ev->pid[i] && lr[lo].b == ev->corr[i]) {
      int64_t l = lr[lo].row;
      out->link[i] = (int32_t)l;
      out->aux[l]++;
      c->n_matched++;
      /* 8. Launch latency: kernel start minus the launch's start (the host
       *    submission time of the operator panel).  Signed.  Bin 0 for
       *    x <= 0, else floor(log2 x) + 1. */
      int64_t x = ts[i] - ts[l];
      if (x < 0) c->n_negative_latency++;
      out->lat_hist[latency_bin(x)]++;
    } else {
      out->link[i] = -1;
      c->n_unmatched_kernels++;
    }
  }
  for (int64_t q = 0; q < nl; ++q)
    if (out->aux[lr[q].row] == 0) c->n_unmatched_launches++;

  /* 9-12. Containment (Section 6.1 "kernel composition"; nested calls are
   * recorded, Section 5.2). */
  if (contain) {
    int64_t nc = c->n_admitted[K_CPU];
    rec4 *cr = (rec4 *)malloc(sizeof(rec4) * (size_t)(nc > 0 ? nc : 1));
    int64_t *par = (int64_t *)malloc(sizeof(int64_t) * (size_t)(nc > 0 ? nc : 1));
    int64_t *segstart = (int64_t *)malloc(sizeof(int64_t) * (size_t)(nc > 0 ? nc : 1));
    int64_t w = 0;
    for (int64_t i = 0; i < n; ++i)
      if (adm[i] && ev->kind[i] == K_CPU) {
        cr[w].a = (int64_t)ev->pid[i] * p->n_threads + ev->lane[i];
        cr[w].b = ts[i];
        cr[w].c = -te[i]; /* te' descending: the outer of two ops starting together first */
        cr[w].row = i;
        ++w;
      }
    qsort(cr, (size_t)nc, sizeof(rec4), cmp_rec4);
    /* 9. Parent of op i: the nearest op before it in the (thread, ts' up,
     *    te' down, row up) order whose end is after i's start.  READING: this
     *    equals the innermost enclosing op for properly nested calls and is
     *    defined for any input.  The backward scan may skip from a failing
     *    candidate j straight to parent(j): every op strictly between them
     *    ends no later than ts'_j <= ts'_i, so none of them qualifies. */
    for (int64_t q = 0; q < nc; ++q) {
      segstart[q] = (q > 0 && cr[q].a == cr[q - 1].a) ? segstart[q - 1] : q;
      int64_t j = q - 1;
      while (j >= segstart[q] && -cr[j].c <= cr[q].b) j = par[j];
      if (j < segstart[q]) j = -1;
      par[q] = j;
      int64_t row = cr[q].row;
      if (j < 0) {
        out->link[row] = -1;
        out->aux[row] = 0;
      } else {
        out->link[row] = (int32_t)cr[j].row;
        out->aux[row] = out->aux[cr[j].row] + 1;
        if (te[row] > te[cr[j].row]) c->n_improper_nesting++;
      }
    }
    /* 10. A launch lies in the innermost op of its thread that contains its
     *     start point t: the last op in the order with ts' <= t and te' > t. */
    for (int64_t i = 0; i < n; ++i) {
      if (!adm[i] || ev->kind[i] != K_LAUNCH) continue;
      int64_t seg = (int64_t)ev->pid[i] * p->n_threads + ev->lane[i], t = ts[i];
      /* last position with (seg, ts') <= (seg, t) */
      int64_t lo = 0, hi = nc;
      while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (cr[mid].a < seg || (cr[mid].a == seg && cr[mid].b <= t))
          lo = mid + 1;
        else
          hi = mid;
      }
      int64_t j = lo - 1;
      if (j >= 0 && cr[j].a != seg) j = -1;
      while (j >= 0 && -cr[j].c <= t) j = par[j];
      out->link[i] = j >= 0 ? (int32_t)cr[j].row : -1;
    }
    /* 11. A kernel belongs to the op its launch lies in. */
    for (int64_t i = 0; i < n; ++i) {
      if (!adm[i] || ev->kind[i] != K_KERNEL) continue;
      int64_t l = out->link[i];
      if (l < 0) {
        out->aux[i] = -1;
      } else {
        out->aux[i] = out->link[l];
        if (out->link[l] < 0) c->n_unattributed_kernels++;
      }
    }
    /* 12. Inclusive per-op aggregates: every kernel counts for its op and
     *     for each ancestor.  T_op runs from the earliest kernel start to the latest
     *     kernel end (Section 6.1), unclipped. */
    for (int64_t q = 0; q < nc; ++q) {
      int64_t r = cr[q].row;
      out->op_nkern[r] = 0;
      out->op_first[r] = I64_MAX;
      out->op_last[r] = I64_MIN;
      out->op_ksum[r] = 0;
    }
    for (int64_t i = 0; i < n; ++i) {
      if (!adm[i] || ev->kind[i] != K_KERNEL) continue;
      int64_t r = out->aux[i];
      while (r >= 0) {
        out->op_nkern[r]++;
        if (ts[i] < out->op_first[r]) out->op_first[r] = ts[i];
        if (te[i] > out->op_last[r]) out->op_last[r] = te[i];
        out->op_ksum[r] = wrap_add(out->op_ksum[r], te[i] - ts[i]);
        r = out->link[r];
      }
    }
    free(cr);
    free(par);
    free(segstart);
  }

  /* 13. Per kernel-name aggregates over all admitted kernels, matched or not:
   *     count, sum, min and max of the unclipped duration te' - ts'. */
  for (int q = 0; q < p->n_names; ++q) {
    out->name_count[q] = 0;
    out->name_sum[q] = 0;
    out->name_min[q] = I64_MAX;
    out->name_max[q] = I64_MIN;
  }
  for (int64_t i = 0; i < n; ++i) {
    if (!adm[i] || ev->kind[i] != K_KERNEL) continue;
    int q = ev->name[i];
    int64_t d = te[i] - ts[i];
    out->name_count[q]++;
    out->name_sum[q] = wrap_add(out->name_sum[q], d);
    if (d < out->name_min[q]) out->name_min[q] = d;
    if (d > out->name_max[q]) out->name_max[q] = d;
  }

  /* 13b. The same per op name over all admitted CPU ops (the per-op-name
   *      variant): count, sum, min and max of te' - ts', unclipped.  Each
   *      output may be NULL. */
  for (int q = 0; q < p->n_op_names; ++q) {
    if (out->opname_count) out->opname_count[q] = 0;
    if (out->opname_sum) out->opname_sum[q] = 0;
    if (out->opname_min) out->opname_min[q] = I64_MAX;
    if (out->opname_max) out->opname_max[q] = I64_MIN;
  }
  for (int64_t i = 0; i < n; ++i) {
    if (!adm[i] || ev->kind[i] != K_CPU) continue;
    int q = ev->name[i];
    int64_t d = te[i] - ts[i];
    if (out->opname_count) out->opname_count[q]++;
    if (out->opname_sum) out->opname_sum[q] = wrap_add(out->opname_sum[q], d);
    if (out->opname_min && d < out->opname_min[q]) out->opname_min[q] = d;
    if (out->opname_max && d > out->opname_max[q]) out->opname_max[q] = d;
  }

  /* 14. Overlap as interval coverage (panel "Overlap and exposed work"):
   *     per process, with U_s the covered set of stream s,
   *     pair_overlap[i][j] = |U_i and U_j|, class_busy[c] = |union over the
   *     class|, class_overlap[c1][c2] = |class c1 union and class c2 union|,
   *     any_busy = |union over all streams|. */
  if (overlap) {
    for (int pp = 0; pp < P; ++pp) {
      ival **L = runs + (int64_t)pp * S;
      int64_t *N = nruns + (int64_t)pp * S;
      for (int i = 0; i < S; ++i)
        for (int j = 0; j < S; ++j)
          out->pair_overlap[((int64_t)pp * S + i) * S + j] =
              runs_intersection(L[i], N[i], L[j], N[j]);
      ival *cls[3];
      int64_t ncls[3];
      for (int cc = 0; cc < 3; ++cc) {
        ival *sel[64];
        int64_t seln[64];
        int ns = 0;
        for (int s = 0; s < S; ++s) {
          int sc = p->stream_class ? p->stream_class[s] : 0;
          if (sc == cc) {
            sel[ns] = L[s];
            seln[ns] = N[s];
            ++ns;
          }
        }
        ncls[cc] = union_of(sel, seln, ns, &cls[cc]);
        out->class_busy[(int64_t)pp * 3 + cc] = runs_length(cls[cc], ncls[cc]);
      }
      for (int c1 = 0; c1 < 3; ++c1)
        for (int c2 = 0; c2 < 3; ++c2)
          out->class_overlap[((int64_t)pp * 3 + c1) * 3 + c2] =
              runs_intersection(cls[c1], ncls[c1], cls[c2], ncls[c2]);
      ival *all;
      int64_t nall = union_of(L, N, S, &all);
      out->any_busy[pp] = runs_length(all, nall);
      free(all);
      for (int cc = 0; cc < 3; ++cc) free(cls[cc]);
    }
  }

  /* 15. Cross-process dependency waits (panel "Cross-process blocking"):
   *     producer = the admitted kernel with (prod_pid, prod_corr) that ends
   *     last, consumer = the one with (cons_pid, cons_corr) that starts first;
   *     wait = consumer start - producer end, signed.  Missing side: status
   *     bit (0 producer, 1 consumer) and wait = INT64_MIN. */
  if (p->n_edges > 0) {
    rec4 *kc = (rec4 *)malloc(sizeof(rec4) * (size_t)(nk > 0 ? nk : 1));
    int64_t w = 0;
    for (int64_t i = 0; i < n; ++i)
      if (adm[i] && ev->kind[i] == K_KERNEL) {
        kc[w].a = ev->pid[i];
        kc[w].b = ev->corr[i];
        kc[w].c = 0;
        kc[w].row = i;
        ++w;
      }
    qsort(kc, (size_t)nk, sizeof(rec4), cmp_rec4);
    for (int64_t e = 0; e < p->n_edges; ++e) {
      int found[2] = {0, 0};
      int64_t prod_end = I64_MIN, cons_start = I64_MAX;
      for (int side = 0; side < 2; ++side) {
        int64_t qp = side == 0 ? p->edges[e].prod_pid : p->edges[e].cons_pid;
        int64_t qc = side == 0 ? p->edges[e].prod_corr : p->edges[e].cons_corr;
        int64_t lo = 0, hi = nk;
        while (lo < hi) {
          int64_t mid = lo + (hi - lo) / 2;
          if (kc[mid].a < qp || (kc[mid].a == qp && kc[mid].b < qc))
            lo = mid + 1;
          else
            hi = mid;
        }
        for (int64_t q = lo; q < nk && kc[q].a == qp && kc[q].b == qc; ++q) {
          int64_t r = kc[q].row;
          found[side] = 1;
          if (side == 0 && te[r] > prod_end) prod_end = te[r];
          if (side == 1 && ts[r] < cons_start) cons_start = ts[r];
        }
      }
      out->edge_status[e] = (found[0] ? 0 : 1) | (found[1] ? 0 : 2);
      out->edge_wait[e] = (found[0] && found[1]) ? wrap_sub(cons_start, prod_end) : I64_MIN;
    }
    free(kc);
  }

  /* 16. GPU idle coinciding with CPU ops, by op name (the evidence of the
   *     case study in Section 9.1: idle intervals of the GPU activity that
   *     coincide with the Worker's waits in one Python call).  READING: the
   *     GPU of process p is idle where none of its streams' kernels covers
   *     the time; its idle intervals are the maximal such sub-intervals of
   *     [W0, W1), kept when longer than the gap threshold (as gaps are).
   *     Per op name o of process p, U = the union of its admitted ops'
   *     ranges [ts', min(te', W1)); op_span = |U|, op_idle = |U and the kept
   *     idle intervals|, dev_idle[p] = their total length. */
  if ((p->flags & 4u) != 0) {
    const int NOP = p->n_op_names;
    /* the admitted ops' non-empty clipped ranges, by (process, name, start) */
    int64_t nc = 0;
    for (int64_t i = 0; i < n; ++i)
      if (adm[i] && ev->kind[i] == K_CPU) ++nc;
    rec4 *orc = (rec4 *)malloc(sizeof(rec4) * (size_t)(nc > 0 ? nc : 1));
    int64_t no = 0;
    for (int64_t i = 0; i < n; ++i)
      if (adm[i] && ev->kind[i] == K_CPU) {
        int64_t e = te[i] < W1 ? te[i] : W1;
        if (e > ts[i]) {
          orc[no].a = (int64_t)ev->pid[i] * NOP + ev->name[i];
          orc[no].b = ts[i];
          orc[no].c = e;
          orc[no].row = i;
          ++no;
        }
      }
    qsort(orc, (size_t)no, sizeof(rec4), cmp_rec4);
    for (int64_t q = 0; q < (int64_t)P * NOP; ++q) {
      out->op_span[q] = 0;
      out->op_idle[q] = 0;
    }
    ival *u = (ival *)malloc(sizeof(ival) * (size_t)(no > 0 ? no : 1));
    int64_t at = 0;
    for (int pp = 0; pp < P; ++pp) {
      ival *all;
      int64_t nall = union_of(runs + (int64_t)pp * S, nruns + (int64_t)pp * S, S, &all);
      /* the complement of the busy runs in [W0, W1), long ones only */
      ival *idle = (ival *)malloc(sizeof(ival) * (size_t)(nall + 1));
      int64_t ni = 0, prev = W0, tot = 0;
      for (int64_t q = 0; q <= nall; ++q) {
        int64_t gb = prev, ge = q < nall ? all[q].s : W1;
        if (ge > gb && ge - gb > p->thr) {
          idle[ni].s = gb;
          idle[ni].e = ge;
          tot += ge - gb;
          ++ni;
        }
        if (q < nall) prev = all[q].e;
      }
      out->dev_idle[pp] = tot;
      /* each op name of this process: union of its ranges, then the idle part */
      while (at < no && orc[at].a / NOP == pp) {
        int64_t seg = orc[at].a, w = 0;
        while (at < no && orc[at].a == seg) {
          u[w].s = orc[at].b;
          u[w].e = orc[at].c;
          ++w;
          ++at;
        }
        int64_t r = merge_runs(u, w);
        out->op_span[seg] = runs_length(u, r);
        out->op_idle[seg] = runs_intersection(u, r, idle, ni);
      }
      free(idle);
      free(all);
    }
    free(u);
    free(orc);
  }

  /* 17. Operator efficiency (Section 6.1, "Operator execution and
   *     efficiency"): the op's operation count F and logical bytes B,
   *     normalized by T_op = op_last - op_first and the device peaks, give
   *     MFU and MBU; SOL = max(MFU, MBU).  READING: parts per million,
   *     floor(10^15 F / (T_op[ns] peak_flops[/s])), exact in 128 bits; an op
   *     without kernels or with T_op = 0 is unmeasured (-1).  Per op name,
   *     over its measured ops: the sums of F, B and T_op (wrapping), SOL of
   *     the sums, and Hotness, the time recoverable at the name's reference
   *     SOL: sum of floor(T_op (ref - SOL) / ref) over ops below it
   *     (Section 6.2 weights that fraction by time). */
  if ((p->flags & 8u) != 0) {
    const int NOP = p->n_op_names;
    for (int o = 0; o < NOP; ++o) {
      out->opn_flops[o] = 0;
      out->opn_bytes[o] = 0;
      out->opn_time[o] = 0;
      out->opn_hot[o] = 0;
    }
    for (int64_t i = 0; i < n; ++i) {
      if (!adm[i] || ev->kind[i] != K_CPU) continue;
      int64_t T = out->op_nkern[i] > 0 ? wrap_sub(out->op_last[i], out->op_first[i]) : 0;
      if (T <= 0) {
        out->op_mfu[i] = out->op_mbu[i] = out->op_sol[i] = -1;
        continue;
      }
      out->op_mfu[i] = ppm_of((uint64_t)ev->flops[i], (uint64_t)T, (uint64_t)p->peak_flops);
      out->op_mbu[i] = ppm_of((uint64_t)ev->bytes[i], (uint64_t)T, (uint64_t)p->peak_bytes);
      out->op_sol[i] = out->op_mfu[i] > out->op_mbu[i] ? out->op_mfu[i] : out->op_mbu[i];
      int o = ev->name[i];
      out->opn_flops[o] = wrap_add(out->opn_flops[o], ev->flops[i]);
      out->opn_bytes[o] = wrap_add(out->opn_bytes[o], ev->bytes[i]);
      out->opn_time[o] = wrap_add(out->opn_time[o], T);
      int64_t ref = p->ref_sol_ppm ? p->ref_sol_ppm[o] : 0;
      if (ref > 0 && out->op_sol[i] < ref) {
        unsigned __int128 x = (unsigned __int128)(uint64_t)T * (uint64_t)(ref - out->op_sol[i]);
        out->opn_hot[o] = wrap_add(out->opn_hot[o], (int64_t)(uint64_t)(x / (uint64_t)ref));
      }
    }
    for (int o = 0; o < NOP; ++o) {
      uint64_t t = (uint64_t)out->opn_time[o];
      if (t == 0) {
        out->opn_sol[o] = -1;
      } else {
        int64_t f = ppm_of((uint64_t)out->opn_flops[o], t, (uint64_t)p->peak_flops);
        int64_t b = ppm_of((uint64_t)out->opn_bytes[o], t, (uint64_t)p->peak_bytes);
        out->opn_sol[o] = f > b ? f : b;
      }
    }
  }

  /* 18. Critical path (Section 6.1, "Execution progress and state"; the
   *     figure of the critical path: submission, execution-order and
   *     synchronization dependencies).  READING: every admitted record x has
   *     a start event S(x) at ts' and an end event E(x) at min(te', W1).
   *     Walking back from the end event of the process's last-ending record
   *     (largest end, then largest row), each event steps to the one event
   *     that released it:
   *       E(kernel)        <- its own S (it ran);
   *       E(launch)        <- E(g) when the launch has no kernels of its own
   *                           and g, the process's kernel ending last strictly
   *                           inside the call (largest end, then row), exists
   *                           (a synchronizing call returns when g completes);
   *                           else its own S;
   *       E(op)            <- E(last child) if that child ends no later than
   *                           the op, else its own S;
   *       S(kernel)        <- of E(previous kernel on its stream), if it ended
   *                           by the kernel's start, and its launch (E(launch)
   *                           if the launch ended by then, else S(launch),
   *                           if it started by then): the later release,
   *                           the launch on a tie;
   *       S(op or launch)  <- of E(previous sibling), if it ended by the
   *                           start, and S(parent): the later, the sibling on
   *                           a tie; none: the path starts here.
   *     Children and siblings are ordered by the containment order of the
   *     thread (ts' up, ops before launches, ops by te' down, row up).  Each
   *     step's time difference is attributed: kernel run, launch API time
   *     (its own interval, or the part before its kernel started), the sync
   *     tail after the releasing kernel, op self time (the part after its
   *     last child or before a child's start, or all of a leaf op), and the
   *     unattributed gaps (launch gap: launch end to kernel start; queue gap:
   *     previous kernel end to kernel start; host gap: previous sibling end
   *     to start).  A strictly earlier release makes the steps acyclic. */
  if ((p->flags & 16u) != 0) {
    const int T = p->n_threads;
    int64_t *tS = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *tE = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *kprev = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *sib = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *lastc = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *gate = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    int64_t *pos = (int64_t *)malloc(sizeof(int64_t) * (size_t)(n > 0 ? n : 1));
    rec4 *hr = (rec4 *)malloc(sizeof(rec4) * (size_t)(n > 0 ? n : 1));
    rec4 *ke = (rec4 *)malloc(sizeof(rec4) * (size_t)(n > 0 ? n : 1));
    int64_t nh = 0, nk = 0, nke = 0;
    for (int64_t i = 0; i < n; ++i) {
      kprev[i] = sib[i] = lastc[i] = gate[i] = pos[i] = -1;
      if (!adm[i]) continue;
      tS[i] = ts[i];
      tE[i] = te[i] < W1 ? te[i] : W1;
      out->crit_time[i] = 0;
      out->crit_flags[i] = 0;
    }
    for (int64_t q = 0; q < (int64_t)P * 8; ++q) out->crit_proc[q] = 0;
    /* stream order of the kernels: (pid, stream, ts', row) */
    for (int64_t i = 0; i < n; ++i)
      if (adm[i] && ev->kind[i] == K_KERNEL) {
        hr[nk].a = (int64_t)ev->pid[i] * S + ev->lane[i];
        hr[nk].b = ts[i];
        hr[nk].c = 0;
        hr[nk].row = i;
        ++nk;
        ke[nke].a = ev->pid[i];
        ke[nke].b = tE[i];
        ke[nke].c = 0;
        ke[nke].row = i;
        ++nke;
      }
    qsort(hr, (size_t)nk, sizeof(rec4), cmp_rec4);
    for (int64_t q = 1; q < nk; ++q)
      if (hr[q].a == hr[q - 1].a) kprev[hr[q].row] = hr[q - 1].row;
    /* kernels by (pid, end, row), for the synchronizing calls */
    qsort(ke, (size_t)nke, sizeof(rec4), cmp_rec4);
    for (int64_t i = 0; i < n; ++i) {
      if (!adm[i] || ev->kind[i] != K_LAUNCH || out->aux[i] != 0) continue;
      /* last kernel with (pid, end) < (pid, E(L)) */
      int64_t lo = 0, hi = nke;
      while (lo < hi) {
        int64_t mid = lo + (hi - lo) / 2;
        if (ke[mid].a < ev->pid[i] || (ke[mid].a == ev->pid[i] && ke[mid].b < tE[i]))
          lo = mid + 1;
        else
          hi = mid;
      }
      if (lo > 0 && ke[lo - 1].a == ev->pid[i] && ke[lo - 1].b > tS[i]) {
        /* the largest row among the kernels with that end */
        int64_t j = lo - 1;
        gate[i] = ke[j].row;
      }
    }
    /* host order of a thread: ops and launches, (thread, ts', ops before
     * launches, ops by te' down, row) */
    nh = 0;
    for (int64_t i = 0; i < n; ++i)
      if (adm[i] && ev->kind[i] != K_KERNEL) {
        hr[nh].a = (int64_t)ev->pid[i] * T + ev->lane[i];
        hr[nh].b = ts[i];
        hr[nh].c = ev->kind[i] == K_LAUNCH ? I64_MAX : -te[i];
        hr[nh].row = i;
        ++nh;
      }
    qsort(hr, (size_t)nh, sizeof(rec4), cmp_rec4);
    for (int64_t q = 0; q < nh; ++q) pos[hr[q].row] = q;
    for (int64_t q = 0; q < nh; ++q) {
      const int64_t x = hr[q].row, par = out->link[x];
      /* previous sibling: the nearest earlier record of the thread with the
       * same parent, not passing the parent itself */
      for (int64_t j = q - 1; j >= 0 && hr[j].a == hr[q].a; --j) {
        const int64_t y = hr[j].row;
        if (y == par) break;
        if (out->link[y] == par) {
          sib[x] = y;
          break;
        }
      }
      if (par >= 0) lastc[par] = x; /* later children overwrite earlier */
    }
    /* the walk, per process from its last-ending record */
    int64_t *zrow = (int64_t *)malloc(sizeof(int64_t) * (size_t)P);
    for (int q = 0; q < P; ++q) zrow[q] = -1;
    for (int64_t i = 0; i < n; ++i) {
      if (!adm[i]) continue;
      int64_t z = zrow[ev->pid[i]];
      if (z < 0 || tE[i] > tE[z] || (tE[i] == tE[z] && i > z)) zrow[ev->pid[i]] = i;
    }
    for (int q = 0; q < P; ++q) {
      if (zrow[q] < 0) continue;
      int64_t *cp = out->crit_proc + (int64_t)q * 8;
      int64_t x = zrow[q];
      int side = 1; /* 0: S(x), 1: E(x) */
      const int64_t tend = tE[x];
      for (;;) {
        out->crit_flags[x] |= (uint8_t)(side ? 2 : 1);
        const int64_t t = side ? tE[x] : tS[x];
        int64_t y = -1;
        int ys = 0, cat = -1;
        int64_t who = -1; /* the row an attributed step is charged to */
        const int k = ev->kind[x];
        if (side == 1) {
          if (k == K_LAUNCH && gate[x] >= 0 && tE[gate[x]] < tE[x]) {
            y = gate[x], ys = 1, cat = 3, who = x;
          } else if (k == K_CPU && lastc[x] >= 0 && tE[lastc[x]] <= tE[x]) {
            y = lastc[x], ys = 1, cat = 4, who = x;
          } else {
            y = x, ys = 0, cat = k == K_KERNEL ? 1 : k == K_LAUNCH ? 2 : 4, who = x;
          }
        } else if (k == K_KERNEL) {
          int64_t rel = I64_MIN;
          const int64_t kp = kprev[x], l = out->link[x];
          if (kp >= 0 && tE[kp] <= t) y = kp, ys = 1, rel = tE[kp], cat = 6, who = -1;
          if (l >= 0) {
            if (tE[l] <= t && tE[l] >= rel) y = l, ys = 1, rel = tE[l], cat = 5, who = -1;
            else if (tE[l] > t && tS[l] <= t && tS[l] >= rel) y = l, ys = 0, rel = tS[l], cat = 2, who = l;
          }
        } else {
          int64_t rel = I64_MIN;
          const int64_t par = out->link[x], sb = sib[x];
          if (par >= 0) y = par, ys = 0, rel = tS[par], cat = 4, who = par;
          if (sb >= 0 && tE[sb] <= t && tE[sb] >= rel) y = sb, ys = 1, rel = tE[sb], cat = 7, who = -1;
        }
        if (y < 0) {
          cp[0] = tend - t;
          break;
        }
        const int64_t ty = ys ? tE[y] : tS[y];
        cp[cat] += t - ty;
        if (who >= 0) out->crit_time[who] += t - ty;
        x = y;
        side = ys;
      }
    }
    free(zrow);
    free(tS);
    free(tE);
    free(kprev);
    free(sib);
    free(lastc);
    free(gate);
    free(pos);
    free(hr);
    free(ke);
  }

  /* 19. Graph replay separation (Section 6.1: graph replay hides the
   *     operator calls; graph identities and launch correlations separate
   *     the replays).  READING: a replay is one admitted launch and the
   *     kernels joined to it; its span runs from their first start to their
   *     last end (corrected, unclipped; INT64_MAX / INT64_MIN with none),
   *     reported for every admitted launch.  A kernel's graph node (a dense
   *     id the caller gives to each node of each captured graph, -1 for a
   *     kernel launched on its own) identifies the same operator across
   *     replays: per node, over admitted kernels joined to a launch, the
   *     count, sum, minimum and maximum of the duration te' - ts', and the
   *     sum of the offsets ts' - the replay's first start (its place along
   *     the replayed layer sequence). */
  if ((p->flags & 32u) != 0) {
    for (int64_t i = 0; i < n; ++i) {
      if (!adm[i] || ev->kind[i] != K_LAUNCH) continue;
      out->launch_first[i] = I64_MAX;
      out->launch_last[i] = I64_MIN;
    }
    for (int64_t i = 0; i < n; ++i) {
      if (!adm[i] || ev->kind[i] != K_KERNEL || out->link[i] < 0) continue;
      const int64_t l = out->link[i];
      if (ts[i] < out->launch_first[l]) out->launch_first[l] = ts[i];
      if (te[i] > out->launch_last[l]) out->launch_last[l] = te[i];
    }
    for (int q = 0; q < p->n_graph_nodes; ++q) {
      out->gn_count[q] = 0;
      out->gn_sum[q] = 0;
      out->gn_min[q] = I64_MAX;
      out->gn_max[q] = I64_MIN;
      out->gn_offset[q] = 0;
    }
    for (int64_t i = 0; i < n; ++i) {
      if (!adm[i] || ev->kind[i] != K_KERNEL || out->link[i] < 0 || ev->graph_node[i] < 0) continue;
      const int q = ev->graph_node[i];
      const int64_t d = te[i] - ts[i];
      out->gn_count[q]++;
      out->gn_sum[q] = wrap_add(out->gn_sum[q], d);
      if (d < out->gn_min[q]) out->gn_min[q] = d;
      if (d > out->gn_max[q]) out->gn_max[q] = d;
      out->gn_offset[q] = wrap_add(out->gn_offset[q], ts[i] - out->launch_first[out->link[i]]);
    }
  }

  for (int64_t ps = 0; ps < (int64_t)P * S; ++ps) free(runs[ps]);
  free(runs);
  free(nruns);
  free(kr);
  free(lr);
  free(ts);
  free(te);
  free(adm);
  return gw > out->gap_capacity ? -3 : 0;
}
