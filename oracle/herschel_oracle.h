/*
 * herschel_oracle.h -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow CPU reference for the trace-reconstruction results of the
 * Herschel analyzer (Section 6.1 of the paper).  Only the tests, the smoke
 * check and the CPU baseline of the benchmark use it; the product library
 * never links or calls it.  It shares no code or header with the product:
 * these declarations are written separately, with host pointers throughout.
 *
 * Parity status: every function is pinned by the tests (hand-built worked
 * timeline, per-nanosecond brute force on tiny traces, invariants and
 * generator ground truth); see the header of herschel_oracle.c.
 */
#ifndef HERSCHEL_ORACLE_H
#define HERSCHEL_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  const int64_t *ts, *te, *corr;
  const int32_t *pid, *lane, *name;
  const uint8_t *kind;
  const int64_t *flops, *bytes; /* per CPU op (flags bit 3); may be NULL otherwise */
  const int32_t *graph_node;    /* per kernel (flags bit 5): node of a captured graph, -1 none */
} hro_events;

typedef struct {
  int32_t prod_pid, cons_pid;
  int64_t prod_corr, cons_corr;
} hro_edge;

typedef struct {
  int64_t w0, w1, thr;
  int32_t n_procs, n_streams, n_threads, n_names, n_op_names;
  const int64_t *clock_offset; /* may be NULL */
  const uint8_t *stream_class; /* may be NULL */
  const hro_edge *edges;
  int64_t n_edges;
  uint32_t flags; /* bit0: containment, bit1: overlap, bit2: idle coincidence, bit3: SOL */
  int64_t peak_flops, peak_bytes;   /* per second (bit 3) */
  const int64_t *ref_sol_ppm;       /* [n_op_names] or NULL (bit 3) */
  int32_t n_graph_nodes;            /* (bit 5) */
} hro_params;

typedef struct {
  int64_t n_admitted[3], n_outside_window, n_matched, n_unmatched_kernels,
      n_unmatched_launches, n_dup_launch_corr, n_unattributed_kernels,
      n_improper_nesting, n_negative_latency, n_gaps_total, first_invalid,
      device_status;
} hro_counters;

typedef struct {
  int32_t *link, *aux, *op_nkern;
  int64_t *op_first, *op_last, *op_ksum;
  int64_t *busy, *idle, *pair_overlap, *class_busy, *class_overlap, *any_busy;
  int64_t *name_count, *name_sum, *name_min, *name_max, *lat_hist;
  int64_t *edge_wait;
  int32_t *edge_status;
  int64_t gap_capacity;
  int32_t *gap_pid, *gap_stream;
  int64_t *gap_begin, *gap_end;
  uint8_t *gap_flags;
  hro_counters *counters;
  int64_t *dev_idle;        /* [n_procs] (flags bit 2) */
  int64_t *op_span, *op_idle; /* [n_procs * n_op_names] (flags bit 2) */
  int64_t *op_mfu, *op_mbu, *op_sol; /* [n] ppm at CPU_OP rows (flags bit 3) */
  int64_t *opn_flops, *opn_bytes, *opn_time, *opn_sol, *opn_hot; /* [n_op_names] (flags bit 3) */
  int64_t *crit_time;    /* [n] critical-path time attributed to each admitted row (flags bit 4) */
  uint8_t *crit_flags;   /* [n] bit0: the row's start event on the path, bit1: its end event (bit 4) */
  int64_t *crit_proc;    /* [n_procs * 8] length, kernel, api, sync, op, launch gap, queue gap, host gap */
  int64_t *launch_first, *launch_last; /* [n] at admitted launches: span of their kernels (bit 5) */
  int64_t *gn_count, *gn_sum, *gn_min, *gn_max, *gn_offset; /* [n_graph_nodes] (bit 5) */
  int64_t *opname_count, *opname_sum, *opname_min, *opname_max; /* [n_op_names], each may be NULL */
} hro_outputs;

/* Same return codes as the product: 0 ok, -1 bad parameter, -2 invalid row,
 * -3 gap capacity exceeded. */
int herschel_oracle_analyze(const hro_events *ev, int64_t n, const hro_params *p,
                            hro_outputs *out);

#ifdef __cplusplus
}
#endif

#endif
