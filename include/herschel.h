/*
 * herschel.h -- C ABI of the MI355X trace-reconstruction library.
 *
 * The library reconstructs operator executions from one bounded profiling
 * window, the data-parallel core of the analyzer in "Herschel: Continuous
 * Optimization of Production LLM Inference through On-Demand Profiling".
 *
 *  - The records it consumes are the three kinds the profiler emits
 *    (Section 5.2, "Python calls and object fields" and "Host API calls and
 *    device activity"): CPU operator ranges with their native thread and
 *    entry/return times, host launch-API intervals carrying a correlation id,
 *    and device kernel records located by device stream and linked to their
 *    launch by the same correlation id.
 *  - Records are admitted to the window by their start time (Section 5.2,
 *    "Session transitions").
 *  - The results are the observations of Section 6.1 ("Operator execution and
 *    efficiency", "Execution progress and state") and of Figure "Key
 *    performance observations": kernel composition of each operator from
 *    call-to-kernel links, the operator span T_op (from the earliest start
 *    to the latest end of the op's kernels), idle intervals of the GPU activity (the idle
 *    evidence of the case study in Section 9.1), communication overlapped
 *    with computation measured as interval coverage, and cross-process waits.
 *  - Operator efficiency (Section 6.1): MFU, MBU and SOL = max(MFU, MBU) of
 *    each op from its operation count and logical bytes over T_op and the
 *    device peaks, and per op name the time that reaching a reference SOL
 *    would save (the time-weighted gap to the reference of Section 6.2).
 *
 * Every entry point takes DEVICE pointers for all arrays (events, params
 * arrays, outputs, workspace), enqueues its kernels on params->hip_stream,
 * waits for that stream once at the end and reads the counters back to form
 * the return code.  The library never allocates device memory, keeps no
 * pointer after it returns and is re-entrant given distinct workspaces.
 * Arithmetic is integer only (int64 nanoseconds); sums wrap modulo 2^64.
 */
#ifndef HERSCHEL_H
#define HERSCHEL_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Record kinds (Section 5.2). */
enum {
  HERSCHEL_CPU_OP = 0, /* a recorded Python call: native thread, entry and return time */
  HERSCHEL_LAUNCH = 1, /* a host API interval that submits device work; carries corr */
  HERSCHEL_KERNEL = 2  /* a device activity record: stream, start, end, corr, name */
};

/* Return codes.  Precedence when several apply:
 * EINVAL > EWORKSPACE (ETOOBIG) > EEVENT > EDEVICE > ECAPACITY. */
enum {
  HERSCHEL_OK = 0,
  HERSCHEL_EINVAL = -1,     /* a required pointer (events, params, outputs, counters) is NULL or a
                               parameter is out of range */
  HERSCHEL_EEVENT = -2,     /* an input row is invalid; counters->first_invalid = smallest such row */
  HERSCHEL_ECAPACITY = -3,  /* more gaps than gap_capacity; the first gap_capacity are written */
  HERSCHEL_EWORKSPACE = -4, /* workspace is NULL, not 256-byte aligned, or smaller than herschel_workspace_size() */
  HERSCHEL_EDEVICE = -5,    /* a HIP call failed or a device-side consistency check tripped */
  HERSCHEL_ETOOBIG = -6     /* herschel_trace_analyze_static: the call needs more than its static scratch */
};

/* Optional outputs (params.flags).  Timelines, gaps, the launch/kernel join,
 * the latency histogram and the per-name aggregates are always produced. */
#define HERSCHEL_OUT_CONTAIN 0x1u /* op nesting, launch->op, kernel->op, per-op aggregates */
#define HERSCHEL_OUT_OVERLAP 0x2u /* cross-stream overlap and class coverage */
#define HERSCHEL_OUT_WAITS 0x4u   /* GPU idle coinciding with CPU ops, by op name (Section 9.1) */
#define HERSCHEL_OUT_SOL 0x8u     /* operator efficiency: MFU, MBU, SOL, per-name hotness (Section 6.1);
                                     needs HERSCHEL_OUT_CONTAIN */
#define HERSCHEL_OUT_CRIT 0x10u   /* critical path (Section 6.1, execution progress and state);
                                     needs HERSCHEL_OUT_CONTAIN */
#define HERSCHEL_OUT_GRAPH 0x20u  /* graph replay separation (Section 6.1, operator execution);
                                     needs HERSCHEL_OUT_CONTAIN */
/* Not an output: repeated calls with equal arguments replay a captured HIP
 * graph of their launches (herschel_trace_analyze).  Off by default. */
#define HERSCHEL_REPLAY 0x100u

/* Implementation limits (checked; EINVAL when exceeded). */
#define HERSCHEL_MAX_PROCS 4096
#define HERSCHEL_MAX_STREAMS 64
#define HERSCHEL_MAX_THREADS 2048
#define HERSCHEL_MAX_WINDOW (1LL << 40)  /* W1 - W0 in ns (about 18 minutes) */
#define HERSCHEL_MAX_ABS_TIME (1LL << 62) /* |ts|, |te|, |W0|, |W1|, |clock offset| must be below */
#define HERSCHEL_MAX_NAMES (1 << 24)
#define HERSCHEL_MAX_WAIT_OP_NAMES 2048   /* n_op_names with HERSCHEL_OUT_WAITS */
#define HERSCHEL_MAX_ROWS (1LL << 30)      /* n must be below: overlap endpoints (two per kernel) are
                                              indexed with int32, radix look-back words hold 30-bit prefixes */

/* Input records as a structure of arrays, n rows, in any order (delivery
 * order).  37 bytes per row (+16 with HERSCHEL_OUT_SOL, +4 with HERSCHEL_OUT_GRAPH).  Row i is valid iff
 *   kind[i] in {CPU_OP, LAUNCH, KERNEL}, 0 <= pid[i] < n_procs,
 *   KERNEL: 0 <= lane < n_streams and 0 <= name < n_names,
 *   CPU_OP: 0 <= lane < n_threads and 0 <= name < n_op_names,
 *           and with HERSCHEL_OUT_SOL flops >= 0 and bytes >= 0,
 *   KERNEL with HERSCHEL_OUT_GRAPH: -1 <= graph_node < n_graph_nodes,
 *   LAUNCH: 0 <= lane < n_threads and name >= 0 (an API id),
 *   -2^62 < ts <= te < 2^62.
 * corr may be any int64 (an opaque per-process id, Section 5.2). */
typedef struct {
  const int64_t *ts;   /* start, ns on the process clock */
  const int64_t *te;   /* end, ns on the process clock */
  const int64_t *corr; /* correlation id, per process, any value; ignored for CPU_OP */
  const int32_t *pid;  /* process index */
  const int32_t *lane; /* KERNEL: device stream; CPU_OP / LAUNCH: native thread */
  const int32_t *name; /* KERNEL: kernel-name id; CPU_OP: op-name id; LAUNCH: API id */
  const uint8_t *kind; /* HERSCHEL_CPU_OP / _LAUNCH / _KERNEL */
  /* HERSCHEL_OUT_SOL only (else may be NULL): per CPU_OP row, the op's
   * floating-point operation count F and the logical bytes B it must move,
   * as the analyzer derives them from the call's arguments (Section 5.2,
   * "Python calls and object fields"); read at CPU_OP rows only. */
  const int64_t *flops;
  const int64_t *bytes;
  /* HERSCHEL_OUT_GRAPH only (else may be NULL): per KERNEL row, the node
   * of a captured graph that the kernel replays, as a dense id the caller
   * gives to each node of each captured graph (graph identity and node, as
   * activity records report them), or -1 for a kernel launched on its own;
   * read at KERNEL rows only. */
  const int32_t *graph_node;
} herschel_events;

/* A cross-process dependency edge (Figure "Key performance observations",
 * panel "Cross-process blocking"): the consumer's work waits on the
 * producer's.  Keyed by (process, correlation id) of the two kernels. */
typedef struct {
  int32_t prod_pid, cons_pid;
  int64_t prod_corr, cons_corr;
} herschel_edge;

typedef struct {
  int64_t window_begin, window_end; /* [W0, W1) on the corrected clock; 0 < W1-W0 <= 2^40 */
  int64_t gap_threshold;            /* a gap is emitted iff its length > gap_threshold */
  int32_t n_procs, n_streams, n_threads, n_names, n_op_names;
  const int64_t *clock_offset;  /* [n_procs] or NULL (all zero); corrected = raw - offset */
  const uint8_t *stream_class;  /* [n_streams] 0 compute, 1 comm, 2 copy; NULL = all compute */
  const herschel_edge *edges;   /* [n_edges]; may be NULL when n_edges == 0 */
  int64_t n_edges;
  uint32_t flags;               /* HERSCHEL_OUT_* */
  void *hip_stream;             /* hipStream_t to enqueue on; NULL = the null stream */
  void *workspace;              /* device scratch owned by the caller, 256-byte aligned (hipMalloc's are) */
  size_t workspace_bytes;
  /* HERSCHEL_OUT_SOL only: the device's peak compute (FLOP/s) and memory
   * bandwidth (B/s), both > 0, and per op name a reference SOL in parts per
   * million (>= 0; the SOL the same op reaches elsewhere, Section 9.4), or
   * NULL for no reference. */
  int64_t peak_flops, peak_bytes;
  const int64_t *ref_sol_ppm;   /* [n_op_names] or NULL */
  int32_t n_graph_nodes;        /* HERSCHEL_OUT_GRAPH only: graph node ids, >= 1 */
} herschel_params;

typedef struct {
  int64_t n_admitted[3];          /* admitted rows per kind (W0 <= ts' < W1) */
  int64_t n_outside_window;       /* rows not admitted */
  int64_t n_matched;              /* admitted kernels joined to an admitted launch */
  int64_t n_unmatched_kernels;    /* admitted kernels without a launch */
  int64_t n_unmatched_launches;   /* admitted launches with no kernel joined to them */
  int64_t n_dup_launch_corr;      /* extra admitted launches sharing a (pid, corr) */
  int64_t n_unattributed_kernels; /* matched kernels whose launch lies in no op (CONTAIN) */
  int64_t n_improper_nesting;     /* ops ending after their parent (CONTAIN) */
  int64_t n_negative_latency;     /* matched kernels starting before their launch */
  int64_t n_gaps_total;           /* gaps above the threshold (may exceed gap_capacity) */
  int64_t first_invalid;          /* smallest invalid row, -1 if none */
  int64_t device_status;          /* 0, or bits of internal device-side failures */
} herschel_counters;

/* Outputs.  Per-row arrays are indexed by input row.  Rows outside the
 * window get link = aux = -2.  For admitted rows:
 *   link: KERNEL -> row of its launch (-1 none); LAUNCH -> row of the innermost
 *         enclosing CPU op (-1 none); CPU_OP -> row of its parent op (-1 root)
 *   aux:  KERNEL -> row of the op its launch lies in (-1 none); LAUNCH -> number
 *         of kernels joined to it; CPU_OP -> nesting depth (0 for a root)
 * Without HERSCHEL_OUT_CONTAIN, the CPU_OP and LAUNCH link, the CPU_OP and
 * KERNEL aux are -1 and the op_* arrays are not touched.
 * op_* are written at admitted CPU_OP rows only: the inclusive aggregates of
 * the kernels attributed to the op or to any of its descendants; an op with
 * none gets (0, INT64_MAX, INT64_MIN, 0).  T_op = op_last - op_first.
 * Every pointer but counters may be NULL: that output is not written (and
 * the work only it needs is skipped), as are outputs whose HERSCHEL_OUT_*
 * flag is clear.  The batch workload of many traces, for example, wants
 * only the per-name aggregates, busy / idle, gaps and the latency histogram. */
typedef struct {
  int32_t *link, *aux;               /* [n] */
  int32_t *op_nkern;                 /* [n] */
  int64_t *op_first, *op_last;       /* [n] first kernel start, last kernel end (unclipped) */
  int64_t *op_ksum;                  /* [n] sum of kernel durations */
  int64_t *busy, *idle;              /* [n_procs * n_streams] */
  int64_t *pair_overlap;             /* [n_procs * n_streams * n_streams] (OVERLAP) */
  int64_t *class_busy;               /* [n_procs * 3] (OVERLAP) */
  int64_t *class_overlap;            /* [n_procs * 3 * 3] (OVERLAP) */
  int64_t *any_busy;                 /* [n_procs] (OVERLAP) */
  int64_t *name_count, *name_sum;    /* [n_names] */
  int64_t *name_min, *name_max;      /* [n_names]; empty names: INT64_MAX, INT64_MIN */
  int64_t *lat_hist;                 /* [64]: bin 0 for latency <= 0, else floor(log2)+1 */
  int64_t *edge_wait;                /* [n_edges]; INT64_MIN when unresolved */
  int32_t *edge_status;              /* [n_edges]; bit0 producer missing, bit1 consumer missing */
  int64_t gap_capacity;              /* entries available in the gap_* arrays */
  int32_t *gap_pid, *gap_stream;     /* [gap_capacity] */
  int64_t *gap_begin, *gap_end;      /* [gap_capacity] */
  uint8_t *gap_flags;                /* [gap_capacity] bit0 leading (at W0), bit1 trailing (at W1) */
  herschel_counters *counters;       /* device pointer */
  /* HERSCHEL_OUT_WAITS (the idle evidence of the case study in Section 9.1):
   * the GPU of process p is idle where no kernel of any of its streams covers
   * the time; its idle intervals are the maximal ones in [W0, W1) longer
   * than gap_threshold.  For op name o of process p, U(p, o) is the union of
   * its admitted ops' ranges [ts', min(te', W1)). */
  int64_t *dev_idle;                 /* [n_procs] total length of the idle intervals */
  int64_t *op_span;                  /* [n_procs * n_op_names] |U(p, o)| */
  int64_t *op_idle;                  /* [n_procs * n_op_names] |U(p, o) within the idle intervals| */
  /* HERSCHEL_OUT_SOL (Section 6.1, "Operator execution and efficiency"): an
   * admitted op is measured when it has kernels and T_op = op_last - op_first
   * > 0.  In parts per million, exact (integer arithmetic in 128 bits),
   * saturating at INT64_MAX:
   *   MFU = floor(10^15 F / (T_op peak_flops)), MBU = floor(10^15 B / (T_op peak_bytes)),
   *   SOL = max(MFU, MBU);
   * an unmeasured op gets -1 in all three.  Per op name o, over its measured
   * ops: the sums of F, B and T_op (wrapping), the SOL of those sums (-1
   * with no measured op), and the hotness, the sum over ops below the
   * name's reference ref of floor(T_op (ref - SOL) / ref): the time the
   * name's ops would save at the reference SOL. */
  int64_t *op_mfu, *op_mbu, *op_sol; /* [n], written at admitted CPU_OP rows only */
  int64_t *opn_flops, *opn_bytes;    /* [n_op_names] */
  int64_t *opn_time, *opn_sol;       /* [n_op_names] */
  int64_t *opn_hot;                  /* [n_op_names] ns */
  /* HERSCHEL_OUT_CRIT (Section 6.1, "Execution progress and state": the
   * submission, execution-order and synchronization dependencies that
   * identify the critical path).  Each admitted record x has a start event
   * at ts' and an end event at min(te', W1); each event is released by one
   * other event:
   *   a kernel's end by its start; a launch's end by the end of g, when the
   *   launch has no kernel of its own and g, the process's kernel ending last
   *   strictly inside the call (then the largest row), exists (a
   *   synchronizing call), else by its start; an op's end by its last
   *   child's end if that child ends no later, else by its start;
   *   a kernel's start by the later of the previous kernel of its stream's
   *   end (if by then) and its launch (its end if by then, else its start if
   *   by then), the launch on a tie; an op's or launch's start by the later
   *   of its previous sibling's end (if by then) and its parent's start, the
   *   sibling on a tie.
   * Children and siblings are ordered as the thread's containment (ts' up,
   * ops before launches, ops by te' down, row up).  A process's path runs
   * back from the end event of its last-ending record (largest end, then
   * row) to an event nothing releases; each step's time is charged to one
   * part and, for the first four parts, to one record. */
  int64_t *crit_time;                /* [n] time charged to each admitted row (0 off the path) */
  uint8_t *crit_flags;               /* [n] admitted rows: bit0 start on the path, bit1 end on the path */
  int64_t *crit_proc;                /* [n_procs * 8] per process: length, then kernel run, API time
                                        (a launch's interval, or the part before its kernel started),
                                        sync tail (after the releasing kernel), op self time, launch gap
                                        (launch end to kernel start), queue gap (previous kernel end to
                                        kernel start), host gap (sibling end to start); all zero for a
                                        process without admitted rows */
  /* HERSCHEL_OUT_GRAPH (Section 6.1: graph replay hides operator calls;
   * graph identities and launch correlations separate replays).  A replay
   * is an admitted launch and the kernels joined to it; per graph node, over
   * the admitted kernels of that node joined to a launch: count, sum,
   * minimum and maximum of te' - ts', and the sum of the offsets
   * ts' - launch_first of the kernel's launch (its place along the replayed
   * layer sequence).  Empty nodes: 0, 0, INT64_MAX, INT64_MIN, 0. */
  int64_t *launch_first, *launch_last; /* [n] at admitted launches: first start and last end of their
                                          kernels (INT64_MAX, INT64_MIN with none) */
  int64_t *gn_count, *gn_sum;        /* [n_graph_nodes] */
  int64_t *gn_min, *gn_max;          /* [n_graph_nodes] */
  int64_t *gn_offset;                /* [n_graph_nodes] */
  /* The per-name aggregates of the kernels, for the admitted CPU ops by op
   * name (no flag; each may be NULL): count, sum, min and max of the
   * unclipped te' - ts'; empty names: 0, 0, INT64_MAX, INT64_MIN. */
  int64_t *opname_count, *opname_sum;  /* [n_op_names] */
  int64_t *opname_min, *opname_max;    /* [n_op_names] */
} herschel_outputs;

/* Bytes of device workspace that herschel_trace_analyze needs for n rows
 * under params *p (only the sizes and limits in *p are read). */
int herschel_workspace_size(int64_t n, const herschel_params *p, size_t *bytes);

/* Reconstruct one window: n rows of ev under *p into *out.  Returns a
 * HERSCHEL_* code.  On EEVENT only counters->first_invalid is defined.
 * The work is ordered on p->hip_stream (it also runs on two library
 * streams that wait for, and are waited on by, that stream); the call
 * returns once the device has finished all of it.  A call that launches
 * its kernels directly learns that from pinned host memory that its last
 * kernel writes (one small block per calling thread and device, allocated
 * on the thread's first call and held until the process ends), so HIP may
 * report the stream's last commands, and events recorded among them, as
 * pending for a few microseconds more: synchronise the stream before
 * querying such events.  A replayed call synchronises with the stream.
 * With HERSCHEL_REPLAY in
 * params->flags, a call whose event columns, n, parameters (all but
 * hip_stream) and output pointers equal those of one of the last four such
 * argument sets captured on the device replays that call's captured HIP
 * graph (the buffers' contents may differ); without it every call launches
 * its kernels directly.  Calls overlapping from several host threads are
 * serialised while they enqueue. */
int herschel_trace_analyze(const herschel_events *ev, int64_t n, const herschel_params *p,
                           herschel_outputs *out);

/* Device memory, in bytes, of the static scratch that
 * herschel_trace_analyze_static uses in place of a caller's workspace (about
 * 330,000 rows with every output of a 4-stream trace). */
#define HERSCHEL_STATIC_SCRATCH_BYTES (64LL << 20)

/* For callers that cannot allocate device memory (serving loops, harnesses
 * that forbid allocation): herschel_trace_analyze with the same arguments and
 * results, except that p->workspace and p->workspace_bytes are ignored.  The
 * library's own scratch array (HERSCHEL_STATIC_SCRATCH_BYTES, one per device,
 * held until the process ends) serves as the workspace, every kernel runs on
 * p->hip_stream one after another, and the call allocates nothing: no device
 * memory, no streams, no events, no graphs.  Returns HERSCHEL_ETOOBIG (and
 * enqueues nothing) when herschel_workspace_size(n, p) exceeds the scratch.
 * Calls that overlap on one device share its scratch and race: the caller
 * must not issue a second call on a device before the first has returned.
 * Each call clears what it needs, so calls in sequence are independent. */
int herschel_trace_analyze_static(const herschel_events *ev, int64_t n, const herschel_params *p,
                                  herschel_outputs *out);

/* Reconstruct n_traces independent windows stored back to back in ev: trace
 * t holds rows [trace_offsets[t], trace_offsets[t+1]) (a HOST array of
 * n_traces + 1 entries) and uses p[t] and out[t] (HOST arrays of structs whose
 * pointers are device pointers).  Row indices in trace t's outputs are local
 * to the trace.  p[0].workspace must hold the largest herschel_workspace_size()
 * over the traces (each with its own p[t]); the workspace and stream of p[0]
 * are used for all traces, one after the other.
 * Returns the first non-OK code in trace order, or HERSCHEL_OK. */
int herschel_trace_analyze_batch(const herschel_events *ev, const int64_t *trace_offsets,
                                 int32_t n_traces, const herschel_params *p,
                                 herschel_outputs *out);

/* The batch of herschel_trace_analyze_batch over traces that stay in host
 * memory, streamed to the device in chunks of chunk_traces traces with
 * double-buffered uploads: while chunk c is analysed on p[0].hip_stream, chunk
 * c + 1 uploads on a copy stream of the library into the other staging set.
 *   host           HOST struct of HOST column pointers, all traces back to
 *                  back as in herschel_trace_analyze_batch; allocate them
 *                  pinned (hipHostMalloc) for the uploads to overlap the
 *                  analysis (pageable memory works, without overlap).  The
 *                  optional columns (flops, bytes, graph_node) are uploaded
 *                  when non-NULL.
 *   trace_offsets  HOST array of n_traces + 1 row offsets into the host columns.
 *   chunk_traces   traces per chunk (>= 1).
 *   staging        HOST array of two herschel_events whose pointers are DEVICE
 *                  buffers of staging_rows rows each (every column the host
 *                  holds); owned by the caller, overwritten by the call.
 *   p, out         as for herschel_trace_analyze_batch: n_traces entries;
 *                  p[0]'s workspace and stream serve every trace.
 * Returns HERSCHEL_EINVAL (nothing enqueued) for NULL pointers, offsets that
 * fall, a chunk with more rows than staging_rows or a staging set without
 * room for a column the host holds; otherwise the first non-OK code of a
 * chunk in trace order, after which no further chunk is analysed.  Returns
 * when every chunk analysed is done and no upload is in flight.  One call
 * at a time per process (the copy stream is shared; calls are serialized). */
int herschel_trace_analyze_chunked(const herschel_events *host, const int64_t *trace_offsets,
                                   int32_t n_traces, int32_t chunk_traces,
                                   const herschel_events *staging, int64_t staging_rows,
                                   const herschel_params *p, herschel_outputs *out);

const char *herschel_strerror(int code);

/* Diagnostics for benchmarks.  Stages of one analysis call.  INIT, PREP,
 * HIST and SORT (with the refine pass after it) run in this order on
 * params->hip_stream; after SORT the JOIN, EDGES and NAMES stages run on a
 * library stream (JOIN beside the refine pass; with OUT_WAITS the op-name
 * lanes' union after EDGES; with OUT_CRIT the kernels' critical-path
 * releases after NAMES), the TIMELINE, OVERLAP and WAITS stages on another
 * after the refine pass, while CONTAIN, OPAGG, SOL, CRIT and GRAPH follow on
 * params->hip_stream (with OUT_CRIT, OPAGG and SOL move to the end of the
 * TIMELINE stream, beside CRIT); FINAL waits for all of them. */
enum {
  HERSCHEL_STAGE_INIT = 0,     /* clear the workspace state and accumulating outputs */
  HERSCHEL_STAGE_PREP = 1,     /* validate, correct, admit, compact (one kernel) */
  HERSCHEL_STAGE_HIST = 2,     /* digit histograms and pass plans of the timeline and containment sorts */
  HERSCHEL_STAGE_NAMES = 3,    /* per-name and per-op-name tables, then kernel -> op */
  HERSCHEL_STAGE_SORT = 4,     /* radix passes shared by the sorts (the timeline and containment digits) */
  HERSCHEL_STAGE_TIMELINE = 5, /* busy/idle, gaps, coverage runs (one kernel) */
  HERSCHEL_STAGE_OVERLAP = 6,  /* group starts of the coverage-run endpoints and the sweep */
  HERSCHEL_STAGE_CONTAIN = 7,  /* op nesting and launch -> op */
  HERSCHEL_STAGE_JOIN = 8,     /* launch <-> kernel join by correlation table, latency */
  HERSCHEL_STAGE_OPAGG = 9,    /* inclusive per-op aggregates */
  HERSCHEL_STAGE_EDGES = 10,   /* dependency waits */
  HERSCHEL_STAGE_FINAL = 11,   /* counters and histogram totals */
  HERSCHEL_STAGE_WAITS = 12,   /* device-lane and op-name unions, idle coincidence (OUT_WAITS) */
  HERSCHEL_STAGE_SOL = 13,     /* operator efficiency and per-name hotness (OUT_SOL), after OPAGG */
  HERSCHEL_STAGE_CRIT = 14,    /* critical path (OUT_CRIT), after CONTAIN and the join */
  HERSCHEL_STAGE_GRAPH = 15,   /* graph replay separation (OUT_GRAPH), after CRIT */
  HERSCHEL_N_STAGES = 16
};

/* Record start_event / stop_event (hipEvent_t, created by the caller) on
 * the stream that stage `stage` runs on, around that stage of every
 * following analysis call in this process, for measuring one stage's device
 * time live (such calls launch their kernels directly, not from a captured
 * graph).  NULL events turn
 * the recording off.  Returns HERSCHEL_EINVAL for an unknown stage.  Not
 * thread-safe: meant for single-threaded benchmarks. */
int herschel_time_stage(int stage, void *start_event, void *stop_event);

/* Sort statistics of the last analysis call made with this workspace and
 * these params, for computing the bytes the radix passes must move: waits
 * for params->hip_stream, then writes, for s = 0 timeline, 1 join,
 * 2 containment sort: out[3 * s + 0] = its keys, out[3 * s + 1] = bit mask
 * of the digits that no pass moved (bit d: every key agreed on digit d, or
 * digit d was left to the refine pass that orders keys equal above it; bit
 * 31 is set in the second case), out[3 * s + 2] = its digits.  Digits above
 * digit 0 are 8 bits wide; digit 0 is 8 bits, or, when it is left to the
 * refine pass, the 8 to 14 bits below the passes' 8-bit digits.  out
 * must hold 9 entries (host memory).  Returns HERSCHEL_EINVAL for NULL
 * arguments, no workspace or an invalid window or size, HERSCHEL_EDEVICE
 * when the copy fails. */
int herschel_sort_stats(const herschel_params *p, int32_t *out);

#ifdef __cplusplus
}
#endif

#endif /* HERSCHEL_H */
