// C ABI of the trace analyzer: argument checks, workspace layout, the order
// of the stages on the caller's stream, and the return code.
#include <string.h>

#include <chrono>
#include <cstddef>
#include <cstdio>
#include <mutex>
#include <vector>

#include <stdlib.h>

#include "internal.hpp"

namespace hx {

int names_block_count(int64_t n_max, int NN);
int names_lds_limit();

static int bits_host(uint64_t x) {
  int b = 0;
  while (x) {
    ++b;
    x >>= 1;
  }
  return b;
}

// ---------------------------------------------------------------- layout
static size_t align_up(size_t x) { return (x + 255) & ~(size_t)255; }

struct Bump {
  char* base;
  size_t off = 0;
  template <class T>
  T* take(int64_t count) {
    T* p = base ? (T*)(base + off) : nullptr;
    off = align_up(off + (size_t)std::max<int64_t>(count, 1) * sizeof(T));
    return p;
  }
};

// Sorts the call runs: the timeline always, containment and the two
// idle-coincidence sorts with their outputs.
static bool sort_used(const Ctx& c, const SortBufs* s) {
  if (s == &c.sK) return true;
  if (s == &c.sC) return c.contain;
  if (s == &c.sE) return c.crit;
  return c.waits;
}

// refine: whether the lowest bits are left to the refine pass (keys wider
// than 32 bits, whose low bits are nanoseconds: runs of keys equal above
// them are short)
static void sort_plan(SortBufs& s, int id, int64_t n_max, int key_bits, bool refine) {
  s.id = id;
  s.n_max = n_max;
  s.tiles_max = cdiv(std::max<int64_t>(n_max, 1), RS_TILE);
  sort_digits(key_bits, refine, &s.nd, &s.first, &s.sh1);
}

size_t layout_workspace(Ctx& c, char* base) {
  Bump b{base};
  const int64_t n = std::max<int64_t>(c.n, 1);
  c.ds = b.take<DevState>(1);
  // region cleared by the init kernel
  c.zero_begin = base ? base + b.off : nullptr;
  const size_t z0 = b.off;
  c.prep_tiles = cdiv(c.n, prep_tile_rows());
  c.prep_status = b.take<uint64_t>(4 * std::max<int64_t>(c.prep_tiles, 1));
  c.union_tiles = std::max<int64_t>(cdiv(n, union_tile_elems()), 1);
  c.union_status = b.take<uint64_t>(3 * c.union_tiles);
  // key widths (also reported by herschel_sort_stats)
  sort_plan(c.sK, SORT_K, n, c.pb + c.sb + c.wb, true);
  sort_plan(c.sC, SORT_C, n, c.pb + c.tb + c.wb + 1, true);
  if (c.waits) {
    sort_plan(c.sD, SORT_D, n, c.pb + c.wb, true);
    sort_plan(c.sO, SORT_O, n, c.pb + c.nob + c.wb, true);
    c.union_status_d = b.take<uint64_t>(3 * c.union_tiles);
    c.union_status_o = b.take<uint64_t>(3 * c.union_tiles);
    c.dg_cap = n + c.P;  // idle intervals: at most one more per process than kernels
    c.dg_tiles = std::max<int64_t>(cdiv(c.dg_cap, 4096), 1);
    c.dg_status = b.take<uint64_t>(c.dg_tiles);
    c.dbusy_ws = b.take<int64_t>(c.P);
  }
  if (c.sol) c.sol_tot = b.take<uint64_t>((int64_t)c.NOP * 4);
  if (c.crit) {
    sort_plan(c.sE, SORT_E, n, c.pb + c.wb1, true);
    c.crit_mark = b.take<uint8_t>(2 * n);
    c.crit_lastc1 = b.take<uint32_t>(n);
    c.crit_hasnext = b.take<uint8_t>(n);
    c.crit_zmax = b.take<uint64_t>(c.P);
    c.crit_zrow1 = b.take<uint32_t>(c.P);
  }
  if (c.contain) {
    c.vb_tiles = std::max<int64_t>(cdiv(n, 4096), 1);
    c.vb_status = b.take<uint64_t>(c.vb_tiles);
    // pyramid levels above the tile maxima: built by atomic maxima, from zero
    c.nlev = 3;
    while (cdiv(n, (int64_t)1 << (6 * (c.nlev - 1))) > 64) ++c.nlev;
    for (int l = 3; l < c.nlev; ++l) {
      c.Mn[l] = cdiv(n, (int64_t)1 << (6 * l));
      c.M[l] = b.take<uint64_t>(c.Mn[l]);
    }
  }
  c.zero_bytes = align_up(b.off - z0);
  // the first digit's look-back words are cleared by the histogram kernel
  // (for the tiles of the call), each later digit's by the pass before it
  for (SortBufs* s : {&c.sK, &c.sC, &c.sD, &c.sO, &c.sE}) {
    if (!sort_used(c, s)) continue;
    s->status0 = b.take<uint32_t>(s->tiles_max * RS_LB_WORDS);
    s->status1 = b.take<uint32_t>((int64_t)std::max(s->nd - 1, 1) * s->tiles_max * RS_LB_WORDS);
  }
  c.hist_part = b.take<uint32_t>((int64_t)N_SORTS * HIST_MAX_BLOCKS * 8 * 256);
  c.k_rows = b.take<uint32_t>(n);
  // the join: prep's list, the correlation table (two slots per row bound
  // every dense id range it accepts; hashed slots use the power of two
  // above), each entry's hashed slot and the fix-up list
  c.jkey = b.take<uint64_t>(n);
  c.jrow = b.take<uint32_t>(n);
  c.jslot = b.take<uint32_t>(n);
  c.jt_cap = 2 * n;
  c.jt_hsize = 64;
  while (c.jt_hsize < c.jt_cap) c.jt_hsize <<= 1;
  c.jt_L = b.take<uint32_t>(c.jt_hsize);
  c.jt_K = b.take<uint32_t>(c.jt_hsize);
  c.jt_C = b.take<uint32_t>(c.jt_hsize);
  if (c.p.n_edges > 0) {
    c.jt_kmax = b.take<int64_t>(c.jt_hsize);
    c.jt_kmin = b.take<int64_t>(c.jt_hsize);
  }
  c.jt_fix_cap = n;
  c.jt_fix = b.take<uint32_t>(3 * c.jt_fix_cap);
  // sort buffers
  for (SortBufs* s : {&c.sK, &c.sC, &c.sD, &c.sO, &c.sE}) {
    if ((s == &c.sD || s == &c.sO) && !c.waits) continue;
    if (s == &c.sE && !c.crit) continue;
    if (s == &c.sC && !c.contain) {
      // the containment list is still compacted by prep (ops and launches)
      s->k[0] = b.take<uint64_t>(n);
      s->v[0] = b.take<uint32_t>(n);
      continue;
    }
    s->k[0] = b.take<uint64_t>(n);
    s->k[1] = b.take<uint64_t>(n);
    s->v[0] = b.take<uint32_t>(n);
    s->v[1] = b.take<uint32_t>(n);
  }
  if (c.overlap) {
    c.ev_cap = 2 * n;
    c.ev_keys = b.take<uint64_t>(c.ev_cap);
    c.seg_off = b.take<int32_t>((int64_t)c.P * c.S + 1);
  }
  if (c.contain) {
    c.V = b.take<uint64_t>(n);
    c.M[0] = nullptr;
    c.Mn[0] = n;
    for (int l = 1; l < 3; ++l) {
      c.Mn[l] = cdiv(n, (int64_t)1 << (6 * l));
      c.M[l] = b.take<uint64_t>(c.Mn[l]);
    }
    c.pmt = b.take<uint64_t>(c.vb_tiles);
    c.par = b.take<int32_t>(n);
    c.lk_first = b.take<int64_t>(n);
    c.lk_last = b.take<int64_t>(n);
    c.lk_sum = b.take<int64_t>(n);
    c.ag_tiles = cdiv(n, AG_TILE);
    c.ag_chain = b.take<int32_t>(c.ag_tiles * AG_CHAIN);
    c.ag_nchain = b.take<int32_t>(c.ag_tiles);
    // the per-row links stand in for NULL link / aux outputs: containment reads them back
    c.link_ws = b.take<int32_t>(n);
    c.aux_ws = b.take<int32_t>(n);
  }
  c.busy_ws = b.take<int64_t>((int64_t)c.P * c.S);
  if (c.waits) {
    c.dg_pid = b.take<int32_t>(c.dg_cap);
    c.dg_begin = b.take<int64_t>(c.dg_cap);
    c.dg_end = b.take<int64_t>(c.dg_cap);
    c.dg_pre = b.take<int64_t>(c.dg_cap);
    c.dg_key = b.take<uint64_t>(c.dg_cap);
    c.oev_cap = 2 * n;
    c.oev = b.take<uint64_t>(c.oev_cap);
    c.op_span_ws = b.take<int64_t>((int64_t)c.P * c.NOP);
  }
  c.opn_blocks = opnames_block_count(n, c.NOP);
  if (opnames_use_tables(c.NOP)) c.opn_part = b.take<uint64_t>((int64_t)c.opn_blocks * c.NOP * 4);
  c.name_blocks = names_block_count(n, c.NN);
  if (c.NN <= names_lds_limit()) c.name_part = b.take<uint64_t>((int64_t)c.name_blocks * c.NN * 4);
  if (c.sol) {
    c.sol_blocks = sol_block_count(n, c.NOP);
    if (sol_uses_tables(c.NOP)) c.sol_part = b.take<uint64_t>((int64_t)c.sol_blocks * c.NOP * 4);
    c.op_nkern_ws = b.take<int32_t>(n);
    c.op_first_ws = b.take<int64_t>(n);
    c.op_last_ws = b.take<int64_t>(n);
  }
  if (c.graph) {
    c.graph_blocks = graph_block_count(n, c.NG);
    if (graph_uses_tables(c.NG)) c.graph_part = b.take<uint64_t>((int64_t)c.graph_blocks * c.NG * 5);
  }
  if (c.crit) {
    c.crit_pred = b.take<int32_t>(2 * n);
    c.crit_code = b.take<uint8_t>(2 * n);
    c.crit_ptr[0] = b.take<int32_t>(2 * n);
    c.crit_ptr[1] = b.take<int32_t>(2 * n);
  }
  return b.off;
}

// ------------------------------------------------------------ init, final
struct InitArgs {
  DevState* ds;
  uint4* zero;
  int64_t zero_n;  // 16-byte words
  herschel_counters* cnt;
  int64_t* busy;
  int nps;
  int64_t* lat_hist;
  bool overlap;
  int64_t* pair;
  int64_t* class_busy;
  int64_t* class_overlap;
  int64_t* any_busy;
  int P, S;
  int NN;
  int64_t* name_count;
  int64_t* name_sum;
  int64_t* name_min;
  int64_t* name_max;
  const int64_t* off;
  const uint8_t* cls;
  int64_t n_opn;      // P * n_op_names with the idle-coincidence outputs, else 0
  int64_t n_crit;     // P * 8 with the critical path, else 0
  int64_t* crit_proc;
  int NOP;
  int64_t* opn[4];    // per op name: count, sum, min, max (each may be NULL)
  int64_t n_gn;       // graph nodes with the graph replay outputs, else 0
  int64_t* gn[5];     // count, sum, min, max, offset (each may be NULL)
  int64_t* op_span;
  int64_t* op_idle;
};

// The device state is cleared up to its digit offsets (the plan kernel
// writes those whole, after this; the last 16-byte word may reach into
// them), 16 bytes a thread over the grid; the word of the smallest invalid
// row starts at INT64_MAX.  The status word lies in the first workgroup's
// share, so its parameter check follows the clearing.
constexpr int64_t DS_CLEAR = ((int64_t)offsetof(DevState, hist) + 15) / 16;
constexpr int64_t DS_FI = (int64_t)offsetof(DevState, first_invalid);
static_assert(DS_CLEAR * 16 <= (int64_t)sizeof(DevState) && DS_FI % 8 == 0, "16-byte clearing of the device state");
static_assert(alignof(DevState) >= 8, "the device state starts the 256-byte aligned workspace");
static_assert(offsetof(DevState, status) < 256 * 16, "the status word is cleared by the first workgroup");

__global__ __launch_bounds__(256) void k_init(InitArgs a) {
  const int64_t tid = (int64_t)blockIdx.x * 256 + threadIdx.x, nth = (int64_t)gridDim.x * 256;
  for (int64_t i = tid; i < a.zero_n; i += nth) a.zero[i] = make_uint4(0, 0, 0, 0);
  for (int64_t i = tid; i < DS_CLEAR; i += nth) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (i == DS_FI / 16) {
      if (DS_FI % 16 == 0) {
        v.x = 0xffffffffu;
        v.y = 0x7fffffffu;
      } else {
        v.z = 0xffffffffu;
        v.w = 0x7fffffffu;
      }
    }
    reinterpret_cast<uint4*>(a.ds)[i] = v;
  }
  if (blockIdx.x == 0) {
    __syncthreads();
    int64_t* cz = (int64_t*)a.cnt;
    for (int i = threadIdx.x; i < (int)(sizeof(herschel_counters) / 8); i += 256) cz[i] = 0;
    if (a.lat_hist && threadIdx.x < 64) a.lat_hist[threadIdx.x] = 0;
    bool bad = false;
    if (a.off)
      for (int q = threadIdx.x; q < a.P; q += 256)
        bad |= !(a.off[q] > -HERSCHEL_MAX_ABS_TIME && a.off[q] < HERSCHEL_MAX_ABS_TIME);
    if (a.cls)
      for (int s = threadIdx.x; s < a.S; s += 256) bad |= a.cls[s] > 2;
    if (bad) atomicOr(&a.ds->status, DS_PARAM);
  }
  for (int64_t i = tid; i < a.nps; i += nth) a.busy[i] = 0;
  if (a.overlap) {
    if (a.pair)
      for (int64_t i = tid; i < (int64_t)a.nps * a.S; i += nth) a.pair[i] = 0;
    if (a.class_busy)
      for (int64_t i = tid; i < (int64_t)a.P * 3; i += nth) a.class_busy[i] = 0;
    if (a.class_overlap)
      for (int64_t i = tid; i < (int64_t)a.P * 9; i += nth) a.class_overlap[i] = 0;
    if (a.any_busy)
      for (int64_t i = tid; i < a.P; i += nth) a.any_busy[i] = 0;
  }
  // the name outputs start as the identities: the per-block tables (or,
  // with many names, the kernels themselves) are combined into them with
  // atomics
  for (int64_t i = tid; i < a.n_crit; i += nth) a.crit_proc[i] = 0;  // accumulated with atomics
  for (int64_t i = tid; i < a.NOP; i += nth) {  // combined with atomics
    if (a.opn[0]) a.opn[0][i] = 0;
    if (a.opn[1]) a.opn[1][i] = 0;
    if (a.opn[2]) a.opn[2][i] = I64MAX;
    if (a.opn[3]) a.opn[3][i] = I64MIN;
  }
  for (int64_t i = tid; i < a.n_gn; i += nth) {  // combined with atomics
    if (a.gn[0]) a.gn[0][i] = 0;
    if (a.gn[1]) a.gn[1][i] = 0;
    if (a.gn[2]) a.gn[2][i] = I64MAX;
    if (a.gn[3]) a.gn[3][i] = I64MIN;
    if (a.gn[4]) a.gn[4][i] = 0;
  }
  for (int64_t i = tid; i < a.n_opn; i += nth) {  // accumulated with atomics
    if (a.op_span) a.op_span[i] = 0;
    if (a.op_idle) a.op_idle[i] = 0;
  }
  for (int64_t i = tid; i < a.NN; i += nth) {
    if (a.name_count) a.name_count[i] = 0;
    if (a.name_sum) a.name_sum[i] = 0;
    if (a.name_min) a.name_min[i] = I64MAX;
    if (a.name_max) a.name_max[i] = I64MIN;
  }
}

void launch_init(Ctx& c) {
  InitArgs a;
  a.ds = c.ds;
  a.zero = (uint4*)c.zero_begin;
  a.zero_n = (int64_t)(c.zero_bytes / 16);
  a.cnt = c.o.counters;
  a.busy = c.o.busy ? c.o.busy : c.busy_ws;
  a.nps = c.P * c.S;
  a.lat_hist = c.o.lat_hist;
  a.overlap = c.overlap;
  a.pair = c.o.pair_overlap;
  a.class_busy = c.o.class_busy;
  a.class_overlap = c.o.class_overlap;
  a.any_busy = c.o.any_busy;
  a.P = c.P;
  a.S = c.S;
  a.NN = c.NN;
  a.name_count = c.o.name_count;
  a.name_sum = c.o.name_sum;
  a.name_min = c.o.name_min;
  a.name_max = c.o.name_max;
  a.off = c.p.clock_offset;
  a.cls = c.p.stream_class;
  a.n_opn = c.waits ? (int64_t)c.P * c.NOP : 0;
  a.n_crit = c.crit && c.o.crit_proc ? (int64_t)c.P * 8 : 0;
  a.crit_proc = c.o.crit_proc;
  a.NOP = c.NOP;
  a.opn[0] = c.o.opname_count;
  a.opn[1] = c.o.opname_sum;
  a.opn[2] = c.o.opname_min;
  a.opn[3] = c.o.opname_max;
  a.n_gn = c.graph ? c.NG : 0;
  a.gn[0] = c.o.gn_count;
  a.gn[1] = c.o.gn_sum;
  a.gn[2] = c.o.gn_min;
  a.gn[3] = c.o.gn_max;
  a.gn[4] = c.o.gn_offset;
  a.op_span = c.o.op_span ? c.o.op_span : c.op_span_ws;
  a.op_idle = c.o.op_idle;
  const int64_t work =
      std::max<int64_t>({a.zero_n, (int64_t)a.nps * (c.overlap ? c.S : 1), (int64_t)c.NN, a.n_opn, a.n_gn,
                         (int64_t)c.NOP, DS_CLEAR, 1});
  const int grid = (int)std::min<int64_t>(std::max<int64_t>(cdiv(work, 256 * 2), 8), 2048);
  hipLaunchKernelGGL(k_init, dim3(std::max(grid, 1)), dim3(256), 0, c.st, a);
}

// Without containment, admitted ops and launches have no op links (either
// output may be NULL).
__global__ __launch_bounds__(256) void k_nocontain(const uint64_t* keys, const uint32_t* rows, DevState* ds,
                                                    int32_t* link, int32_t* aux) {
  const int64_t n = ds->nCL;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const uint32_t r = rows[i];
    if (link) link[r] = -1;
    if (aux && (keys[i] & 1) == 0) aux[r] = -1;
  }
}

// Exits the critical path's walk follows per process before the doubling
// pass takes over ($HERSCHEL_CRIT_WALK, for tests of that pass; 64 by default).
static int crit_walk_max() {
  const char* e = getenv("HERSCHEL_CRIT_WALK");
  if (!e || !*e) return 64;
  const long v = strtol(e, nullptr, 10);
  return v < 0 ? 0 : v > (1L << 20) ? (1 << 20) : (int)v;
}

__global__ __launch_bounds__(256) void k_finalize(DevState* ds, herschel_counters* cnt, int64_t* lat_hist,
                                                  const int64_t* busy, int64_t* idle, int nps, int64_t W,
                                                  Mailbox* mb, int64_t seq) {
  if (idle)
    for (int i = threadIdx.x; i < nps; i += 256) idle[i] = W - busy[i];
  // join counts and latency bins from their accumulator copies
  if (threadIdx.x < JC_N + 64) {
    unsigned long long v = 0;
#pragma unroll
    for (int k = 0; k < JOIN_COPIES; ++k) v += ds->join_acc[k][threadIdx.x];
    if (threadIdx.x >= JC_N) {
      if (v && lat_hist) lat_hist[threadIdx.x - JC_N] += (int64_t)v;
    } else {
      int64_t* dst = nullptr;
      int64_t val = (int64_t)v;
      switch (threadIdx.x) {
        case JC_MATCHED: dst = &cnt->n_matched; break;
        case JC_UNM_K: dst = &cnt->n_unmatched_kernels; break;
        case JC_DUP: dst = &cnt->n_dup_launch_corr; break;
        case JC_NEG: dst = &cnt->n_negative_latency; break;
        case JC_UNATTR: dst = &cnt->n_unattributed_kernels; break;
        default:  // JC_MLAUNCH: the unmatched launches are the others
          dst = &cnt->n_unmatched_launches;
          val = cnt->n_admitted[HERSCHEL_LAUNCH] - val;
          break;
      }
      *dst = val;
    }
  }
  if (threadIdx.x == 0) {
    cnt->first_invalid = ds->first_invalid == I64MAX ? -1 : ds->first_invalid;
    cnt->device_status = ds->status;
  }
  if (!mb) return;
  // the counters to the calling thread's mailbox, then the sequence number
  // with a release at system scope: the host that reads the number reads
  // this call's counters
  __syncthreads();
  if (threadIdx.x < (int)(sizeof(herschel_counters) / 8)) {
    const int64_t v = ((const int64_t*)cnt)[threadIdx.x];
    __hip_atomic_store(&mb->c[threadIdx.x], v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
  if (threadIdx.x == 0)
    __hip_atomic_store(&mb->crit_more, (int64_t)ds->crit_more, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_store(&mb->seq, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

void launch_finalize(Ctx& c) {
  hipLaunchKernelGGL(k_finalize, dim3(1), dim3(256), 0, c.st, c.ds, c.o.counters, c.o.lat_hist,
                     c.o.busy ? c.o.busy : c.busy_ws, c.o.idle, c.P * c.S, c.W, c.mailbox, c.mailbox_seq);
}

// ------------------------------------------------------------- the call
static int check_and_plan(Ctx& c, const herschel_events* ev, int64_t n, const herschel_params* p,
                          const herschel_outputs* out) {
  if (!ev || !p || !out) return HERSCHEL_EINVAL;
  if (n < 0 || n >= (1LL << 30)) return HERSCHEL_EINVAL;
  if (n > 0 && (!ev->ts || !ev->te || !ev->corr || !ev->pid || !ev->lane || !ev->name || !ev->kind))
    return HERSCHEL_EINVAL;
  const int64_t W0 = p->window_begin, W1 = p->window_end;
  if (!(W0 > -HERSCHEL_MAX_ABS_TIME && W0 < HERSCHEL_MAX_ABS_TIME)) return HERSCHEL_EINVAL;
  if (!(W1 > -HERSCHEL_MAX_ABS_TIME && W1 < HERSCHEL_MAX_ABS_TIME)) return HERSCHEL_EINVAL;
  if (W1 <= W0 || W1 - W0 > HERSCHEL_MAX_WINDOW) return HERSCHEL_EINVAL;
  if (p->n_procs < 1 || p->n_procs > HERSCHEL_MAX_PROCS) return HERSCHEL_EINVAL;
  if (p->n_streams < 1 || p->n_streams > HERSCHEL_MAX_STREAMS) return HERSCHEL_EINVAL;
  if (p->n_threads < 1 || p->n_threads > HERSCHEL_MAX_THREADS) return HERSCHEL_EINVAL;
  if (p->n_names < 1 || p->n_names > HERSCHEL_MAX_NAMES) return HERSCHEL_EINVAL;
  if (p->n_op_names < 1) return HERSCHEL_EINVAL;
  if (p->n_edges < 0 || (p->n_edges > 0 && !p->edges)) return HERSCHEL_EINVAL;
  if (p->flags & ~(HERSCHEL_OUT_CONTAIN | HERSCHEL_OUT_OVERLAP | HERSCHEL_OUT_WAITS | HERSCHEL_OUT_SOL |
                   HERSCHEL_OUT_CRIT | HERSCHEL_OUT_GRAPH | HERSCHEL_REPLAY))
    return HERSCHEL_EINVAL;
  // graph replay separation reads the join's per-launch spans (kept with
  // containment), the kernels' nodes and their number
  if (p->flags & HERSCHEL_OUT_GRAPH) {
    if (!(p->flags & HERSCHEL_OUT_CONTAIN) || p->n_graph_nodes < 1) return HERSCHEL_EINVAL;
    if (n > 0 && !ev->graph_node) return HERSCHEL_EINVAL;
  }
  // the critical path walks the host nesting
  if ((p->flags & HERSCHEL_OUT_CRIT) && !(p->flags & HERSCHEL_OUT_CONTAIN)) return HERSCHEL_EINVAL;
  // operator efficiency reads the per-op aggregates of containment, the
  // ops' counts and the device's peaks
  if (p->flags & HERSCHEL_OUT_SOL) {
    if (!(p->flags & HERSCHEL_OUT_CONTAIN)) return HERSCHEL_EINVAL;
    if (p->peak_flops <= 0 || p->peak_bytes <= 0) return HERSCHEL_EINVAL;
    if (n > 0 && (!ev->flops || !ev->bytes)) return HERSCHEL_EINVAL;
  }
  // the op-name key (pid, name, ts') and its run endpoints must fit 64 bits
  if ((p->flags & HERSCHEL_OUT_WAITS) && p->n_op_names > HERSCHEL_MAX_WAIT_OP_NAMES) return HERSCHEL_EINVAL;
  const bool contain = (p->flags & HERSCHEL_OUT_CONTAIN) != 0, overlap = (p->flags & HERSCHEL_OUT_OVERLAP) != 0;
  // every output but the counters may be NULL: that output is skipped
  if (!out->counters) return HERSCHEL_EINVAL;
  if (out->gap_capacity < 0) return HERSCHEL_EINVAL;

  c.st = (hipStream_t)p->hip_stream;
  c.ev = *ev;
  c.n = n;
  c.p = *p;
  c.o = *out;
  c.W0 = W0;
  c.W1 = W1;
  c.W = W1 - W0;
  c.thr = p->gap_threshold;
  c.P = p->n_procs;
  c.S = p->n_streams;
  c.T = p->n_threads;
  c.NN = p->n_names;
  c.NOP = p->n_op_names;
  c.contain = contain;
  c.overlap = overlap;
  c.waits = (p->flags & HERSCHEL_OUT_WAITS) != 0;
  c.sol = (p->flags & HERSCHEL_OUT_SOL) != 0;
  c.crit = (p->flags & HERSCHEL_OUT_CRIT) != 0;
  c.crit_walk_max = crit_walk_max();
  c.graph = (p->flags & HERSCHEL_OUT_GRAPH) != 0;
  c.NG = c.graph ? p->n_graph_nodes : 0;
  c.nob = bits_host((uint64_t)(c.NOP - 1));
  c.pb = bits_host((uint64_t)(c.P - 1));
  c.sb = bits_host((uint64_t)(c.S - 1));
  c.tb = bits_host((uint64_t)(c.T - 1));
  c.wb = bits_host((uint64_t)(c.W - 1));
  c.wb1 = bits_host((uint64_t)c.W);
  c.vb = bits_host((uint64_t)c.W + 1);
  return HERSCHEL_OK;
}

// Stage timing for benchmarks (herschel_time_stage).
static int g_stage = -1;
static hipEvent_t g_ev0 = nullptr, g_ev1 = nullptr;
static inline void stage_begin(Ctx& c, int s) {
  if (s == g_stage && g_ev0) (void)hipEventRecord(g_ev0, c.st);
}
static inline void stage_end(Ctx& c, int s) {
  if (s == g_stage && g_ev1) (void)hipEventRecord(g_ev1, c.st);
}

// After the sorts three chains are independent and each is latency-bound,
// so they run side by side: the timeline, overlap and name tables on one
// library stream, the join on another, containment on the caller's stream,
// which then waits for both.  The library's streams and events are created
// once per device (default priority); enqueueing is serialised so that
// concurrent callers cannot interleave their event records.
struct DeviceStreams {
  hipStream_t s[2] = {nullptr, nullptr};
  hipStream_t cap = nullptr;  // graphs are captured here (the caller's stream may be the null stream)
  hipEvent_t e[9] = {};  // sorts, timeline chain, join, launches' ops, name tables, radix passes, depths,
                         // kernels' critical-path releases, op-name lanes' union
  hipStream_t copy = nullptr;  // uploads of the chunked entry point
  hipEvent_t up[2] = {};       // a staging set's upload done
  bool ok = false;
};
static std::mutex g_enqueue_mutex;
static DeviceStreams g_dev_streams[64];

static DeviceStreams* device_streams() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  DeviceStreams& d = g_dev_streams[dev];
  if (!d.ok) {
    for (auto& st : d.s)
      if (hipStreamCreateWithFlags(&st, hipStreamNonBlocking) != hipSuccess) return nullptr;
    if (hipStreamCreateWithFlags(&d.cap, hipStreamNonBlocking) != hipSuccess) return nullptr;
    if (hipStreamCreateWithFlags(&d.copy, hipStreamNonBlocking) != hipSuccess) return nullptr;
    for (auto& ev : d.e)
      if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) return nullptr;
    for (auto& ev : d.up)
      if (hipEventCreateWithFlags(&ev, hipEventDisableTiming) != hipSuccess) return nullptr;
    d.ok = true;
  }
  return &d;
}

static bool env_flag(const char* name, bool dflt) {
  const char* e = getenv(name);
  if (!e || !e[0]) return dflt;
  return e[0] != '0';
}

// Enqueues one call's kernels (the caller holds g_enqueue_mutex).  With
// HERSCHEL_SERIAL=1, or without library streams (dsx == nullptr, the
// entry point that allocates nothing), every chain runs on the caller's
// stream, one kernel after another, and no event is recorded.
static int enqueue_locked(Ctx& c, DeviceStreams* dsx) {
  static const bool serial_env = env_flag("HERSCHEL_SERIAL", false);
  const bool serial = serial_env || !dsx;
  const hipStream_t s0 = c.st;
  const hipStream_t lib0 = serial ? s0 : dsx->s[0], lib1 = serial ? s0 : dsx->s[1];
  // cross-stream edges (nothing to order when every chain is on one stream)
  auto rec = [&](int e, hipStream_t s) {
    if (!serial) (void)hipEventRecord(dsx->e[e], s);
  };
  auto wait = [&](hipStream_t s, int e) {
    if (!serial) (void)hipStreamWaitEvent(s, dsx->e[e], 0);
  };
  stage_begin(c, HERSCHEL_STAGE_INIT);
  launch_init(c);
  stage_end(c, HERSCHEL_STAGE_INIT);
  stage_begin(c, HERSCHEL_STAGE_PREP);
  launch_prep(c);
  if (c.crit) launch_crit_elist(c);  // the kernel-end list joins the sorts
  stage_end(c, HERSCHEL_STAGE_PREP);

  // The timeline and containment sorts share their digit passes, pass p of
  // a sort being its digit first + p (a sort whose digit is skipped has no
  // tiles in the launch); both leave their lowest digit to the refine pass.
  // The histogram launch also takes the correlation table's plan and empties
  // the table.  Nothing else runs beside the sorts: a large grid on another
  // stream would take the CUs first and hold up the passes, which every
  // later stage waits for.
  SortBufs* ss[N_SORTS];
  const int32_t* cc[N_SORTS];
  int ks = 0;
  ss[ks] = &c.sK;
  cc[ks++] = &c.ds->nK;
  if (c.contain) {
    ss[ks] = &c.sC;
    cc[ks++] = &c.ds->nCL;
  }
  if (c.waits) {  // the device lane and the op-name lanes
    ss[ks] = &c.sD;
    cc[ks++] = &c.ds->nK;
    ss[ks] = &c.sO;
    cc[ks++] = &c.ds->nO;
  }
  if (c.crit) {  // kernel ends, for the synchronizing calls of the critical path
    ss[ks] = &c.sE;
    cc[ks++] = &c.ds->nK;
  }
  int p_shared = 0;
  for (int i = 0; i < ks; ++i) p_shared = std::max(p_shared, ss[i]->nd - ss[i]->first);
  stage_begin(c, HERSCHEL_STAGE_HIST);
  launch_hist_multi(c, ss, cc, ks);
  stage_end(c, HERSCHEL_STAGE_HIST);
  stage_begin(c, HERSCHEL_STAGE_SORT);
  launch_sort_multi(c, ss, cc, ks, 0, p_shared);
  stage_end(c, HERSCHEL_STAGE_SORT);
  rec(5, s0);  // the join reads no sorted list: it starts beside the refine pass
  launch_refine(c);
  rec(0, s0);

  // chain 3 on the caller's stream, enqueued first: containment is the
  // longest of the three chains, and of work that becomes ready together
  // the first enqueued takes the CUs first
  c.st = s0;
  if (c.contain) {
    stage_begin(c, HERSCHEL_STAGE_CONTAIN);
    launch_contain(c);
    rec(3, s0);  // each launch's op is known
    launch_depth(c);
    if (c.crit) rec(6, s0);  // the per-op aggregates move beside the critical path
    stage_end(c, HERSCHEL_STAGE_CONTAIN);
  } else if (c.o.link || c.o.aux) {
    const int grid = (int)std::min<int64_t>(std::max<int64_t>(cdiv(c.n, 256 * 8), 1), 2048);
    hipLaunchKernelGGL(k_nocontain, dim3(grid), dim3(256), 0, c.st, c.sC.k[0], c.sC.v[0], c.ds, c.o.link, c.o.aux);
  }

  // chain 2: the join by the correlation table, then the dependency waits
  c.st = lib1;
  wait(c.st, 5);
  stage_begin(c, HERSCHEL_STAGE_JOIN);
  launch_join_table(c);
  stage_end(c, HERSCHEL_STAGE_JOIN);
  stage_begin(c, HERSCHEL_STAGE_EDGES);
  launch_edges(c);
  stage_end(c, HERSCHEL_STAGE_EDGES);
  rec(2, c.st);
  if (c.waits) {  // the op-name lanes' union, beside the timeline stream's device lane
    wait(c.st, 0);
    launch_union_opnames(c);
    rec(8, c.st);
  }
  // the per-name tables need neither the join nor containment; each kernel
  // takes its launch's op once the containment query has given launches
  // their ops
  stage_begin(c, HERSCHEL_STAGE_NAMES);
  launch_names(c);
  launch_names_reduce(c);
  wait(c.st, 0);  // the op-name tables read the refined containment list
  launch_opnames(c);
  if (c.contain) {
    wait(c.st, 3);
    launch_kernel_ops(c);
  }
  stage_end(c, HERSCHEL_STAGE_NAMES);
  if (c.crit) {  // the kernels' releases (the join and the timeline order), beside the host records'
    launch_crit_kernels(c);
    rec(7, c.st);
  }
  rec(4, c.st);

  // chain 1: timeline and overlap
  c.st = lib0;
  wait(c.st, 0);
  stage_begin(c, HERSCHEL_STAGE_TIMELINE);
  launch_timeline(c);
  stage_end(c, HERSCHEL_STAGE_TIMELINE);
  stage_begin(c, HERSCHEL_STAGE_OVERLAP);
  if (c.overlap) launch_overlap(c);
  stage_end(c, HERSCHEL_STAGE_OVERLAP);
  stage_begin(c, HERSCHEL_STAGE_WAITS);
  if (c.waits) {
    launch_union_device(c);
    launch_dg_scan(c);
    wait(c.st, 8);
    launch_waits(c);
  }
  stage_end(c, HERSCHEL_STAGE_WAITS);
  // with the critical path (which needs containment and the join, not the
  // per-op aggregates) the aggregates and what reads them run here, beside it
  const bool agg_side = c.crit && c.contain;
  if (agg_side) {
    wait(c.st, 6);
    wait(c.st, 2);
    stage_begin(c, HERSCHEL_STAGE_OPAGG);
    launch_opagg(c);
    stage_end(c, HERSCHEL_STAGE_OPAGG);
    stage_begin(c, HERSCHEL_STAGE_SOL);
    if (c.sol) launch_sol(c);
    stage_end(c, HERSCHEL_STAGE_SOL);
  }
  rec(1, c.st);

  // back on the caller's stream: what needs both containment and the join
  c.st = s0;
  wait(c.st, 2);
  if (!agg_side) {
    stage_begin(c, HERSCHEL_STAGE_OPAGG);
    if (c.contain) launch_opagg(c);
    stage_end(c, HERSCHEL_STAGE_OPAGG);
    stage_begin(c, HERSCHEL_STAGE_SOL);
    if (c.sol) launch_sol(c);
    stage_end(c, HERSCHEL_STAGE_SOL);
  }
  stage_begin(c, HERSCHEL_STAGE_CRIT);
  if (c.crit) {
    launch_crit_front(c);
    wait(c.st, 7);
    launch_crit(c);
  }
  stage_end(c, HERSCHEL_STAGE_CRIT);
  stage_begin(c, HERSCHEL_STAGE_GRAPH);
  if (c.graph) launch_graph(c);
  stage_end(c, HERSCHEL_STAGE_GRAPH);
  wait(c.st, 1);
  wait(c.st, 4);
  stage_begin(c, HERSCHEL_STAGE_FINAL);
  launch_finalize(c);
  stage_end(c, HERSCHEL_STAGE_FINAL);
  return hipGetLastError() == hipSuccess ? HERSCHEL_OK : HERSCHEL_EDEVICE;
}

static DeviceStreams* enqueue_setup() {
  static bool lds_attr = false;
  if (!lds_attr) {
    names_set_lds_attr();
    lds_attr = true;
  }
  return device_streams();
}

static int enqueue(Ctx& c) {
  std::lock_guard<std::mutex> lock(g_enqueue_mutex);
  DeviceStreams* dsx = enqueue_setup();
  if (!dsx) return HERSCHEL_EDEVICE;
  return enqueue_locked(c, dsx);
}

// With HERSCHEL_REPLAY in the flags, a call with exactly the arguments of
// an earlier one on this device (events, size, parameters except the
// stream, outputs) replays a HIP graph of that call's launches: about 35
// launches and the streams' event edges become one graph launch on the
// caller's stream.  Each device keeps the graphs of its last four distinct
// argument sets; any other call captures a new graph in place of the
// oldest.  The graph is captured on a private stream, so the caller's stream
// may be the null stream.  Not used while a stage is being timed, nor after
// a capture has failed once in this process (the calls then launch their
// kernels directly); HERSCHEL_GRAPHS=0 turns it off and HERSCHEL_DEBUG=1
// reports why a capture failed.  Replay is opt-in: it saves about 1.5% of a
// call on the decode-step trace, and stream capture across three streams is
// the part of the runtime this library leans on least in tested volume.
struct GraphKey {
  herschel_events ev;
  int64_t n;
  herschel_params p;
  herschel_outputs out;
};
struct DeviceGraph {
  bool valid = false;
  GraphKey key;
  hipGraphExec_t exec = nullptr;
};
constexpr int GRAPHS_PER_DEVICE = 4;
static DeviceGraph g_graphs[64][GRAPHS_PER_DEVICE];
static unsigned g_graph_next[64];
static bool g_graphs_failed = false;
static bool graphs_enabled() {
  static const bool on = env_flag("HERSCHEL_GRAPHS", true);
  return on && !g_graphs_failed;
}
static int graph_failed(const char* what, hipError_t e) {
  static const bool dbg = env_flag("HERSCHEL_DEBUG", false);
  if (dbg) fprintf(stderr, "herschel: graph capture off: %s: %s\n", what, hipGetErrorString(e));
  g_graphs_failed = true;
  return 0;
}

static int enqueue_cached(Ctx& c, const herschel_events* ev, int64_t n, const herschel_params* p,
                          const herschel_outputs* out) {
  if (g_stage >= 0 || !graphs_enabled() || !(c.p.flags & HERSCHEL_REPLAY)) return enqueue(c);
  std::lock_guard<std::mutex> lock(g_enqueue_mutex);
  DeviceStreams* dsx = enqueue_setup();
  int dev = 0;
  if (!dsx || hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return HERSCHEL_EDEVICE;
  GraphKey key;
  memset(&key, 0, sizeof(key));
  key.ev = *ev;
  key.n = n;
  key.p = *p;
  key.p.hip_stream = nullptr;
  key.out = *out;
  for (DeviceGraph& g : g_graphs[dev]) {
    if (!g.valid || memcmp(&g.key, &key, sizeof(key)) != 0) continue;
    const hipError_t e = hipGraphLaunch(g.exec, c.st);
    if (e == hipSuccess) return HERSCHEL_OK;
    graph_failed("hipGraphLaunch", e);
    (void)hipGetLastError();
    return enqueue_locked(c, dsx);
  }
  DeviceGraph& g = g_graphs[dev][g_graph_next[dev]++ % GRAPHS_PER_DEVICE];
  if (g.valid) {
    (void)hipGraphExecDestroy(g.exec);
    g.valid = false;
  }
  Ctx cc = c;
  cc.st = dsx->cap;
  hipError_t e = hipStreamBeginCapture(cc.st, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) {
    graph_failed("hipStreamBeginCapture", e);
    (void)hipGetLastError();
    return enqueue_locked(c, dsx);
  }
  const int code = enqueue_locked(cc, dsx);
  hipGraph_t graph = nullptr;
  e = hipStreamEndCapture(cc.st, &graph);
  if (code != HERSCHEL_OK || e != hipSuccess || !graph) {
    graph_failed("hipStreamEndCapture", e);
    if (graph) (void)hipGraphDestroy(graph);
    (void)hipGetLastError();
    return code != HERSCHEL_OK ? code : enqueue_locked(c, dsx);
  }
  hipGraphExec_t exec = nullptr;
  e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  (void)hipGraphDestroy(graph);
  if (e != hipSuccess || !exec) {
    graph_failed("hipGraphInstantiate", e);
    (void)hipGetLastError();
    return enqueue_locked(c, dsx);
  }
  g.key = key;
  g.exec = exec;
  g.valid = true;
  e = hipGraphLaunch(exec, c.st);
  if (e == hipSuccess) return HERSCHEL_OK;
  graph_failed("hipGraphLaunch", e);
  (void)hipGetLastError();
  return enqueue_locked(c, dsx);
}

// ------------------------------------------------------- static scratch
// The workspace of herschel_trace_analyze_static: one array per device that
// loads the library, held until the process ends.  Host code never passes
// the array's name to a kernel (on the host it is a stand-in, not a device
// address): the device address is taken once per device with
// hipGetSymbolAddress and every use goes through it.
static __device__ __align__(256) char scratch[HERSCHEL_STATIC_SCRATCH_BYTES];
static void* g_scratch_ptr[64];
static bool g_scratch_ok[64];

// The current device's address of `scratch` (the caller holds
// g_enqueue_mutex); nullptr when the lookup fails.
static void* static_scratch() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  if (!g_scratch_ok[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
    g_scratch_ok[dev] = true;
  }
  return g_scratch_ptr[dev];
}

// ------------------------------------------------------- completion
// A call's end reaches the host through a mailbox in pinned host memory
// (one per calling thread and device, allocated on the thread's first call
// on the device and held until the process ends): the finalize kernel
// copies the counters into it and then stores the call's sequence number.
// The thread spins on that number, about 15 us sooner per call than a copy
// of the counters back and a stream synchronisation.  It asks the stream
// for errors every 100 us and blocks in hipStreamSynchronize after 2 ms (a
// long call gains nothing from spinning).
static thread_local Mailbox* tl_mailbox[64];
static thread_local int64_t tl_mailbox_seq = 0;
constexpr int MAILBOX_MISSED = -1000;  // the stream ended without the number: copy back instead

static Mailbox* thread_mailbox() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return nullptr;
  if (!tl_mailbox[dev]) {
    void* m = nullptr;
    if (hipHostMalloc(&m, sizeof(Mailbox), hipHostMallocCoherent) != hipSuccess || !m) {
      (void)hipGetLastError();
      return nullptr;
    }
    memset(m, 0, sizeof(Mailbox));
    tl_mailbox[dev] = (Mailbox*)m;
  }
  return tl_mailbox[dev];
}

static int wait_mailbox(hipStream_t st, Mailbox* mb, int64_t seq, herschel_counters* h) {
  using clk = std::chrono::steady_clock;
  const clk::time_point t0 = clk::now();
  clk::time_point next_query = t0 + std::chrono::microseconds(100);
  while (__atomic_load_n(&mb->seq, __ATOMIC_ACQUIRE) != seq) {
    const clk::time_point t = clk::now();
    if (t >= next_query) {
      hipError_t e = hipStreamQuery(st);
      if (e == hipErrorNotReady && t - t0 > std::chrono::milliseconds(2)) e = hipStreamSynchronize(st);
      if (e == hipSuccess) {
        if (__atomic_load_n(&mb->seq, __ATOMIC_ACQUIRE) == seq) break;
        return MAILBOX_MISSED;
      }
      if (e != hipErrorNotReady) return HERSCHEL_EDEVICE;
      next_query = t + std::chrono::microseconds(100);
    }
    __builtin_ia32_pause();
  }
  int64_t* dst = (int64_t*)h;
  for (int i = 0; i < (int)(sizeof(herschel_counters) / 8); ++i) dst[i] = __atomic_load_n(&mb->c[i], __ATOMIC_RELAXED);
  return HERSCHEL_OK;
}

// The critical path's doubling pass when the call left it out and a walk
// stopped short (DevState::crit_more), on the caller's stream, waited for.
static int finish_crit(Ctx& c, uint32_t more) {
  if (!c.crit_deferred || !more) return HERSCHEL_OK;
  launch_crit_deferred(c);
  if (hipGetLastError() != hipSuccess || hipStreamSynchronize(c.st) != hipSuccess) return HERSCHEL_EDEVICE;
  return HERSCHEL_OK;
}

static int code_from(const herschel_counters& h, int64_t gap_capacity) {
  if (h.device_status & DS_PARAM) return HERSCHEL_EINVAL;
  if (h.first_invalid >= 0) return HERSCHEL_EEVENT;
  if (h.device_status) return HERSCHEL_EDEVICE;
  if (h.n_gaps_total > gap_capacity) return HERSCHEL_ECAPACITY;
  return HERSCHEL_OK;
}

}  // namespace hx

using namespace hx;

extern "C" {

const char* herschel_strerror(int code) {
  switch (code) {
    case HERSCHEL_OK: return "ok";
    case HERSCHEL_EINVAL: return "invalid argument";
    case HERSCHEL_EEVENT: return "invalid input row (see counters.first_invalid)";
    case HERSCHEL_ECAPACITY: return "gap list capacity exceeded (see counters.n_gaps_total)";
    case HERSCHEL_EWORKSPACE: return "workspace missing, misaligned or too small";
    case HERSCHEL_EDEVICE: return "device error";
    case HERSCHEL_ETOOBIG: return "input too large for the static scratch of herschel_trace_analyze_static";
    default: return "unknown error";
  }
}

int herschel_time_stage(int stage, void* start_event, void* stop_event) {
  if (stage < 0 || stage >= HERSCHEL_N_STAGES) return HERSCHEL_EINVAL;
  g_stage = (start_event && stop_event) ? stage : -1;
  g_ev0 = (hipEvent_t)start_event;
  g_ev1 = (hipEvent_t)stop_event;
  return HERSCHEL_OK;
}

int herschel_sort_stats(const herschel_params* p, int32_t* out) {
  if (!p || !out || !p->workspace) return HERSCHEL_EINVAL;
  if (p->window_end <= p->window_begin || p->n_procs < 1 || p->n_streams < 1 || p->n_threads < 1)
    return HERSCHEL_EINVAL;
  DevState ds;  // the workspace starts with the device state of the last call
  if (hipStreamSynchronize((hipStream_t)p->hip_stream) != hipSuccess ||
      hipMemcpy(&ds, p->workspace, sizeof(DevState), hipMemcpyDeviceToHost) != hipSuccess)
    return HERSCHEL_EDEVICE;
  // digit passes per sort, as layout_workspace plans them; the join has no
  // sort (the correlation table serves it), so its entries are zero
  const int pb = bits_host((uint64_t)(p->n_procs - 1)), sb = bits_host((uint64_t)(p->n_streams - 1));
  const int tb = bits_host((uint64_t)(p->n_threads - 1));
  const int wb = bits_host((uint64_t)(p->window_end - p->window_begin - 1));
  // the timeline and containment sorts, reported as s = 0 and s = 2
  const int key_bits[2] = {pb + sb + wb, pb + tb + wb + 1};
  const int32_t counts[2] = {ds.nK, ds.nCL};
  const int slot_of[2] = {0, 2};
  for (int i = 0; i < 9; ++i) out[i] = 0;
  for (int i = 0; i < 2; ++i) {
    int nd, first, sh1;
    sort_digits(key_bits[i], true, &nd, &first, &sh1);
    const int o = 3 * slot_of[i];
    out[o + 0] = counts[i];
    out[o + 1] = (int32_t)ds.sort_trivial[i];
    out[o + 2] = nd;
  }
  return HERSCHEL_OK;
}

int herschel_workspace_size(int64_t n, const herschel_params* p, size_t* bytes) {
  if (!p || !bytes || n < 0 || n >= (1LL << 30)) return HERSCHEL_EINVAL;
  if (p->window_end <= p->window_begin || p->window_end - p->window_begin > HERSCHEL_MAX_WINDOW)
    return HERSCHEL_EINVAL;
  if (p->n_procs < 1 || p->n_procs > HERSCHEL_MAX_PROCS || p->n_streams < 1 ||
      p->n_streams > HERSCHEL_MAX_STREAMS || p->n_threads < 1 || p->n_threads > HERSCHEL_MAX_THREADS ||
      p->n_names < 1 || p->n_names > HERSCHEL_MAX_NAMES)
    return HERSCHEL_EINVAL;
  if ((p->flags & HERSCHEL_OUT_WAITS) && (p->n_op_names < 1 || p->n_op_names > HERSCHEL_MAX_WAIT_OP_NAMES))
    return HERSCHEL_EINVAL;
  if ((p->flags & HERSCHEL_OUT_SOL) && p->n_op_names < 1) return HERSCHEL_EINVAL;
  Ctx c;
  c.p = *p;
  c.n = n;
  c.P = p->n_procs;
  c.S = p->n_streams;
  c.T = p->n_threads;
  c.NN = p->n_names;
  c.W = p->window_end - p->window_begin;
  c.contain = (p->flags & HERSCHEL_OUT_CONTAIN) != 0;
  c.waits = (p->flags & HERSCHEL_OUT_WAITS) != 0;
  c.sol = (p->flags & HERSCHEL_OUT_SOL) != 0;
  c.crit = (p->flags & HERSCHEL_OUT_CRIT) != 0;
  c.crit_walk_max = crit_walk_max();
  c.graph = (p->flags & HERSCHEL_OUT_GRAPH) != 0;
  if (c.graph && p->n_graph_nodes < 1) return HERSCHEL_EINVAL;
  c.NG = c.graph ? p->n_graph_nodes : 0;
  c.NOP = p->n_op_names;
  c.nob = bits_host((uint64_t)(c.NOP > 0 ? c.NOP - 1 : 0));
  c.overlap = (p->flags & HERSCHEL_OUT_OVERLAP) != 0;
  c.pb = bits_host((uint64_t)(c.P - 1));
  c.sb = bits_host((uint64_t)(c.S - 1));
  c.tb = bits_host((uint64_t)(c.T - 1));
  c.wb = bits_host((uint64_t)(c.W - 1));
  c.wb1 = bits_host((uint64_t)c.W);
  c.vb = bits_host((uint64_t)c.W + 1);
  *bytes = layout_workspace(c, nullptr);
  return HERSCHEL_OK;
}

// Containment reads the per-row links back (each launch's op, each op's
// depth): NULL link / aux outputs are then served by workspace arrays.
static void redirect_outputs(Ctx& c) {
  if (!c.contain) return;
  if (!c.o.link) c.o.link = c.link_ws;
  if (!c.o.aux) c.o.aux = c.aux_ws;
  // operator efficiency reads the per-op aggregates back
  if (!c.sol) return;
  if (!c.o.op_nkern) c.o.op_nkern = c.op_nkern_ws;
  if (!c.o.op_first) c.o.op_first = c.op_first_ws;
  if (!c.o.op_last) c.o.op_last = c.op_last_ws;
}

static int prepare(Ctx& c, const herschel_events* ev, int64_t n, const herschel_params* p, const herschel_outputs* out,
                   void* ws, size_t ws_bytes) {
  int code = check_and_plan(c, ev, n, p, out);
  if (code) return code;
  const size_t need = layout_workspace(c, nullptr);
  // the layout aligns every buffer to 256 bytes from the base (16-byte loads)
  if (!ws || ((uintptr_t)ws & 255) != 0 || ws_bytes < need) return HERSCHEL_EWORKSPACE;
  layout_workspace(c, (char*)ws);
  redirect_outputs(c);
  return HERSCHEL_OK;
}

int herschel_trace_analyze(const herschel_events* ev, int64_t n, const herschel_params* p, herschel_outputs* out) {
  Ctx c;
  int code = prepare(c, ev, n, p, out, p ? p->workspace : nullptr, p ? p->workspace_bytes : 0);
  if (code) return code;
  // a call that launches its kernels directly reports its counters through
  // the calling thread's mailbox (a replayed graph keeps the arguments it
  // was captured with, so it copies them back)
  if (!(c.p.flags & HERSCHEL_REPLAY)) {
    c.mailbox = thread_mailbox();
    c.mailbox_seq = c.mailbox ? ++tl_mailbox_seq : 0;
  }
  // the critical path's doubling pass is needed only when a walk stopped
  // short: it is enqueued after the call if the call reports so (a replayed
  // graph keeps it inline)
  c.crit_deferred = c.crit && !(c.p.flags & HERSCHEL_REPLAY);
  code = enqueue_cached(c, ev, n, p, out);
  if (code) return code;
  herschel_counters h;
  uint32_t more = 0;
  bool have = false;
  if (c.mailbox) {
    code = wait_mailbox(c.st, c.mailbox, c.mailbox_seq, &h);
    if (code == HERSCHEL_OK) {
      have = true;
      more = __atomic_load_n(&c.mailbox->crit_more, __ATOMIC_RELAXED) != 0;
    } else if (code != MAILBOX_MISSED) {
      return code;
    }
  }
  if (!have) {
    if (hipMemcpyAsync(&h, out->counters, sizeof(h), hipMemcpyDeviceToHost, c.st) != hipSuccess) return HERSCHEL_EDEVICE;
    if (c.crit_deferred &&
        hipMemcpyAsync(&more, &c.ds->crit_more, sizeof(more), hipMemcpyDeviceToHost, c.st) != hipSuccess)
      return HERSCHEL_EDEVICE;
    if (hipStreamSynchronize(c.st) != hipSuccess) return HERSCHEL_EDEVICE;
  }
  code = finish_crit(c, more);
  return code ? code : code_from(h, out->gap_capacity);
}

int herschel_trace_analyze_static(const herschel_events* ev, int64_t n, const herschel_params* p,
                                  herschel_outputs* out) {
  Ctx c;
  int code = check_and_plan(c, ev, n, p, out);
  if (code) return code;
  if (layout_workspace(c, nullptr) > (size_t)HERSCHEL_STATIC_SCRATCH_BYTES) return HERSCHEL_ETOOBIG;
  c.crit_deferred = c.crit;  // the critical path's doubling pass only if the call reports it needed
  {
    std::lock_guard<std::mutex> lock(g_enqueue_mutex);
    void* base = static_scratch();
    if (!base) return HERSCHEL_EDEVICE;
    layout_workspace(c, (char*)base);
    redirect_outputs(c);
    static bool lds_attr = false;
    if (!lds_attr) {
      names_set_lds_attr();
      lds_attr = true;
    }
    code = enqueue_locked(c, nullptr);
  }
  if (code) return code;
  herschel_counters h;
  uint32_t more = 0;
  if (hipMemcpyAsync(&h, out->counters, sizeof(h), hipMemcpyDeviceToHost, c.st) != hipSuccess) return HERSCHEL_EDEVICE;
  if (c.crit_deferred &&
      hipMemcpyAsync(&more, &c.ds->crit_more, sizeof(more), hipMemcpyDeviceToHost, c.st) != hipSuccess)
    return HERSCHEL_EDEVICE;
  if (hipStreamSynchronize(c.st) != hipSuccess) return HERSCHEL_EDEVICE;
  code = finish_crit(c, more);
  return code ? code : code_from(h, out->gap_capacity);
}

int herschel_trace_analyze_batch(const herschel_events* ev, const int64_t* trace_offsets, int32_t n_traces,
                                 const herschel_params* p, herschel_outputs* out) {
  if (!ev || !trace_offsets || !p || !out || n_traces < 0) return HERSCHEL_EINVAL;
  if (n_traces == 0) return HERSCHEL_OK;
  for (int32_t t = 0; t < n_traces; ++t)
    if (trace_offsets[t + 1] < trace_offsets[t] || trace_offsets[t] < 0) return HERSCHEL_EINVAL;
  int first_err = HERSCHEL_OK;
  int32_t launched = 0;
  for (int32_t t = 0; t < n_traces; ++t) {
    herschel_events e = *ev;
    const int64_t o = trace_offsets[t];
    if (trace_offsets[t + 1] > o) {
      e.ts += o;
      e.te += o;
      e.corr += o;
      e.pid += o;
      e.lane += o;
      e.name += o;
      e.kind += o;
      if (e.flops) e.flops += o;
      if (e.bytes) e.bytes += o;
      if (e.graph_node) e.graph_node += o;
    }
    herschel_params pt = p[t];
    pt.hip_stream = p[0].hip_stream;
    pt.workspace = p[0].workspace;
    pt.workspace_bytes = p[0].workspace_bytes;
    Ctx c;
    int code = prepare(c, &e, trace_offsets[t + 1] - o, &pt, &out[t], pt.workspace, pt.workspace_bytes);
    if (!code) code = enqueue(c);
    if (code) {
      if (first_err == HERSCHEL_OK) first_err = code;
      break;
    }
    launched = t + 1;
  }
  hipStream_t st = (hipStream_t)p[0].hip_stream;
  if (hipStreamSynchronize(st) != hipSuccess) return HERSCHEL_EDEVICE;
  for (int32_t t = 0; t < launched; ++t) {
    herschel_counters h;
    if (hipMemcpy(&h, out[t].counters, sizeof(h), hipMemcpyDeviceToHost) != hipSuccess) return HERSCHEL_EDEVICE;
    const int code = code_from(h, out[t].gap_capacity);
    if (code != HERSCHEL_OK) return code;
  }
  return first_err;
}

// Chunks of chunk_traces traces: chunk c + 1 uploads into the other staging
// set on the library's copy stream while chunk c is analysed by the batch
// entry point on the caller's stream (which waits for the upload's event).
// A batch call returns after its work is done, so the set that chunk c - 1
// used is free when chunk c + 1's upload is enqueued.  One chunked call at a
// time per process: the copy stream and its events are shared.
static std::mutex g_chunk_mutex;

int herschel_trace_analyze_chunked(const herschel_events* host, const int64_t* trace_offsets, int32_t n_traces,
                                   int32_t chunk_traces, const herschel_events* staging, int64_t staging_rows,
                                   const herschel_params* p, herschel_outputs* out) {
  if (!host || !trace_offsets || !staging || !p || !out || n_traces < 0 || chunk_traces < 1 || staging_rows < 0)
    return HERSCHEL_EINVAL;
  if (n_traces == 0) return HERSCHEL_OK;
  for (int32_t t = 0; t < n_traces; ++t)
    if (trace_offsets[t + 1] < trace_offsets[t] || trace_offsets[t] < 0) return HERSCHEL_EINVAL;
  const int32_t n_chunks = (int32_t)cdiv((int64_t)n_traces, (int64_t)chunk_traces);
  for (int32_t ch = 0; ch < n_chunks; ++ch) {
    const int32_t t0 = ch * chunk_traces, t1 = std::min(n_traces, t0 + chunk_traces);
    if (trace_offsets[t1] - trace_offsets[t0] > staging_rows) return HERSCHEL_EINVAL;
  }
  // the columns every call reads, on both sides; an optional column the host
  // holds must have room in both staging sets
  if (!host->ts || !host->te || !host->corr || !host->pid || !host->lane || !host->name || !host->kind)
    return HERSCHEL_EINVAL;
  for (int b = 0; b < 2; ++b) {
    const herschel_events& d = staging[b];
    if (!d.ts || !d.te || !d.corr || !d.pid || !d.lane || !d.name || !d.kind) return HERSCHEL_EINVAL;
    if ((host->flops && !d.flops) || (host->bytes && !d.bytes) || (host->graph_node && !d.graph_node))
      return HERSCHEL_EINVAL;
  }
  std::lock_guard<std::mutex> chunk_lock(g_chunk_mutex);
  DeviceStreams* dsx;
  {
    std::lock_guard<std::mutex> lock(g_enqueue_mutex);
    dsx = enqueue_setup();
  }
  if (!dsx) return HERSCHEL_EDEVICE;
  const hipStream_t cs = dsx->copy, st = (hipStream_t)p[0].hip_stream;
  auto upload = [&](int32_t ch) -> bool {
    const herschel_events& d = staging[ch & 1];
    const int32_t t0 = ch * chunk_traces, t1 = std::min(n_traces, t0 + chunk_traces);
    const int64_t r0 = trace_offsets[t0], rows = trace_offsets[t1] - r0;
    bool ok = true;
    auto put = [&](const void* dst, const void* src, size_t elem) {
      if (ok && rows > 0 && src)
        ok = hipMemcpyAsync(const_cast<void*>(dst), static_cast<const char*>(src) + r0 * elem, (size_t)rows * elem,
                            hipMemcpyHostToDevice, cs) == hipSuccess;
    };
    put(d.ts, host->ts, 8);
    put(d.te, host->te, 8);
    put(d.corr, host->corr, 8);
    put(d.pid, host->pid, 4);
    put(d.lane, host->lane, 4);
    put(d.name, host->name, 4);
    put(d.kind, host->kind, 1);
    put(d.flops, host->flops, 8);
    put(d.bytes, host->bytes, 8);
    put(d.graph_node, host->graph_node, 4);
    return ok && hipEventRecord(dsx->up[ch & 1], cs) == hipSuccess;
  };
  int code = upload(0) ? HERSCHEL_OK : HERSCHEL_EDEVICE;
  std::vector<int64_t> offs;
  std::vector<herschel_params> pc;
  for (int32_t ch = 0; ch < n_chunks && code == HERSCHEL_OK; ++ch) {
    if (ch + 1 < n_chunks && !upload(ch + 1)) {
      code = HERSCHEL_EDEVICE;
      break;
    }
    if (hipStreamWaitEvent(st, dsx->up[ch & 1], 0) != hipSuccess) {
      code = HERSCHEL_EDEVICE;
      break;
    }
    const int32_t t0 = ch * chunk_traces, t1 = std::min(n_traces, t0 + chunk_traces);
    offs.assign(trace_offsets + t0, trace_offsets + t1 + 1);
    for (auto& o : offs) o -= trace_offsets[t0];
    pc.assign(p + t0, p + t1);
    pc[0].hip_stream = p[0].hip_stream;
    pc[0].workspace = p[0].workspace;
    pc[0].workspace_bytes = p[0].workspace_bytes;
    // the staging set, without the optional columns the host does not hold
    herschel_events e = staging[ch & 1];
    if (!host->flops) e.flops = nullptr;
    if (!host->bytes) e.bytes = nullptr;
    if (!host->graph_node) e.graph_node = nullptr;
    code = herschel_trace_analyze_batch(&e, offs.data(), t1 - t0, pc.data(), out + t0);
  }
  // no upload outlives the call
  if (hipStreamSynchronize(cs) != hipSuccess && code == HERSCHEL_OK) code = HERSCHEL_EDEVICE;
  return code;
}

}  // extern "C"
