// Host-side plan of one analysis call and the launchers of each stage.
#pragma once

#include <algorithm>

#include "common.hpp"

namespace hx {

// One LSD radix sort: 64-bit keys with a 32-bit payload, ping-pong
// buffers, digit histograms in DevState::hist[id], result buffer index in
// DevState::sort_parity[id].
struct SortBufs {
  uint64_t* k[2] = {nullptr, nullptr};
  uint32_t* v[2] = {nullptr, nullptr};
  uint32_t* status0 = nullptr;          // [tiles_max * RS_LB_WORDS] look-back words of the first digit
  uint32_t* status1 = nullptr;          // [nd - 1][tiles_max * RS_LB_WORDS] the later digits
  int64_t n_max = 0;                    // capacity (host upper bound of the count)
  int64_t tiles_max = 0;
  int nd = 0;                           // digits of the key: digit 0 below bit sh1, 8-bit digits above
  int id = 0;                           // sort index: histogram, parity
  int first = 0;                        // first digit sorted by passes (1: digit 0 left to the refine pass)
  int sh1 = 8;                          // lowest bit of digit 1 (digit d >= 1 is bits sh1 + 8(d-1) ..)
};

// Digits of a key_bits-bit sort key.  With `refine` (keys wider than 32
// bits), the passes take 8-bit digits from the top down and leave the bits
// below them to the refine pass: as few passes as leave it at most
// RF_LOW_MAX bits (8 at least).  Otherwise every digit is 8 bits, from bit 0.
constexpr int RF_LOW_MAX = 14;
inline void sort_digits(int key_bits, bool refine, int* nd, int* first, int* sh1) {
  if (refine && key_bits > 32) {
    int passes = (key_bits - RF_LOW_MAX + 7) / 8;
    if (passes < 1) passes = 1;
    int lo = key_bits - 8 * passes;
    if (lo < 8) lo = 8;
    *first = 1;
    *sh1 = lo;
    *nd = 1 + (key_bits - lo + 7) / 8;
  } else {
    *first = 0;
    *sh1 = 8;
    *nd = (key_bits + 7) / 8;
  }
}

// Pinned host memory that the finalize kernel copies the counters into, with
// a sequence number written last (one per calling thread and device).
struct Mailbox {
  int64_t c[sizeof(herschel_counters) / 8];
  int64_t crit_more;  // the critical path needs its doubling pass (DevState::crit_more)
  int64_t seq;
};

struct Ctx {
  hipStream_t st = nullptr;
  Mailbox* mailbox = nullptr;  // NULL: the caller copies the counters back itself
  int64_t mailbox_seq = 0;
  herschel_events ev{};
  int64_t n = 0;
  herschel_params p{};
  herschel_outputs o{};
  int64_t W0 = 0, W1 = 0, W = 0, thr = 0;
  int P = 0, S = 0, T = 0, NN = 0, NOP = 0;
  bool contain = false, overlap = false, waits = false, sol = false, crit = false, graph = false;
  int NG = 0;                          // graph nodes (graph replay separation)
  int nob = 0;                         // bits of an op name (idle coincidence)
  int pb = 0, sb = 0, tb = 0, wb = 0;  // key field widths: pid, stream, thread, ts'-W0
  int wb1 = 0;                         // bits of W (values 0..W)
  int vb = 0;                          // bits of W+1 (containment encoding)

  // workspace
  DevState* ds = nullptr;
  uint64_t* prep_status = nullptr;   // [prep_tiles * 3]
  int64_t prep_tiles = 0;
  uint64_t* union_status = nullptr;  // [union_tiles * 3]
  uint64_t* union_status_d = nullptr;  // [union_tiles * 3] the device-lane union
  uint64_t* union_status_o = nullptr;  // [union_tiles * 3] the op-name union
  uint64_t* dg_status = nullptr;     // [dg_tiles] look-back of the idle-length scan
  int64_t dg_tiles = 0;
  int32_t* dg_pid = nullptr;         // [dg_cap] device idle intervals, in (pid, begin) order
  int64_t* dg_begin = nullptr;
  int64_t* dg_end = nullptr;
  int64_t* dg_pre = nullptr;         // [dg_cap] idle length before each interval (exclusive prefix)
  uint64_t* dg_key = nullptr;        // [dg_cap] (pid, begin - W0) of each interval, one word
  int64_t dg_cap = 0;
  uint64_t* oev = nullptr;           // [oev_cap] op-name run endpoints
  int64_t oev_cap = 0;
  int64_t* op_span_ws = nullptr;     // [P * NOP] when the op_span output is NULL
  int64_t* dbusy_ws = nullptr;       // [P] busy time of the device lane (zeroed with the state)
  int64_t union_tiles = 0;
  uint64_t* vb_status = nullptr;     // [vb_tiles]
  int64_t vb_tiles = 0;
  int64_t* corr_min = nullptr;       // [P]
  SortBufs sK, sC;                   // timeline, containment
  SortBufs sD, sO;                   // device lane, op names (idle coincidence)
  SortBufs sE;                       // kernel ends (critical path)
  uint32_t* k_rows = nullptr;        // [n] admitted kernels' rows in row order (per-name tables)
  uint32_t* hist_part = nullptr;     // [N_SORTS][HIST_MAX_BLOCKS][8 * 256] per-workgroup digit counts
  uint64_t* jkey = nullptr;          // [n] join list (prep): admitted launches and kernels in row order
  uint32_t* jrow = nullptr;          // [n] their rows
  uint32_t* jslot = nullptr;         // [n] their hashed slots
  uint32_t* jt_L = nullptr;          // [jt_hsize] launch word per correlation slot
  uint32_t* jt_K = nullptr;          // [jt_hsize] kernel word per slot
  uint32_t* jt_C = nullptr;          // [jt_hsize] claiming row per slot (hashed slots)
  int64_t* jt_kmax = nullptr;        // [jt_hsize] latest kernel end per slot (edges only)
  int64_t* jt_kmin = nullptr;        // [jt_hsize] earliest kernel start per slot (edges only)
  uint32_t* jt_fix = nullptr;        // [jt_fix_cap][3] the join's fix-up list
  int64_t jt_fix_cap = 0;
  int64_t jt_cap = 0;                // most dense slots (two per row)
  int64_t jt_hsize = 0;              // hashed table size: a power of two of at least jt_cap
  int64_t* busy_ws = nullptr;        // [P * S] busy time when the busy output is NULL
  int32_t* link_ws = nullptr;        // [n] link when the output is NULL (containment reads it)
  int32_t* aux_ws = nullptr;         // [n] aux likewise
  uint64_t* ev_keys = nullptr;       // [ev_cap] coverage run endpoints, grouped by (pid, stream)
  int64_t ev_cap = 0;
  int32_t* seg_off = nullptr;        // [P * S + 1] first endpoint of each (pid, stream)
  uint64_t* V = nullptr;             // [n] containment encoding per sorted position
  uint64_t* M[6] = {};               // max pyramid, level l covers 64^l positions
  int64_t Mn[6] = {};
  int nlev = 0;
  uint64_t* pmt = nullptr;           // [vb_tiles] exclusive prefix max before each tile
  int32_t* par = nullptr;            // [n] answer position per sorted position
  int64_t* lk_first = nullptr;       // [n] per launch row: first start of its kernels
  int64_t* lk_last = nullptr;        // [n] last end of its kernels
  int64_t* lk_sum = nullptr;         // [n] sum of its kernels' durations
  int32_t* ag_chain = nullptr;       // [ag_tiles * AG_CHAIN] ops open at each aggregate tile's start
  int32_t* ag_nchain = nullptr;      // [ag_tiles] their number (may exceed AG_CHAIN)
  int64_t ag_tiles = 0;
  uint64_t* name_part = nullptr;     // [name_blocks * NN * 4] per-block name tables
  int name_blocks = 0;
  uint64_t* sol_part = nullptr;      // [sol_blocks * NOP * 4] per-block op-name tables (operator efficiency)
  uint64_t* sol_tot = nullptr;       // [NOP * 4] per-name totals (zeroed with the state)
  int sol_blocks = 0;
  int32_t* op_nkern_ws = nullptr;    // [n] per-op aggregates when those outputs are NULL
  int64_t* op_first_ws = nullptr;    //     (operator efficiency reads them back)
  int64_t* op_last_ws = nullptr;
  int32_t* crit_pred = nullptr;      // [2n] critical path: each event's release
  uint8_t* crit_code = nullptr;      // [2n] its part and charged record
  uint8_t* crit_mark = nullptr;      // [2n] on the path (zeroed)
  int32_t* crit_ptr[2] = {nullptr, nullptr};  // [2n] exits, then doubling pointers
  int crit_walk_max = 64;            // exits a process's walk follows before the doubling takes over
  bool crit_deferred = false;        // the doubling pass, if needed, is enqueued after the call
  uint32_t* crit_lastc1 = nullptr;   // [n] by containment position (zeroed)
  uint8_t* crit_hasnext = nullptr;   // [n] by containment position (zeroed)
  uint64_t* crit_zmax = nullptr;     // [P] (zeroed)
  uint32_t* crit_zrow1 = nullptr;    // [P] (zeroed)
  uint64_t* opn_part = nullptr;      // [opn_blocks * NOP * 4] per-block op-name tables
  int opn_blocks = 0;
  uint64_t* graph_part = nullptr;    // [graph_blocks * NG * 5] per-block graph-node tables
  int graph_blocks = 0;
  char* zero_begin = nullptr;        // region cleared at the start of a call
  size_t zero_bytes = 0;
};

// Returns the workspace bytes and, when base != nullptr, points c's workspace
// members into it.
size_t layout_workspace(Ctx& c, char* base);

void launch_init(Ctx& c);
void launch_prep(Ctx& c);
void launch_hist_multi(Ctx& c, SortBufs* const* s, const int32_t* const* count, int k);
void launch_sort_multi(Ctx& c, SortBufs* const* s, const int32_t* const* count, int k, int p0, int p1);
void launch_refine(Ctx& c);
void launch_names(Ctx& c);
void launch_timeline(Ctx& c);
// idle coincidence: the device lane's union, the op-name lanes' union, the
// prefix sums of the idle intervals (after the device lane's), the search
// (after all three)
void launch_union_device(Ctx& c);
void launch_union_opnames(Ctx& c);
void launch_dg_scan(Ctx& c);
void launch_waits(Ctx& c);
void launch_overlap(Ctx& c);
void launch_contain(Ctx& c);
void launch_depth(Ctx& c);
void launch_opagg(Ctx& c);
void launch_names_reduce(Ctx& c);
void launch_kernel_ops(Ctx& c);
void launch_crit_deferred(Ctx& c);
void launch_opnames(Ctx& c);
bool opnames_use_tables(int NOP);
int opnames_block_count(int64_t n_max, int NOP);
void launch_join_table(Ctx& c);
void launch_edges(Ctx& c);
void launch_finalize(Ctx& c);
void launch_sol(Ctx& c);
void launch_crit_elist(Ctx& c);
// the critical path: the kernels' releases (after the join and the
// timeline sort; beside the host records'), the host records' releases, last
// children and ops' ends (after containment and the join), then, once both
// are done, the rows, the marking and the charges
void launch_crit_kernels(Ctx& c);
void launch_crit_front(Ctx& c);
void launch_crit(Ctx& c);
void launch_graph(Ctx& c);
bool graph_uses_tables(int NG);
int graph_block_count(int64_t n_max, int NG);
int sol_block_count(int64_t n_max, int NOP);
bool sol_uses_tables(int NOP);

int64_t prep_tile_rows();
int64_t union_tile_elems();
void names_set_lds_attr();

// digit histograms: keys per workgroup (at least), most workgroups per sort
constexpr int HIST_CHUNK = 4096;
constexpr int HIST_MAX_BLOCKS = 256;

// per-op aggregates: positions per workgroup, open ops kept per tile start
constexpr int AG_TILE = 512;
constexpr int AG_CHAIN = 64;

constexpr int RS_THREADS = 512;
constexpr int RS_ITEMS = 8;
constexpr int RS_TILE = RS_THREADS * RS_ITEMS;  // 4096 keys per tile
constexpr int RS_LB_WORDS = 512;                // look-back words per tile: 256 counts, 256 window sums
constexpr int RS_WAVES_PER_EU = 6;              // three workgroups of 8 waves per CU
// Keys wider than 32 bits leave their lowest digit to the refine pass, which
// orders the runs of keys equal above it; runs up to RF_SHORT are fixed in
// place, longer ones listed.
constexpr int RF_SHORT = 32;

__host__ __device__ inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Workgroups of the histogram kernel for n keys (each stores one table).
__host__ __device__ inline int hist_blocks(int64_t n) {
  const int64_t b = cdiv(n, HIST_CHUNK);
  return (int)(b < 1 ? 1 : b > HIST_MAX_BLOCKS ? HIST_MAX_BLOCKS : b);
}

}  // namespace hx
