// Shared device helpers and internal data layout of the HIP trace analyzer.
//
// Everything here is CDNA4 (gfx950) wave64 code: 64-bit ballots, LDS
// staging, decoupled look-back scans with a tile ticket, and agent-scope
// atomics for the few cross-workgroup values.  Arithmetic is integer only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "herschel.h"

#ifndef HERSCHEL_CHECKED
#define HERSCHEL_CHECKED 0
#endif

namespace hx {

constexpr int WAVE = 64;
constexpr int64_t I64MAX = INT64_MAX;
constexpr int64_t I64MIN = INT64_MIN;

// Internal device-status bits (herschel_counters::device_status).
enum : uint32_t {
  DS_SPIN = 1u,      // a look-back wait exceeded its bound
  DS_OOB = 2u,       // checked build: an index left its buffer
  DS_PARAM = 4u,     // clock_offset or stream_class out of range
  DS_CAPACITY = 16u, // an internal list overflowed its bound
  DS_LOGIC = 32u     // an internal consistency check failed
};

// Ticket slots: look-back kernels whose tiles are numbered in arrival order.
// (The others number them by workgroup index: a tile waits only for tiles of
// lower index, whose workgroups the dispatcher started first.)
enum : int {
  TK_UNION = 0,    // the timeline (per stream)
  TK_UNION_D = 1,  // the device lane (all streams of a process)
  TK_UNION_O = 2,  // the op-name lanes
  N_TICKETS = 3
};

// 0 timeline (pid, stream, ts'), 1 containment, with the idle-coincidence
// outputs 2 device lane (pid, ts') and 3 op names (pid, op name, ts'), with
// the critical path 4 kernel ends (pid, min(te', W1))
constexpr int N_SORTS = 5;
enum : int { SORT_K = 0, SORT_C = 1, SORT_D = 2, SORT_O = 3, SORT_E = 4 };
// Rounds of the critical path's pointer doubling (its events number 2n < 2^31).
constexpr int CRIT_MAX_ROUNDS = 32;
// join counters (JC_MLAUNCH: launches with at least one kernel; the
// unmatched launches are the admitted ones without)
enum { JC_MATCHED, JC_UNM_K, JC_DUP, JC_NEG, JC_UNATTR, JC_MLAUNCH, JC_N };
constexpr int JOIN_COPIES = 16;
// The correlation table takes dense slots (process base + id - smallest id)
// when the call has at most JT_PROCS processes and their id ranges fit two
// slots per row; otherwise hashed slots.
constexpr int JT_PROCS = 64;
// Join keys: (pid << 52) | ((corr mod 2^51) << 1) | is_kernel.  Dense slots
// subtract ids modulo 2^51, exact since a dense range is far below 2^51.
constexpr int JK_PID_SHIFT = 52;
constexpr uint64_t JK_CORR_MASK = (1ull << 51) - 1;
constexpr uint32_t JT_EMPTY = ~0u;
constexpr uint64_t SIGN64 = 1ull << 63;

// Per-call device state, zeroed by the init kernel.
struct DevState {
  uint32_t ticket[N_TICKETS];
  uint32_t status;
  uint32_t sort_parity[N_SORTS];  // buffer holding each sort's result
  int32_t nK;   // admitted kernels (timeline list)
  int32_t nCL;  // admitted ops + launches (containment list)
  int32_t nJ;   // admitted launches + kernels (join list)
  int32_t nEv;  // overlap events (2 per coverage run)
  int32_t nO;          // admitted CPU ops (op-name list, idle coincidence)
  int32_t nOev;        // op-name run endpoints
  int64_t nDgap;       // device idle intervals
  int64_t nOgap;       // gaps of the op-name lanes (not used)
  int32_t nDev;        // endpoints of the device lane (none)
  uint32_t pad2;
  uint32_t crit_new[CRIT_MAX_ROUNDS];  // critical path: events newly marked in each doubling round
  int64_t first_invalid;  // smallest bad row (INT64_MAX = none)
  int64_t n_gaps;
  uint32_t sort_trivial[N_SORTS];  // bit d: digit d moves no data (every key agrees on it, or it is
                                   // left to the refine pass: then bit 31 is set too)
  uint32_t crit_more;              // critical path: a walk stopped short, the doubling must finish the path
  uint32_t join_direct;            // 1: dense correlation slots, 0: hashed slots
  uint32_t jt_nfix;                // entries of the join's fix-up list
  int64_t jt_slots;                // table slots in use (dense: the ids' ranges; hashed: the table)
  uint64_t jt_present;             // bit p: process p has an admitted launch or kernel
  uint64_t jt_lo[JT_PROCS];        // per process: max of ~(corr ^ 2^63), the smallest id
  uint64_t jt_hi[JT_PROCS];        // per process: max of corr ^ 2^63, the largest id
  int64_t jt_cmin[JT_PROCS];       // smallest correlation id of each process
  int64_t jt_base[JT_PROCS];       // first table slot of each process
  // join counts (JC_* order) and latency bins, in copies summed at the end
  unsigned long long join_acc[JOIN_COPIES][JC_N + 64];
  // radix digit offsets: each digit's exclusive prefix over its values (the
  // global offset of every bin), from the plan kernel
  uint32_t hist[N_SORTS][8][256];
};

// Largest process count the per-process correlation-id table supports.
constexpr int MAX_PROCS = HERSCHEL_MAX_PROCS;

// ---------------------------------------------------------------- wave ops
__device__ __forceinline__ int lane_id() { return __lane_id(); }
__device__ __forceinline__ uint64_t lanemask_lt() {
  int l = lane_id();
  return l == 0 ? 0ull : (~0ull >> (64 - l));
}
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ int popc(uint64_t m) { return __popcll(m); }

template <class T>
__device__ __forceinline__ T shfl(T v, int src) { return __shfl(v, src, WAVE); }
template <class T>
__device__ __forceinline__ T shfl_up(T v, unsigned d) { return __shfl_up(v, d, WAVE); }
template <class T>
__device__ __forceinline__ T shfl_down(T v, unsigned d) { return __shfl_down(v, d, WAVE); }
template <class T>
__device__ __forceinline__ T shfl_xor(T v, int m) { return __shfl_xor(v, m, WAVE); }

// The correlation-table plan, by one wave (lane p is process p): dense
// slots when the call has at most JT_PROCS processes (P > 0 here) and their
// id ranges, from prep's per-process smallest and largest ids, fit `cap`
// slots together (process p's ids then start at slot jt_base[p]); hashed
// slots over the whole table of `hsize` slots otherwise.  With `write` the
// lanes store the plan (one wave of the call does); every caller gets the
// decision and the number of slots in use.
__device__ __forceinline__ bool jt_plan_wave(DevState* ds, int P, int64_t cap, int64_t hsize, bool write,
                                             int64_t* slots) {
  const int p = threadIdx.x & (WAVE - 1);
  const bool present = P > 0 && p < P && ((ds->jt_present >> p) & 1);
  const uint64_t ulo = present ? ~ds->jt_lo[p] : 0ull, uhi = present ? ds->jt_hi[p] : 0ull;
  const int64_t cmin = (int64_t)(ulo ^ SIGN64);
  // largest - smallest id, exact in unsigned arithmetic; ranges beyond the
  // capacity saturate, so the sum cannot overflow
  const uint64_t span = uhi - ulo;
  const int64_t range = !present ? 0 : span >= (uint64_t)cap ? cap + 1 : (int64_t)span + 1;
  int64_t inc = range;
  for (int d = 1; d < WAVE; d <<= 1) {
    const int64_t o = (int64_t)__shfl_up((uint64_t)inc, d, WAVE);
    if (p >= d) inc += o;
  }
  const int64_t total = (int64_t)__shfl((uint64_t)inc, WAVE - 1, WAVE);
  const bool direct = P > 0 && total <= cap;
  *slots = direct ? total : hsize;
  if (write) {
    ds->jt_cmin[p] = present ? cmin : 0;
    ds->jt_base[p] = inc - range;
    if (p == 0) {
      ds->join_direct = direct ? 1u : 0u;
      ds->jt_slots = direct ? total : hsize;
    }
  }
  return direct;
}

// Dense slot of a join key (the plan chose dense slots).
__device__ __forceinline__ int64_t jt_dense_slot(const DevState* ds, uint64_t key) {
  const int p = (int)(key >> JK_PID_SHIFT);
  const uint64_t rel = (((key >> 1) & JK_CORR_MASK) - ((uint64_t)ds->jt_cmin[p] & JK_CORR_MASK)) & JK_CORR_MASK;
  return ds->jt_base[p] + (int64_t)rel;
}

// First probe of a join key's hashed slot: the SplitMix64 finalizer (Steele,
// Lea and Flood, "Fast splittable pseudorandom number generators", 2014) of
// the key without its kind bit.
__device__ __forceinline__ uint64_t jt_hash(uint64_t key) {
  uint64_t x = key >> 1;
  x ^= x >> 30;
  x *= 0xbf58476d1ce4e5b9ull;
  x ^= x >> 27;
  x *= 0x94d049bb133111ebull;
  x ^= x >> 31;
  return x;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
  for (int d = 32; d >= 1; d >>= 1) v += shfl_down(v, d);
  return shfl(v, 0);
}
__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
  return (int64_t)wave_sum_u64((uint64_t)v);
}
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  for (int d = 32; d >= 1; d >>= 1) {
    uint64_t o = shfl_down(v, d);
    v = o > v ? o : v;
  }
  return shfl(v, 0);
}
__device__ __forceinline__ int64_t wave_min_i64(int64_t v) {
  for (int d = 32; d >= 1; d >>= 1) {
    int64_t o = shfl_down(v, d);
    v = o < v ? o : v;
  }
  return shfl(v, 0);
}
__device__ __forceinline__ int64_t wave_max_i64(int64_t v) {
  for (int d = 32; d >= 1; d >>= 1) {
    int64_t o = shfl_down(v, d);
    v = o > v ? o : v;
  }
  return shfl(v, 0);
}
// DPP (data-parallel primitives: a VALU move that reads another lane of the
// same row) in its GFX9 forms.  A row is 16 lanes: row_shr:d moves lane
// l - d of the row to lane l; row_bcast:15 carries lane 15 of each row to
// the next row, row_bcast:31 lane 31 to rows 2 and 3; wave_shr:1 moves lane
// l - 1 of the wave to lane l.  Lanes outside the row mask, and lanes whose
// source lies outside the row (or the wave), keep `old`.  No LDS crossbar
// and no LDS round trip, unlike the shuffles above.  Every lane of the wave
// must be active.
constexpr int DPP_ROW_SHR1 = 0x111;
constexpr int DPP_ROW_SHR2 = 0x112;
constexpr int DPP_ROW_SHR4 = 0x114;
constexpr int DPP_ROW_SHR8 = 0x118;
constexpr int DPP_WAVE_SHR1 = 0x138;
constexpr int DPP_ROW_BCAST15 = 0x142;
constexpr int DPP_ROW_BCAST31 = 0x143;

template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ uint32_t dpp32(uint32_t old, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROWS, 0xf, false);
}
template <int CTRL, int ROWS = 0xf>
__device__ __forceinline__ uint64_t dpp64(uint64_t old, uint64_t v) {
  return ((uint64_t)dpp32<CTRL, ROWS>((uint32_t)(old >> 32), (uint32_t)(v >> 32)) << 32) |
         dpp32<CTRL, ROWS>((uint32_t)old, (uint32_t)v);
}
// Inclusive prefix maximum over the wave (unsigned, identity 0): doubling
// shifts inside each row, then each row takes the maxima of the rows
// before it by the two broadcasts.
__device__ __forceinline__ uint64_t wave_prefix_max_u64(uint64_t v) {
  uint64_t o;
  o = dpp64<DPP_ROW_SHR1>(0ull, v);
  v = o > v ? o : v;
  o = dpp64<DPP_ROW_SHR2>(0ull, v);
  v = o > v ? o : v;
  o = dpp64<DPP_ROW_SHR4>(0ull, v);
  v = o > v ? o : v;
  o = dpp64<DPP_ROW_SHR8>(0ull, v);
  v = o > v ? o : v;
  o = dpp64<DPP_ROW_BCAST15, 0xa>(0ull, v);
  v = o > v ? o : v;
  o = dpp64<DPP_ROW_BCAST31, 0xc>(0ull, v);
  v = o > v ? o : v;
  return v;
}
// Lane l takes v of lane l - 1; lane 0 takes `fill`.
__device__ __forceinline__ uint64_t wave_shift_up1_u64(uint64_t v, uint64_t fill) {
  return dpp64<DPP_WAVE_SHR1>(fill, v);
}
// Maximum over the wave (unsigned), in every lane.
__device__ __forceinline__ uint64_t wave_allmax_u64(uint64_t v) {
  v = wave_prefix_max_u64(v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, WAVE - 1);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), WAVE - 1);
  return ((uint64_t)hi << 32) | lo;
}

// Inclusive prefix sum across the wave.
__device__ __forceinline__ uint32_t wave_incl_sum_u32(uint32_t v) {
  int l = lane_id();
  for (int d = 1; d < WAVE; d <<= 1) {
    uint32_t o = shfl_up(v, d);
    if (l >= d) v += o;
  }
  return v;
}

// --------------------------------------------------------- memory helpers
__device__ __forceinline__ uint64_t ld_agent(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t ld_agent(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void set_status(DevState* ds, uint32_t bit) {
  atomicOr(&ds->status, bit);
}

// Bounds check of a data-dependent index (only in checked builds): on a
// violation the status bit is set and the caller skips the access.
__device__ __forceinline__ bool in_range(DevState* ds, int64_t i, int64_t n) {
#if HERSCHEL_CHECKED
  if ((uint64_t)i >= (uint64_t)n) {
    set_status(ds, DS_OOB);
    return false;
  }
#else
  (void)ds;
  (void)i;
  (void)n;
#endif
  return true;
}

// Release-build bounds check of an index that one kernel derives from
// another kernel's results (a scatter position): a violation sets DS_OOB and
// the caller skips the access, so a disagreement between two kernels ends in
// HERSCHEL_EDEVICE instead of a stray store.
__device__ __forceinline__ bool in_bounds(DevState* ds, int64_t i, int64_t n) {
  if ((uint64_t)i >= (uint64_t)n) {
    set_status(ds, DS_OOB);
    return false;
  }
  return true;
}

// Bound on look-back waits, in device time: s_memrealtime counts a constant
// 100 MHz clock, and a wait that has lasted SPIN_TICKS (50 ms, thousands of
// times a kernel's run time here) sets DS_SPIN and gives up, so a logic
// error can never hang a queue.
constexpr uint64_t SPIN_TICKS = 5000000;
__device__ __forceinline__ uint64_t spin_clock() { return wall_clock64(); }

// ------------------------------------------------------ decoupled look-back
// 64-bit status words: bits 62-63 flag (0 empty, 1 aggregate, 2 prefix),
// bits 0-61 value.
constexpr uint64_t LB_AGG = 1ull << 62;
constexpr uint64_t LB_PRE = 2ull << 62;
constexpr uint64_t LB_VAL = (1ull << 62) - 1;

struct OpSum {
  __device__ static uint64_t combine(uint64_t older, uint64_t newer) { return (older + newer) & LB_VAL; }
  __device__ static uint64_t identity() { return 0; }
};
struct OpMax {
  __device__ static uint64_t combine(uint64_t older, uint64_t newer) { return older > newer ? older : newer; }
  __device__ static uint64_t identity() { return 0; }
};
struct OpXor32 {
  __device__ static uint64_t combine(uint64_t older, uint64_t newer) { return (older ^ newer) & 0xffffffffull; }
  __device__ static uint64_t identity() { return 0; }
};
// Segmented max: value = seg (bits 42..59) | head (bit 41) | m (bits 0..40).
// head: the span contains a segment start; m: max over the span's last
// segment (0 = none); seg: segment of the span's last element.
struct OpSegMax {
  static constexpr uint64_t M_MASK = (1ull << 41) - 1;
  static constexpr uint64_t HEAD = 1ull << 41;
  __device__ static uint64_t make(uint32_t seg, bool head, uint64_t m) {
    return ((uint64_t)seg << 42) | (head ? HEAD : 0) | (m & M_MASK);
  }
  __device__ static uint32_t seg(uint64_t v) { return (uint32_t)(v >> 42); }
  __device__ static uint64_t m(uint64_t v) { return v & M_MASK; }
  __device__ static uint64_t combine(uint64_t older, uint64_t newer) {
    if (newer & HEAD) return newer;
    uint64_t a = older & M_MASK, b = newer & M_MASK;
    return (newer & ~(M_MASK | HEAD)) | (older & HEAD) | (a > b ? a : b);
  }
  __device__ static uint64_t identity() { return 0; }
};

// Decoupled look-back executed by ONE whole wave.  Publishes the tile's
// aggregate, combines the predecessors' values newest-first 64 at a time,
// publishes the inclusive prefix and returns the exclusive prefix (all
// lanes).  Tile 0 publishes its prefix directly.
template <class Op>
__device__ uint64_t wave_lookback(uint64_t* status, int tile, uint64_t agg, DevState* ds) {
  const int lane = lane_id();
  if (tile == 0) {
    if (lane == 0) st_agent(&status[0], LB_PRE | (agg & LB_VAL));
    return Op::identity();
  }
  if (lane == 0) st_agent(&status[tile], LB_AGG | (agg & LB_VAL));
  uint64_t acc = Op::identity();  // combination of the newer windows so far
  bool have = false;
  int pred = tile - 1;
  bool give_up = false;
  while (true) {
    int idx = pred - lane;
    uint64_t s = idx >= 0 ? ld_agent(&status[idx]) : (LB_PRE | Op::identity());
    uint64_t t0 = 0;
    while (ballot((s >> 62) == 0)) {
      if ((s >> 62) == 0) s = ld_agent(&status[idx]);
      const uint64_t now = spin_clock();
      if (t0 == 0) t0 = now;
      if (now - t0 > SPIN_TICKS) {
        give_up = true;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (give_up) break;
    uint64_t pre_mask = ballot((s >> 62) == 2);
    int last = pre_mask ? (__ffsll((unsigned long long)pre_mask) - 1) : (WAVE - 1);
    // ordered fold over lanes 0..last, lane 0 newest: w = v[last] o ... o v[0]
    uint64_t v = (lane <= last) ? (s & LB_VAL) : Op::identity();
    for (int d = 1; d < WAVE; d <<= 1) {
      uint64_t o = shfl_down(v, d);  // lane + d is older
      if (lane + d <= last && (lane & ((d << 1) - 1)) == 0) v = Op::combine(o, v);
    }
    uint64_t w = shfl(v, 0);
    acc = have ? Op::combine(w, acc) : w;
    have = true;
    if (pre_mask) break;
    pred -= WAVE;
  }
  if (give_up) {
    if (lane == 0) set_status(ds, DS_SPIN);
    acc = Op::identity();
  }
  if (lane == 0) st_agent(&status[tile], LB_PRE | (Op::combine(acc, agg) & LB_VAL));
  return acc;
}

// Tile ticket: tiles are handed out in launch order, so every predecessor a
// look-back waits on is already running.
__device__ __forceinline__ int take_ticket(DevState* ds, int slot, int* smem) {
  if (threadIdx.x == 0) *smem = (int)atomicAdd(&ds->ticket[slot], 1u);
  __syncthreads();
  return *smem;
}

// ------------------------------------------------------------ block scans
// Exclusive sum over a block of NT threads (NT a multiple of 64, <= 1024).
template <int NT>
__device__ uint32_t block_excl_sum(uint32_t v, uint32_t* scratch /* >= NT/64 + 1 */, uint32_t* total) {
  const int lane = lane_id(), wv = threadIdx.x / WAVE;
  uint32_t inc = wave_incl_sum_u32(v);
  if (lane == WAVE - 1) scratch[wv] = inc;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t run = 0;
    for (int w = 0; w < NT / WAVE; ++w) {
      uint32_t t = scratch[w];
      scratch[w] = run;
      run += t;
    }
    scratch[NT / WAVE] = run;
  }
  __syncthreads();
  uint32_t r = scratch[wv] + inc - v;
  if (total) *total = scratch[NT / WAVE];
  __syncthreads();
  return r;
}

__device__ __forceinline__ int bits_of(uint64_t x) { return x == 0 ? 0 : 64 - __clzll((long long)x); }

}  // namespace hx
