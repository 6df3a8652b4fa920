// LSD radix sort of 64-bit keys (optionally with a 32-bit payload) for CDNA4.
//
// One launch per 8-bit digit, shared by the independent sorts of a call.  Each workgroup ranks a tile of 4096 keys with
// wave64 ballots (a 64-lane match of the digit built from 8 ballots gives the
// rank among equal digits in one step), publishes its 256 per-digit counts
// through a decoupled look-back (one chain per digit, two lanes per digit),
// reorders the tile in LDS and writes each digit's run contiguously.  The
// global offset of each digit comes from a histogram of all digits taken in
// one pass before the first digit pass.  A digit on which every key agrees
// is skipped without moving data; the parity of the passes that did run
// tells every consumer which buffer holds the result.  The sort is stable.
#include "internal.hpp"

namespace hx {

constexpr uint32_t RS_FLAG_A = 1u << 30;
constexpr uint32_t RS_FLAG_P = 2u << 30;
constexpr uint32_t RS_VAL = (1u << 30) - 1;

struct HistJob {
  const uint64_t* keys;
  const int32_t* count;
  uint32_t* status0;  // the first digit pass's look-back words, cleared here
  int nd;
  int id;
  int first;  // 1: digit 0 is left to the refine pass
  int sh1;    // lowest bit of digit 1
};
struct HistJobs {
  HistJob j[N_SORTS];
  uint32_t* part;  // [N_SORTS][HIST_MAX_BLOCKS][8 * 256] per-workgroup counts
  // the correlation table's plan and emptying, by the workgroups of slice
  // blockIdx.y == jt_slice
  int jt_slice;
  int jt_P;          // processes (0: more than JT_PROCS, hashed slots)
  int64_t jt_cap;    // most dense slots
  int64_t jt_hsize;  // hashed table size (a power of two, a multiple of 4)
  uint32_t* jt_L;
  uint32_t* jt_K;
  uint32_t* jt_C;
};

// Digit histograms of several sort inputs in one launch (blockIdx.y picks
// the sort).  Each workgroup counts a contiguous share of the keys in LDS
// and stores its table; the plan kernel that follows sums the tables.  One
// more slice of workgroups takes the correlation-table plan and empties the
// table's slots in use, beside the counting.  No
// global atomics and no fences: counters shared by many workgroups serialise
// on their cache line, and a device-scope fence writes back the whole L2.
// The grid is sized so that every CU holds a share (HIST_CHUNK keys at
// least per workgroup, HIST_MAX_BLOCKS at most per sort).
//
// A round takes HIST_ROUND keys: the workgroup loads them coalesced (16
// bytes a lane) into LDS, then each thread reads back HIST_U consecutive
// keys (one row, padded so that the 16-byte reads of a wave meet distinct
// banks).  The next round's loads are in flight while a round is counted.
constexpr int HIST_THREADS = 512;
constexpr int HIST_U = 8;                           // consecutive keys per thread and round
constexpr int HIST_ROUND = HIST_THREADS * HIST_U;  // keys per round
constexpr int HIST_ROW = HIST_U + 2;                // u64 words per thread row (16 bytes of padding)

// Counts one thread's keys.  Digits below `first` (left to the refine pass)
// are not counted.
//
// A full wave (every lane holds HIST_U valid keys, the usual case) runs
// without branches per key.  Digits 0 and 1 (nanoseconds, correlation ids)
// differ from key to key: every key adds one to its bin.  A higher digit
// that all of the wave's keys share is added once for the wave (the 64
// lanes would otherwise add to one LDS word one after another); otherwise
// each lane adds each run of equal digits once, at its last key, and the
// other keys add to a word of the lane's own (s_spare), which costs an LDS
// access but neither a conflict nor a branch.
//
// A partial wave (the end of the range; nv valid keys, 0 past the end)
// takes the same counts with a branch per key.
template <int ND>
__device__ __forceinline__ void hist_count(uint32_t* h, uint32_t* s_spare, const uint64_t* k, int nv, int first,
                                           bool full) {
  const int lane = threadIdx.x & (WAVE - 1);
  if (full) {
    // bits that differ between any two keys of the wave
    const uint32_t f_lo = __builtin_amdgcn_readfirstlane((uint32_t)k[0]);
    const uint32_t f_hi = __builtin_amdgcn_readfirstlane((uint32_t)(k[0] >> 32));
    uint64_t x = k[0] ^ (((uint64_t)f_hi << 32) | f_lo);
#pragma unroll
    for (int u = 1; u < HIST_U; ++u) x |= k[u] ^ k[0];
#pragma unroll
    for (int d = 0; d < ND; ++d) {
      const int sh = 8 * d;
      if (d < first) continue;
      if (d < 2) {
#pragma unroll
        for (int u = 0; u < HIST_U; ++u) atomicAdd(&h[d * 256 + (uint32_t)((k[u] >> sh) & 255)], 1u);
      } else if (!__any((uint32_t)((x >> sh) & 255) != 0)) {
        if (lane == 0) atomicAdd(&h[d * 256 + (uint32_t)((k[0] >> sh) & 255)], (uint32_t)(WAVE * HIST_U));
      } else {
        uint32_t run = 1, v = (uint32_t)((k[0] >> sh) & 255);
#pragma unroll
        for (int u = 0; u < HIST_U; ++u) {
          const uint32_t nx = u + 1 < HIST_U ? (uint32_t)((k[u + 1] >> sh) & 255) : 256u;
          const bool end = nx != v;
          atomicAdd(end ? &h[d * 256 + v] : &s_spare[lane], run);
          run = end ? 1u : run + 1u;
          v = nx;
        }
      }
    }
    return;
  }
#pragma unroll
  for (int d = 0; d < ND; ++d) {
    const int sh = 8 * d;
    if (d < first) continue;
    if (d < 2) {
#pragma unroll
      for (int u = 0; u < HIST_U; ++u)
        if (u < nv) atomicAdd(&h[d * 256 + (uint32_t)((k[u] >> sh) & 255)], 1u);
    } else {
      uint32_t cur = (uint32_t)((k[0] >> sh) & 255), run = 1;
#pragma unroll
      for (int u = 1; u < HIST_U; ++u) {
        const uint32_t v = (uint32_t)((k[u] >> sh) & 255);
        if (u < nv) {
          if (v != cur) {
            atomicAdd(&h[d * 256 + cur], run);
            cur = v;
            run = 0;
          }
          ++run;
        }
      }
      if (nv > 0) atomicAdd(&h[d * 256 + cur], run);
    }
  }
}

// Round loads: pair q of the round starting at r0 is keys r0 + 2q and
// r0 + 2q + 1 (16-byte loads; r0 is even).
__device__ __forceinline__ void hist_load(uint4* v, const uint64_t* __restrict__ keys, int64_t r0, int64_t hi) {
#pragma unroll
  for (int i = 0; i < HIST_U / 2; ++i) {
    const int64_t g = r0 + 2 * (int64_t)(i * HIST_THREADS + threadIdx.x);
    v[i] = make_uint4(0u, 0u, 0u, 0u);
    if (g + 1 < hi) {
      v[i] = *reinterpret_cast<const uint4*>(keys + g);
    } else if (g < hi) {
      const uint64_t x = keys[g];
      v[i].x = (uint32_t)x;
      v[i].y = (uint32_t)(x >> 32);
    }
  }
}

// The next round's loads are in flight while a round is counted.  Keys are
// shifted right by `pre` (sh1 - 8) as they are read, so that digit d >= 1
// is bits 8d .. 8d+7 of the shifted key.
template <int ND>
__device__ __forceinline__ void hist_range(uint32_t* h, uint32_t* s_spare, uint64_t* s_row,
                                           const uint64_t* __restrict__ keys, int64_t lo, int64_t hi, int first,
                                           int pre) {
  const int t = threadIdx.x;
  uint4 v[HIST_U / 2];
  hist_load(v, keys, lo, hi);
  for (int64_t r0 = lo; r0 < hi; r0 += HIST_ROUND) {
    // pair q goes to row q / (HIST_U / 2)
#pragma unroll
    for (int i = 0; i < HIST_U / 2; ++i) {
      const int q = i * HIST_THREADS + t;
      *reinterpret_cast<uint4*>(s_row + (q / (HIST_U / 2)) * HIST_ROW + 2 * (q % (HIST_U / 2))) = v[i];
    }
    __syncthreads();
    uint64_t k[HIST_U];
#pragma unroll
    for (int i = 0; i < HIST_U / 2; ++i) {
      const uint4 w = *reinterpret_cast<const uint4*>(s_row + t * HIST_ROW + 2 * i);
      k[2 * i] = ((uint64_t)w.x | ((uint64_t)w.y << 32)) >> pre;
      k[2 * i + 1] = ((uint64_t)w.z | ((uint64_t)w.w << 32)) >> pre;
    }
    if (r0 + HIST_ROUND < hi) hist_load(v, keys, r0 + HIST_ROUND, hi);
    const int nv = (int)max<int64_t>(0, min<int64_t>(HIST_U, hi - (r0 + (int64_t)t * HIST_U)));
    const int wv = __builtin_amdgcn_readfirstlane(t / WAVE);
    const bool full = r0 + (int64_t)(wv + 1) * WAVE * HIST_U <= hi;  // the wave's keys are all valid
    hist_count<ND>(h, s_spare, k, nv, first, full);
    __syncthreads();  // the rows are rewritten by the next round
  }
}

__global__ __launch_bounds__(HIST_THREADS) void k_digit_hist(HistJobs jobs, DevState* ds) {
  __shared__ uint32_t h[8 * 256];
  __shared__ uint32_t s_spare[WAVE];  // adds that count nothing (never read)
  __shared__ __align__(16) uint64_t s_row[HIST_THREADS * HIST_ROW];
  __shared__ uint32_t s_direct;
  __shared__ int64_t s_slots;
  if ((int)blockIdx.y == jobs.jt_slice) {
    // every workgroup takes the plan (the first stores it), then they empty
    // the slots in use: launch and kernel words, and with hashed slots the
    // claim words
    if (threadIdx.x < WAVE) {
      int64_t slots = 0;
      const bool direct = jt_plan_wave(ds, jobs.jt_P, jobs.jt_cap, jobs.jt_hsize, blockIdx.x == 0, &slots);
      if (threadIdx.x == 0) {
        s_direct = direct ? 1u : 0u;
        s_slots = slots;
      }
    }
    __syncthreads();
    const int64_t q4 = cdiv(s_slots, 4);  // 16-byte words (the table is a multiple of 4 slots)
    const bool claims = !s_direct;
    const uint4 e4 = make_uint4(JT_EMPTY, JT_EMPTY, JT_EMPTY, JT_EMPTY);
    for (int64_t w = (int64_t)blockIdx.x * HIST_THREADS + threadIdx.x; w < q4; w += (int64_t)gridDim.x * HIST_THREADS) {
      reinterpret_cast<uint4*>(jobs.jt_L)[w] = e4;
      reinterpret_cast<uint4*>(jobs.jt_K)[w] = e4;
      if (claims) reinterpret_cast<uint4*>(jobs.jt_C)[w] = e4;
    }
    return;
  }
  const HistJob jb = jobs.j[blockIdx.y];
  const int64_t n = *jb.count;
  const int nblk = hist_blocks(n);
  const int blk = blockIdx.x;
  // the first digit pass's look-back words of this call's tiles (the passes
  // follow on the same stream), after the counting: its loads go first
  auto clear_status = [&]() {
    const int64_t words = cdiv(n, (int64_t)RS_TILE) * RS_LB_WORDS / 4;
    uint4* st = reinterpret_cast<uint4*>(jb.status0);
    for (int64_t w = (int64_t)blk * HIST_THREADS + threadIdx.x; w < words; w += (int64_t)gridDim.x * HIST_THREADS)
      st[w] = make_uint4(0u, 0u, 0u, 0u);
  };
  if (blk >= nblk) {
    clear_status();
    return;
  }
  // (the first barrier of the count orders these before any add)
  for (int i = threadIdx.x; i < 8 * 256; i += HIST_THREADS) h[i] = 0;
  // shares are whole multiples of 64 keys (the 16-byte loads stay aligned)
  const int64_t per = cdiv(cdiv(n, nblk), 64) * 64;
  const int64_t lo = min<int64_t>(n, (int64_t)blk * per), hi = min<int64_t>(n, lo + per);
  switch (jb.nd) {
    case 1: hist_range<1>(h, s_spare, s_row, jb.keys, lo, hi, jb.first, jb.sh1 - 8); break;
    case 2: hist_range<2>(h, s_spare, s_row, jb.keys, lo, hi, jb.first, jb.sh1 - 8); break;
    case 3: hist_range<3>(h, s_spare, s_row, jb.keys, lo, hi, jb.first, jb.sh1 - 8); break;
    case 4: hist_range<4>(h, s_spare, s_row, jb.keys, lo, hi, jb.first, jb.sh1 - 8); break;
    case 5: hist_range<5>(h, s_spare, s_row, jb.keys, lo, hi, jb.first, jb.sh1 - 8); break;
    case 6: hist_range<6>(h, s_spare, s_row, jb.keys, lo, hi, jb.first, jb.sh1 - 8); break;
    case 7: hist_range<7>(h, s_spare, s_row, jb.keys, lo, hi, jb.first, jb.sh1 - 8); break;
    default: hist_range<8>(h, s_spare, s_row, jb.keys, lo, hi, jb.first, jb.sh1 - 8); break;
  }
  __syncthreads();
  uint32_t* part = jobs.part + ((int64_t)jb.id * HIST_MAX_BLOCKS + blk) * 8 * 256;
  for (int j = threadIdx.x; j < jb.nd * 256; j += HIST_THREADS) part[j] = h[j];
  clear_status();
}

// Plan of one digit of one sort (blockIdx.x = digit, blockIdx.y = sort):
// the digit's counts summed over the workgroup tables, its trivial flag
// (one bin holds every key) and each bin's exclusive offset.  A wave reads a
// table's 256 counts as 16-byte loads (four bins a lane); the 16 waves take
// every 16th table, PLAN_LOADS tables in flight per lane.
constexpr int PLAN_THREADS = 1024;
constexpr int PLAN_GROUPS = PLAN_THREADS / WAVE;
constexpr int PLAN_LOADS = 16;

__global__ __launch_bounds__(PLAN_THREADS) void k_hist_plan(HistJobs jobs, DevState* ds) {
  __shared__ __align__(16) uint32_t s_part[PLAN_GROUPS][256];
  __shared__ uint32_t s_scan[PLAN_THREADS / WAVE + 1];
  const HistJob jb = jobs.j[blockIdx.y];
  const int d = blockIdx.x;
  if (d >= jb.nd) return;
  const int64_t n = *jb.count;
  const int nblk = hist_blocks(n);
  const int lane = threadIdx.x & (WAVE - 1), grp = threadIdx.x / WAVE;
  const uint4* src = reinterpret_cast<const uint4*>(jobs.part + (int64_t)jb.id * HIST_MAX_BLOCKS * 8 * 256 + d * 256) + lane;
  uint4 c4 = make_uint4(0u, 0u, 0u, 0u);
  for (int b0 = grp; b0 < nblk; b0 += PLAN_LOADS * PLAN_GROUPS) {
    uint4 v[PLAN_LOADS];
#pragma unroll
    for (int b = 0; b < PLAN_LOADS; ++b) {
      const int blk = b0 + b * PLAN_GROUPS;
      v[b] = blk < nblk ? src[(int64_t)blk * 8 * 256 / 4] : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int b = 0; b < PLAN_LOADS; ++b) {
      c4.x += v[b].x;
      c4.y += v[b].y;
      c4.z += v[b].z;
      c4.w += v[b].w;
    }
  }
  *reinterpret_cast<uint4*>(&s_part[grp][4 * lane]) = c4;
  __syncthreads();
  const int bin = threadIdx.x & 255;
  uint32_t c = 0;
  if (threadIdx.x < 256) {
#pragma unroll
    for (int g = 0; g < PLAN_GROUPS; ++g) c += s_part[g][bin];
  }
  // every thread joins the barriers below; only the first 256 carry a bin
  const bool full = threadIdx.x < 256 && c == (uint32_t)n;
  if (__syncthreads_or(full) && threadIdx.x == 0) atomicOr(&ds->sort_trivial[jb.id], 1u << d);
  if (d < jb.first && threadIdx.x == 0) atomicOr(&ds->sort_trivial[jb.id], (1u << d) | (1u << 31));
  uint32_t total = 0;
  const uint32_t ex = block_excl_sum<PLAN_THREADS>(threadIdx.x < 256 ? c : 0u, s_scan, &total);
  if (threadIdx.x < 256) ds->hist[jb.id][d][bin] = ex;
  // every key lies in one bin of a counted digit: a total other than n means
  // the histogram and the passes disagree, and the passes must not scatter
  if (d >= jb.first && total != (uint32_t)n && threadIdx.x == 0) set_status(ds, DS_LOGIC);
}

struct SortJob {
  uint64_t* k[2];
  uint32_t* v[2];
  const int32_t* count;
  uint32_t* status0;  // [tiles_max][RS_LB_WORDS] look-back words of the first digit (cleared by the init kernel)
  uint32_t* status1;  // [nd - 1][tiles_max][RS_LB_WORDS] later digits (each cleared by the previous pass)
  int64_t tiles_max;
  int nd, id, first;
  int sh1;  // lowest bit of digit 1 (digit d >= 1 is bits sh1 + 8(d-1) ..)
  int d;    // the digit this launch sorts on
};
struct SortJobs {
  SortJob j[N_SORTS];  // slots m.. repeat slot 0
  int m;               // sorts in the launch
};

// One digit pass of up to N_SORTS independent sorts (each on its own digit).
// 512 threads rank a tile of 4096 keys; the tile (48 KB) and the per-wave
// digit counts (8 KB, in the key area until the keys are placed) keep the
// LDS of a workgroup under a third of the CU's (with the allocation
// granularity), so three tiles share a CU.
//
// The grid is one-dimensional and sized for every sort's largest input.
// The tiles whose digit moves data are numbered sort after sort, and
// workgroup b sorts tile b; the workgroups past the last tile leave at
// once, after the real tiles have been dispatched.  A tile's look-back waits
// only for tiles of lower number, whose workgroups have lower indices: the
// dispatcher starts workgroups in index order, so the lowest unfinished
// tile always has its workgroup running and every wait ends (a wait that
// exceeds its bound gives up with an error all the same).  No tile ticket:
// a counter that every workgroup increments is one address, served one
// request at a time, and it held the last tiles back by microseconds.
static_assert(RS_ITEMS % 4 == 0, "digits are packed four to a register");
static_assert(RS_THREADS % 256 == 0 && RS_LB_WORDS == 512, "look-back slices: 256 digits per slice, counts + window sums");
static_assert(HIST_U % 2 == 0, "histogram keys are loaded in 16-byte pairs");
constexpr int RS_NW = RS_THREADS / WAVE;  // waves per workgroup
constexpr int RS_NSL = RS_THREADS / 256;  // look-back slices per digit
constexpr int RS_LB_WIN = 16;             // positions polled per slice and round trip

__global__ __launch_bounds__(RS_THREADS) __attribute__((amdgpu_waves_per_eu(RS_WAVES_PER_EU)))
void k_radix_pass(SortJobs jobs, DevState* ds) {
  constexpr int NW = RS_NW, NSL = RS_NSL, LB_WIN = RS_LB_WIN;
  __shared__ uint64_t s_key[RS_TILE];
  __shared__ uint32_t s_val[RS_TILE];
  __shared__ uint32_t s_local[256];
  __shared__ uint32_t s_scan[NW + 1];
  __shared__ uint32_t s_lb_sum[NSL][256];
  __shared__ uint8_t s_lb_state[NSL][256];
  static_assert(NW * 256 * 4 <= RS_TILE * 8, "per-wave counts must fit the key area");
  uint32_t(*s_wh)[256] = reinterpret_cast<uint32_t(*)[256]>(s_key);
  // the global offsets reuse the look-back's scratch once the look-back is over
  uint32_t* s_glob = &s_lb_sum[0][0];

  const int tid = threadIdx.x, lane = lane_id(), wv = tid / WAVE;
  const int dgt = tid & 255, slice = tid >> 8;
  const uint32_t b = blockIdx.x;
  // Per sort: the next digit's look-back words of tile index b are cleared
  // here (the next pass starts only after this one has ended; the words of
  // a digit are used by that digit's pass alone), the first
  // pass records which buffer will hold the result (the parity of the
  // digits that move data), and the tiles of a digit on which every key
  // agrees (plan of the histogram kernel) are not sorted at all.
  // The counts and plans of all sorts are loaded together (one round trip;
  // the slots past the launch's sorts repeat its first).
  uint32_t nn[N_SORTS], tr[N_SORTS], nt[N_SORTS];
  const int32_t* cp[N_SORTS];
  if (ds->status & DS_LOGIC) return;  // a digit plan did not add up: nothing is moved
  int ids[N_SORTS];
#pragma unroll
  for (int i = 0; i < N_SORTS; ++i) {
    cp[i] = jobs.j[i].count;
    ids[i] = jobs.j[i].id;
  }
#pragma unroll
  for (int i = 0; i < N_SORTS; ++i) {
    nn[i] = (uint32_t)*cp[i];
    tr[i] = ds->sort_trivial[ids[i]];
  }
#pragma unroll
  for (int i = 0; i < N_SORTS; ++i) {
    nt[i] = 0;
    if (i >= jobs.m) continue;
    const SortJob& jb = jobs.j[i];
    const uint32_t tiles = (nn[i] + RS_TILE - 1) / RS_TILE;
    // (only for a next digit that moves data: a skipped digit's words are never read)
    if (b < tiles && jb.d + 1 < jb.nd && !((tr[i] >> (jb.d + 1)) & 1) && tid < RS_LB_WORDS)
      jb.status1[((int64_t)(jb.d - jb.first) * jb.tiles_max + b) * RS_LB_WORDS + tid] = 0u;
    if (jb.d == jb.first && b == 0 && tid == 0)
      ds->sort_parity[jb.id] = (uint32_t)(popc(~tr[i] & ((jb.nd >= 32 ? 0u : 1u << jb.nd) - 1u)) & 1);
    nt[i] = ((tr[i] >> jb.d) & 1) ? 0u : tiles;
  }
  int sel = -1;
  uint32_t t = b;
#pragma unroll
  for (int i = 0; i < N_SORTS; ++i) {
    if (sel < 0) {
      if (t < nt[i])
        sel = i;
      else
        t -= nt[i];
    }
  }
  if (sel < 0) return;
  const SortJob& jb = jobs.j[sel];
  const int d = jb.d, id = jb.id;
  // selects, not a dynamically indexed array: the values stay in registers
  uint32_t n = nn[0], triv = tr[0];
#pragma unroll
  for (int i = 1; i < N_SORTS; ++i) {
    if (sel == i) {
      n = nn[i];
      triv = tr[i];
    }
  }
  const uint32_t gexcl = ds->hist[id][d][dgt];
  const int parity = popc(~triv & ((1u << d) - 1u)) & 1;
  const uint64_t* kin = jb.k[parity];
  uint64_t* kout = jb.k[parity ^ 1];
  const uint32_t* vin = jb.v[parity];
  uint32_t* vout = jb.v[parity ^ 1];
  uint32_t* status =
      d == jb.first ? jb.status0 : jb.status1 + (int64_t)(d - jb.first - 1) * jb.tiles_max * RS_LB_WORDS;
  const int tile = (int)t;
  const int64_t base = (int64_t)tile * RS_TILE;

  const int shift = d == 0 ? 0 : jb.sh1 + 8 * (d - 1);
  uint64_t key[RS_ITEMS];
  uint32_t val[RS_ITEMS];
  uint32_t rank[RS_ITEMS];  // rank among the wave's equal digits, then the tile position
  // each wave owns RS_ITEMS * 64 consecutive keys, item j of lane l at j*64+l
  // 32-bit offsets from the uniform buffer bases (n < 2^30)
  const uint32_t wbase = (uint32_t)base + (uint32_t)wv * (RS_ITEMS * WAVE) + (uint32_t)lane;
  // Loads past the end read the last key instead (the index is clamped, not
  // branched on, so that all of them are in flight together); such items
  // carry digit 256 and are never placed.
#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) {
    const uint32_t idx = min(wbase + j * WAVE, n - 1);
    key[j] = kin[idx];
    val[j] = vin[idx];
  }
  // the counters are cleared while the loads are in flight; the tile's
  // digit counts sit in the row area until the rows are placed
  uint32_t* s_cnt = s_val;
  for (int i = tid; i < NW * 256; i += RS_THREADS) (&s_wh[0][0])[i] = 0;
  if (tid < 256) s_cnt[tid] = 0;
  __syncthreads();
  // The items' digits, four to a register; the thread's first nv items lie
  // before the end of the input (an item past it has digit 256).
  uint32_t dpk[RS_ITEMS / 4] = {};
#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) dpk[j >> 2] |= (uint32_t)((key[j] >> shift) & 255) << (8 * (j & 3));
  const int nv = wbase < n ? (int)min((n - wbase + WAVE - 1) / WAVE, (uint32_t)RS_ITEMS) : 0;
  auto digit_of = [&](int j) -> int {
    return j < nv ? (int)__builtin_amdgcn_ubfe(dpk[j >> 2], 8 * (j & 3), 8) : 256;
  };

  // The tile's digit counts come first (LDS atomics) and are published
  // before the ranking, so that a successor's look-back finds them ready.
#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) {
    const int dg = digit_of(j);
    if (dg < 256) atomicAdd(&s_cnt[dg], 1u);
  }
  __syncthreads();
  const uint32_t cnt = tid < 256 ? s_cnt[tid] : 0u;
  // this tile's words: its own counts (then its prefix) and its window sums
  uint32_t* st = status + (uint32_t)tile * RS_LB_WORDS;
  if (tid < 256) st_agent(&st[tid], (tile == 0 ? RS_FLAG_P : RS_FLAG_A) | cnt);
  if (tile == 0 && tid < 256) st_agent(&st[256 + tid], RS_FLAG_P | cnt);

  // Wave-private ranking in input order: items in order, lanes in order.
  // A lane's peers (the lanes with its digit) are found bit by bit: for each
  // digit bit, the lanes whose bit differs from this lane's are marked
  // mismatched (m is 0 or all ones, the lane's bit; the ballot holds every
  // lane's), one three-input bit operation per 32-lane half.
  constexpr int OR_XOR = 0xF0 | (0xCC ^ 0xAA);  // truth table of a | (b ^ c)
#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) {
    const int dg = digit_of(j);
    const bool ok = dg < 256;
    const uint64_t okm = ballot(ok);  // lanes past the end are nobody's peers
    uint32_t mis_lo = ~(uint32_t)okm, mis_hi = ~(uint32_t)(okm >> 32);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const uint32_t m = (uint32_t)__builtin_amdgcn_sbfe(dg, b, 1);
      const uint64_t bb = __builtin_amdgcn_uicmp(m, 0u, 33);  // ballot(m != 0)
      mis_lo = __builtin_amdgcn_bitop3_b32(mis_lo, (uint32_t)bb, m, OR_XOR);
      mis_hi = __builtin_amdgcn_bitop3_b32(mis_hi, (uint32_t)(bb >> 32), m, OR_XOR);
    }
    // peers in lower lanes, and all peers
    const uint32_t below = __builtin_amdgcn_mbcnt_hi(~mis_hi, __builtin_amdgcn_mbcnt_lo(~mis_lo, 0u));
    const uint32_t before = ok ? s_wh[wv][dg] : 0u;
    rank[j] = before + below;
    __builtin_amdgcn_wave_barrier();
    if (ok && below == 0) s_wh[wv][dg] = before + (uint32_t)(__builtin_popcount(~mis_lo) + __builtin_popcount(~mis_hi));
    __builtin_amdgcn_wave_barrier();
  }
  __syncthreads();

  // Threads 0..255 own one digit each: the digit's first tile position
  // (exclusive sum over digits), then each wave's (plus the exclusive sum
  // over waves), in the key area.
  const uint32_t local_excl = block_excl_sum<RS_THREADS>(cnt, s_scan, nullptr);
  if (tid < 256) {
    s_local[tid] = local_excl;
    uint32_t run = local_excl;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const uint32_t c = s_wh[w][tid];
      s_wh[w][tid] = run;
      run += c;
    }
  }
  __syncthreads();

  // Tile positions, then the tile is reordered in LDS before the rest of
  // the look-back, so that no key or row stays in a register while the
  // predecessors are polled.
#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) {
    const int dg = digit_of(j);
    if (dg < 256) rank[j] += s_wh[wv][dg];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) {
    if (digit_of(j) < 256 && in_range(ds, rank[j], RS_TILE)) {
      s_key[rank[j]] = key[j];
      s_val[rank[j]] = val[j];
    }
  }

  // Look-back: every digit has NSL threads, each polling LB_WIN positions
  // per round trip (independent loads), WIN = NSL * LB_WIN per round.  The
  // first round polls the WIN nearest predecessors' own counts.  If none of
  // them has published its inclusive prefix, the tile publishes the sum of
  // its window (its count and those WIN), and the later rounds poll the
  // window sums ending WIN + 1, 2 (WIN + 1), ... tiles before it, which
  // tile into the rest: WIN (WIN + 1) tiles per round instead of WIN.  A
  // round is used up to the nearest position that published a prefix; a
  // round with an unpublished position before that is polled again.  The
  // loop condition is uniform over the workgroup.
  uint32_t excl = 0;
  if (tile > 0) {
    constexpr int WIN = NSL * LB_WIN;
    int pred = tile - 1;  // newest position not yet counted
    int stride = 1;       // 1: own counts, WIN + 1: window sums
    bool done = false;
    uint64_t t0 = 0;
    for (;;) {
      const uint32_t* src = status + (stride == 1 ? 0 : 256) + dgt;
      const int top = pred - stride * slice * LB_WIN;
      uint32_t sum = 0;
      int state = 1;  // 0: not ready, 1: all partial sums, 2: reached a prefix
      if (!done) {
        uint32_t sv[LB_WIN];
#pragma unroll
        for (int i = 0; i < LB_WIN; ++i)
          sv[i] = ld_agent(&src[(uint32_t)max(top - stride * i, 0) * RS_LB_WORDS]);
#pragma unroll
        for (int i = 0; i < LB_WIN; ++i) {
          const bool real = top - stride * i >= 0;
          const uint32_t f = real ? sv[i] >> 30 : 2u;  // before tile 0: prefix 0
          if (state == 1) {
            if (f == 0) {
              state = 0;
            } else {
              sum += real ? sv[i] & RS_VAL : 0u;
              if (f == 2) state = 2;
            }
          }
        }
      }
      s_lb_sum[slice][dgt] = sum;
      s_lb_state[slice][dgt] = (uint8_t)state;
      __syncthreads();
      bool again = false;
      if (!done) {
        // combine the slices newest-first; every thread of the digit does it
        uint32_t add = 0;
        int res = 1;
#pragma unroll
        for (int sl = 0; sl < NSL; ++sl) {
          const int stt = s_lb_state[sl][dgt];
          if (res == 1) {
            if (stt == 0) {
              res = 0;
            } else {
              add += s_lb_sum[sl][dgt];
              if (stt == 2) res = 2;
            }
          }
        }
        if (res == 0) {
          const uint64_t now = spin_clock();
          if (t0 == 0) t0 = now;
          if (now - t0 > SPIN_TICKS) {
            set_status(ds, DS_SPIN);
            done = true;
          } else {
            again = true;
          }
        } else {
          excl += add;
          if (res == 2) {
            done = true;
          } else if (stride == 1) {
            if (tid < 256) st_agent(&st[256 + tid], RS_FLAG_A | ((excl + cnt) & RS_VAL));
            pred -= WIN;
            stride = WIN + 1;
          } else {
            pred -= stride * WIN;
          }
          if (pred < 0) done = true;
        }
      }
      if (!__syncthreads_or(!done)) break;
      if (again) __builtin_amdgcn_s_sleep(1);
    }
    if (tid < 256) {
      st_agent(&st[tid], RS_FLAG_P | ((excl + cnt) & RS_VAL));
      st_agent(&st[256 + tid], RS_FLAG_P | ((excl + cnt) & RS_VAL));
    }
  }
  // the look-back loop ends on a barrier after its last read of s_lb_sum
  if (tid < 256) s_glob[tid] = gexcl + excl;
  __syncthreads();

  const uint32_t tile_n = (uint32_t)min((int64_t)RS_TILE, (int64_t)n - base);
  for (uint32_t i = tid; i < tile_n; i += RS_THREADS) {
    const uint64_t kk = s_key[i];
    const int dg = (int)((kk >> shift) & 255);
    const uint32_t gpos = s_glob[dg] + (i - s_local[dg]);
    if (in_bounds(ds, gpos, n)) {
      kout[gpos] = kk;
      vout[gpos] = s_val[i];
    }
  }
}

void launch_hist_multi(Ctx& c, SortBufs* const* s, const int32_t* const* count, int k) {
  HistJobs jobs{};
  jobs.part = c.hist_part;
  int m = 0, nd = 0;
  int64_t n_max = 1;
  for (int i = 0; i < k; ++i) {
    if (s[i]->nd == 0) continue;
    jobs.j[m++] = HistJob{s[i]->k[0], count[i], s[i]->status0, s[i]->nd, s[i]->id, s[i]->first, s[i]->sh1};
    n_max = std::max<int64_t>(n_max, s[i]->n_max);
    nd = std::max(nd, s[i]->nd);
  }
  jobs.jt_slice = m;
  jobs.jt_P = c.P <= JT_PROCS ? c.P : 0;
  jobs.jt_cap = c.jt_cap;
  jobs.jt_hsize = c.jt_hsize;
  jobs.jt_L = c.jt_L;
  jobs.jt_K = c.jt_K;
  jobs.jt_C = c.jt_C;
  const int64_t grid = std::min<int64_t>(cdiv(std::max<int64_t>(n_max, 2 * c.n), HIST_CHUNK), HIST_MAX_BLOCKS);
  hipLaunchKernelGGL(k_digit_hist, dim3((unsigned)grid, (unsigned)(m + 1)), dim3(HIST_THREADS), 0, c.st, jobs,
                     c.ds);
  if (m > 0)
    hipLaunchKernelGGL(k_hist_plan, dim3((unsigned)nd, (unsigned)m), dim3(PLAN_THREADS), 0, c.st, jobs, c.ds);
}

// Passes p0 .. p1-1 of up to N_SORTS sorts, one launch per pass: pass p of
// a sort is its digit first + p (its lowest digit is left to the refine
// pass when first is 1).  The grid covers every sort's largest input.
void launch_sort_multi(Ctx& c, SortBufs* const* s, const int32_t* const* count, int k, int p0, int p1) {
  for (int p = p0; p < p1; ++p) {
    SortJobs jobs{};
    int64_t grid = 0;
    int m = 0;
    for (int i = 0; i < k; ++i) {
      const int d = s[i]->first + p;
      if (d >= s[i]->nd) continue;
      jobs.j[m++] = SortJob{{s[i]->k[0], s[i]->k[1]}, {s[i]->v[0], s[i]->v[1]}, count[i], s[i]->status0,
                            s[i]->status1, s[i]->tiles_max, s[i]->nd, s[i]->id, s[i]->first, s[i]->sh1, d};
      grid += s[i]->tiles_max;
    }
    if (m == 0) continue;
    jobs.m = m;
    for (int i = m; i < N_SORTS; ++i) jobs.j[i] = jobs.j[0];
    hipLaunchKernelGGL(k_radix_pass, dim3((unsigned)grid), dim3(RS_THREADS), 0, c.st, jobs, c.ds);
  }
}

// ------------------------------------------------------------------ refine
// After passes over digits 1.. only, a sort is ordered by key >> sh1 (the
// passes' lowest bit, 8 to RF_LOW_MAX); keys equal above it still sit in
// row order (the passes are stable).  The
// refine pass orders each such run by the full key, and keys that are
// equal by the sort's own tie rule: the row (stable) for the timeline; for
// the containment list, ops of equal key by end time down, then row (the
// rule that nests an op that starts with its parent inside it).  The
// containment list is refined even when every digit was sorted (runs of
// equal keys, shift 0), for that tie rule.  Runs up to RF_SHORT are ordered
// by one thread; the workgroup that finds a longer run sorts it.
struct RefineJob {
  uint64_t* k[2];
  uint32_t* v[2];
  const int32_t* count;
  int id;        // sort index (parity)
  int contain;   // 1: containment tie rule
  int slot;      // list index (the sort's id)
  int shift;     // runs are keys equal above this bit (the passes' lowest, or 0 when every digit was sorted)
};
struct RefineJobs {
  RefineJob j[N_SORTS];
  const int64_t* te;
};

// a before b in the refined order (a and b from one run)
__device__ __forceinline__ bool rf_before(const RefineJob& jb, const int64_t* te, uint64_t ka, uint32_t ra, uint64_t kb,
                                          uint32_t rb) {
  if (ka != kb) return ka < kb;
  if (jb.contain && (ka & 1) == 0) {  // two ops starting together: the longer first
    const int64_t ta = te[ra], tb = te[rb];  // one process: raw ends compare like corrected
    if (ta != tb) return ta > tb;
  }
  return ra < rb;
}

constexpr int RF_THREADS = 256;
constexpr int RF_ITEMS = 4;
constexpr int RF_TILE = RF_THREADS * RF_ITEMS;  // positions whose runs a workgroup orders
constexpr int RF_SPAN = 1 + RF_TILE + RF_SHORT;  // the position before the tile, the tile, and its runs' reach

// One long run (more than RF_SHORT keys, starting at position p), sorted by
// the whole workgroup: the run is copied into the sort's other buffer (free
// once the passes are done) at the same positions, sorted there by a
// bitonic network that only compares pairs inside the run (the positions
// past its end act as +infinity, and every comparator puts the smaller
// element first), and copied back.  Only the high part of the run's keys
// (above the shift) is read by other workgroups meanwhile, and it is the
// same for every key of the run.
__device__ void refine_long_run(const RefineJob& jb, const int64_t* te, uint64_t* keys, uint32_t* vals, uint64_t* sk,
                                uint32_t* sv, int64_t p, int64_t n, int64_t* s_len) {
  const uint64_t hi = keys[p] >> jb.shift;
  if (threadIdx.x == 0) *s_len = n - p;
  __syncthreads();
  // the run's end: the first position past it, found RF_THREADS at a time
  for (int64_t b = p; b < n; b += RF_THREADS) {
    const int64_t i = b + threadIdx.x;
    if (i < n && (keys[i] >> jb.shift) != hi) atomicMin((unsigned long long*)s_len, (unsigned long long)(i - p));
    __syncthreads();
    if (*s_len < n - p) break;
    __syncthreads();
  }
  const int64_t len = *s_len;
  for (int64_t i = threadIdx.x; i < len; i += RF_THREADS) {
    sk[p + i] = keys[p + i];
    sv[p + i] = vals[p + i];
  }
  __syncthreads();
  int64_t m = 1;
  while (m < len) m <<= 1;
  for (int64_t size = 2; size <= m; size <<= 1) {
    for (int64_t stride = size >> 1; stride > 0; stride >>= 1) {
      for (int64_t i = threadIdx.x; i < len; i += RF_THREADS) {
        // first step of a merge: the mirror in the block; then halvings
        const int64_t l = stride == (size >> 1) ? (i ^ (size - 1)) : (i ^ stride);
        if (l > i && l < len) {
          const uint64_t ki = sk[p + i], kl = sk[p + l];
          const uint32_t ri = sv[p + i], rl = sv[p + l];
          if (rf_before(jb, te, kl, rl, ki, ri)) {
            sk[p + i] = kl;
            sv[p + i] = rl;
            sk[p + l] = ki;
            sv[p + l] = ri;
          }
        }
      }
      __syncthreads();
    }
  }
  for (int64_t i = threadIdx.x; i < len; i += RF_THREADS) {
    keys[p + i] = sk[p + i];
    vals[p + i] = sv[p + i];
  }
  __syncthreads();
}

// A workgroup stages its tile's keys and rows in LDS (coalesced), with the
// position before the tile and the RF_SHORT after it, and finds the tile's
// run starts there.  A thread per run orders it in LDS (insertion sort:
// the runs are short, and many are in order already) and marks the
// positions that moved; the workgroup then writes those back, coalesced.
// A run longer than RF_SHORT (rare) is noted, and the workgroup sorts it
// afterwards in the sort's other buffer.
__global__ __launch_bounds__(RF_THREADS) void k_refine(RefineJobs jobs, DevState* ds) {
  __shared__ uint64_t s_k[RF_SPAN];
  __shared__ uint32_t s_v[RF_SPAN];
  __shared__ uint8_t s_chg[RF_SPAN];       // 1: the position moved
  __shared__ int32_t s_run[RF_TILE / 2];  // span indices of the tile's run starts (a run has two keys or more)
  __shared__ int s_nrun;
  __shared__ int64_t s_long[RF_TILE / (RF_SHORT + 1) + 1];  // positions of the tile's long runs
  __shared__ int s_nlong;
  __shared__ int64_t s_len;
  const RefineJob& jb = jobs.j[blockIdx.y];
  const int64_t n = *jb.count;
  const int64_t t0 = (int64_t)blockIdx.x * RF_TILE;
  if (n < 2 || t0 >= n) return;
  const int par = (int)ds->sort_parity[jb.id];
  uint64_t* keys = jb.k[par];
  uint32_t* vals = jb.v[par];
  if (threadIdx.x == 0) {
    s_nrun = 0;
    s_nlong = 0;
  }
  // span index i holds position t0 - 1 + i (clamped to the list); the
  // loads are issued together (the span's last few are loaded twice)
  constexpr int RF_LD = (RF_SPAN + RF_THREADS - 1) / RF_THREADS;
  uint64_t lk[RF_LD];
  uint32_t lv[RF_LD];
#pragma unroll
  for (int u = 0; u < RF_LD; ++u) {
    const int i = min(u * RF_THREADS + (int)threadIdx.x, RF_SPAN - 1);
    int64_t q = t0 - 1 + i;
    q = q < 0 ? 0 : q >= n ? n - 1 : q;
    lk[u] = keys[q];
    lv[u] = vals[q];
  }
#pragma unroll
  for (int u = 0; u < RF_LD; ++u) {
    const int i = min(u * RF_THREADS + (int)threadIdx.x, RF_SPAN - 1);
    s_k[i] = lk[u];
    s_v[i] = lv[u];
    s_chg[i] = 0;
  }
  __syncthreads();
  const int sh = jb.shift;
  // the first positions of runs of two or more keys equal above the shift
#pragma unroll
  for (int u = 0; u < RF_ITEMS; ++u) {
    const int i = 1 + u * RF_THREADS + (int)threadIdx.x;
    const int64_t p = t0 - 1 + i;
    const uint64_t hk = s_k[i] >> sh;
    const bool start = p + 1 < n && (s_k[i + 1] >> sh) == hk && !(p > 0 && (s_k[i - 1] >> sh) == hk);
    const uint64_t b = ballot(start);
    if (b == 0) continue;
    int at = 0;
    if (lane_id() == __ffsll((unsigned long long)b) - 1) at = atomicAdd(&s_nrun, popc(b));
    at = __shfl(at, __ffsll((unsigned long long)b) - 1, WAVE);
    if (start) s_run[at + popc(b & lanemask_lt())] = i;
  }
  __syncthreads();
  const int nrun = s_nrun;
  for (int ri = threadIdx.x; ri < nrun; ri += RF_THREADS) {
    const int i = s_run[ri];
    const int64_t p = t0 - 1 + i;
    const uint64_t hk = s_k[i] >> sh;
    // the run's length (a run that reaches the span's end is longer than RF_SHORT)
    int len = 2;
    while (i + len < RF_SPAN && p + len < n && (s_k[i + len] >> sh) == hk) ++len;
    if (len > RF_SHORT || (i + len == RF_SPAN && p + len < n)) {
      const int at = atomicAdd(&s_nlong, 1);
      if (in_bounds(ds, at, RF_TILE / (RF_SHORT + 1) + 1)) s_long[at] = p;
      continue;
    }
    // insertion sort in LDS; `lo` is the first position that moved
    int lo = len;
    for (int x = i + 1; x < i + len; ++x) {
      const uint64_t k = s_k[x];
      const uint32_t r = s_v[x];
      int y = x - 1;
      while (y >= i && rf_before(jb, jobs.te, k, r, s_k[y], s_v[y])) {
        s_k[y + 1] = s_k[y];
        s_v[y + 1] = s_v[y];
        --y;
      }
      if (y + 1 != x) {
        s_k[y + 1] = k;
        s_v[y + 1] = r;
        lo = min(lo, y + 1 - i);
      }
    }
    for (int j = lo; j < len; ++j) s_chg[i + j] = 1;
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < RF_LD; ++u) {
    const int i = u * RF_THREADS + (int)threadIdx.x;
    if (i < RF_SPAN && s_chg[i]) {
      keys[t0 - 1 + i] = s_k[i];
      vals[t0 - 1 + i] = s_v[i];
    }
  }
  const int nlong = min(s_nlong, RF_TILE / (RF_SHORT + 1) + 1);
  for (int q = 0; q < nlong; ++q)
    refine_long_run(jb, jobs.te, keys, vals, jb.k[par ^ 1], jb.v[par ^ 1], s_long[q], n, &s_len);
}

void launch_refine(Ctx& c) {
  RefineJobs jobs{};
  int m = 0;
  int64_t n_max = 1;
  // the containment list always (its tie rule orders ops that start
  // together); the others when a digit was left to this pass; the device and
  // op-name lists with the idle-coincidence outputs (row order breaks ties)
  const int32_t* counts[N_SORTS] = {&c.ds->nK, &c.ds->nCL, &c.ds->nK, &c.ds->nO, &c.ds->nK};
  static_assert(N_SORTS == 5, "a count for every sort");
  for (SortBufs* s : {&c.sK, &c.sC, &c.sD, &c.sO, &c.sE}) {
    const bool con = s == &c.sC;
    if (con && !c.contain) continue;
    if ((s == &c.sD || s == &c.sO) && !c.waits) continue;
    if (s == &c.sE && !c.crit) continue;
    if (!con && s->first == 0) continue;
    jobs.j[m++] = RefineJob{{s->k[0], s->k[1]}, {s->v[0], s->v[1]}, counts[s->id], s->id, con ? 1 : 0,
                            s->id, s->first ? s->sh1 : 0};
    n_max = std::max<int64_t>(n_max, s->n_max);
  }
  if (m == 0) return;
  jobs.te = c.ev.te;
  const int64_t grid = cdiv(n_max, RF_TILE);
  hipLaunchKernelGGL(k_refine, dim3((unsigned)grid, (unsigned)m), dim3(RF_THREADS), 0, c.st, jobs, c.ds);
}

}  // namespace hx
