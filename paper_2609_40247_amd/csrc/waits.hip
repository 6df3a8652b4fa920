// GPU idle coinciding with CPU ops, by op name: the idle evidence of the
// case study in Section 9.1, where a worker's waits in one Python call
// coincide with most of the GPU's idle time.
//
// Inputs, from the union scan run over two more lanes: the device lane's
// gaps above the threshold (the GPU of a process is idle where none of its
// streams is busy), in (pid, begin) order; and the coverage runs of the
// op-name lanes (the union of each op name's ranges), as start / end
// endpoints grouped by (pid, op name).  With the exclusive prefix sums Pre of
// the idle lengths, the idle time of process p before time t is
//   G(t) = Pre[i] - Pre[first of p] - (the part of interval i-1 past t),
// where i counts the intervals ordered before (p, t); an op-name run [a, b)
// holds G(b) - G(a) of idle time, and the first-of-p terms cancel.  The
// intervals' (pid, begin) are packed into one ordered word each, and every
// S-th word is staged in LDS, so a search takes its first steps in LDS and
// only its last log2(S) in memory.
#include "internal.hpp"

namespace hx {

constexpr int DG_THREADS = 512;
constexpr int DG_ITEMS = 8;
constexpr int DG_TILE = DG_THREADS * DG_ITEMS;

struct WaitsArgs {
  DevState* ds;
  const int32_t* dg_pid;
  const int64_t* dg_begin;
  const int64_t* dg_end;
  int64_t* dg_pre;
  uint64_t* dg_key;
  uint64_t* dg_status;
  const uint64_t* oev;
  int P, NOP, nob, wb1;
  int64_t W0, W1;
  int64_t* dev_idle;
  int64_t* op_idle;
};

// Inclusive sum over the wave.
__device__ __forceinline__ uint64_t wave_incl_sum_u64(uint64_t v) {
  const int l = lane_id();
  for (int d = 1; d < WAVE; d <<= 1) {
    const uint64_t o = shfl_up(v, d);
    if (l >= d) v += o;
  }
  return v;
}

// Exclusive prefix sums of the idle intervals' lengths: a tile of DG_TILE
// intervals per workgroup (consecutive per thread), a block scan, and the
// tiles chained by a decoupled look-back (tiles by workgroup index); and each
// interval's packed key (pid << wb1) | (begin - W0).
__global__ __launch_bounds__(DG_THREADS) void k_dg_scan(WaitsArgs a) {
  __shared__ uint64_t s_w[DG_THREADS / WAVE];
  __shared__ uint64_t s_base;
  const int64_t cnt = a.ds->nDgap;
  const int tile = blockIdx.x;
  const int64_t base = (int64_t)tile * DG_TILE;
  if (base >= cnt) return;  // tiles past the list: no later tile waits for them
  const int tid = threadIdx.x, lane = lane_id(), wv = tid / WAVE;
  const int64_t i0 = base + (int64_t)tid * DG_ITEMS;
  uint64_t len[DG_ITEMS];
  uint64_t sum = 0;
#pragma unroll
  for (int j = 0; j < DG_ITEMS; ++j) {
    const int64_t i = i0 + j;
    const int64_t ic = i < cnt ? i : cnt - 1;
    const uint64_t l = (uint64_t)(a.dg_end[ic] - a.dg_begin[ic]);
    len[j] = i < cnt ? l : 0;
    sum += len[j];
  }
  const uint64_t inc = wave_incl_sum_u64(sum);
  if (lane == WAVE - 1) s_w[wv] = inc;
  __syncthreads();
  if (tid == 0) {
    uint64_t run = 0;
    for (int w = 0; w < DG_THREADS / WAVE; ++w) {
      const uint64_t t = s_w[w];
      s_w[w] = run;
      run += t;
    }
    s_base = run;  // the tile's total, for the look-back
  }
  __syncthreads();
  if (wv == 0) {
    const uint64_t ex = wave_lookback<OpSum>(a.dg_status, tile, s_base, a.ds);
    if (lane == 0) s_base = ex;
  }
  __syncthreads();
  uint64_t pre = s_base + s_w[wv] + inc - sum;
#pragma unroll
  for (int j = 0; j < DG_ITEMS; ++j) {
    const int64_t i = i0 + j;
    if (i < cnt) {
      a.dg_pre[i] = (int64_t)pre;
      a.dg_key[i] = ((uint64_t)a.dg_pid[i] << a.wb1) | (uint64_t)(a.dg_begin[i] - a.W0);
    }
    pre += len[j];
  }
}

constexpr int WT_THREADS = 256;
constexpr int WT_SAMPLES = 1024;  // staged interval keys per workgroup (8 KB)
constexpr int WT_BLOCKS = 2048;
constexpr int WT_ACC = 64;  // names a workgroup sums in LDS (more go to the outputs directly)

// Idle time of process p before absolute time t (W0 <= t <= W1), up to a
// term that depends on p alone (the idle time of the processes before it).
// s_key holds the keys of intervals 0, S, 2S, ... (ns of them).
__device__ __forceinline__ int64_t idle_before(const WaitsArgs& a, const uint64_t* s_key, int ns, int64_t S,
                                               int64_t cnt, int32_t p, int64_t t) {
  const uint64_t target = ((uint64_t)p << a.wb1) | (uint64_t)(t - a.W0);
  int k0 = 0, k1 = ns;  // first staged key at or above the target
  while (k0 < k1) {
    const int mid = (k0 + k1) >> 1;
    if (s_key[mid] < target)
      k0 = mid + 1;
    else
      k1 = mid;
  }
  // the first interval at or after (p, t) lies in ((k0 - 1) S, k0 S]
  int64_t lo = k0 > 0 ? (int64_t)(k0 - 1) * S + 1 : 0;
  int64_t hi = min((int64_t)k0 * S, cnt);
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (a.dg_key[mid] < target)
      lo = mid + 1;
    else
      hi = mid;
  }
  if (lo == 0) return 0;
  const int64_t last = lo - 1;
  const uint64_t lk = a.dg_key[last];
  const int64_t begin = a.W0 + (int64_t)(lk & ((1ull << a.wb1) - 1));
  const int64_t end = a.dg_end[last];
  int64_t g = a.dg_pre[last] + (end - begin);
  if ((int32_t)(lk >> a.wb1) == p && end > t) g -= end - t;
  return g;
}

// One thread per op-name run (its two endpoints), a contiguous chunk of runs
// per workgroup; the runs' idle time summed per (pid, op name) by a segmented
// scan over the wave (a name's runs are consecutive, names ascend), the
// waves' sums of the chunk's first WT_ACC names in LDS, and one atomic per
// name and workgroup; then one thread per process for its total idle time.
__global__ __launch_bounds__(WT_THREADS) void k_waits(WaitsArgs a) {
  __shared__ uint64_t s_key[WT_SAMPLES];
  __shared__ uint64_t s_acc[WT_ACC];  // the chunk's first WT_ACC names' idle time
  const int64_t cnt = a.ds->nDgap;
  const int64_t runs = a.ds->nOev / 2;
  const int64_t nth = (int64_t)gridDim.x * WT_THREADS;
  const int64_t S = cnt > WT_SAMPLES ? cdiv(cnt, (int64_t)WT_SAMPLES) : 1;
  const int ns = (int)cdiv(cnt, S);
  for (int k = threadIdx.x; k < ns; k += WT_THREADS) s_key[k] = a.dg_key[(int64_t)k * S];
  __syncthreads();
  const uint64_t tmask = (1ull << a.wb1) - 1, omask = (1ull << a.nob) - 1;
  if (a.op_idle) {
    // a contiguous chunk of runs per workgroup (a few names each): a wave
    // sums each name's runs by a segmented scan, the workgroup sums the
    // waves' totals in LDS, and each name of the chunk takes one atomic
    const int64_t chunk = cdiv(cdiv(runs, (int64_t)gridDim.x), (int64_t)WT_THREADS) * WT_THREADS;
    const int64_t rb = (int64_t)blockIdx.x * chunk, re = min(runs, rb + chunk);
    if (threadIdx.x < WT_ACC) s_acc[threadIdx.x] = 0;
    const uint64_t k0 = rb < re ? a.oev[2 * rb] : 0;
    const int64_t seg0 = (int64_t)(int32_t)(k0 >> (a.wb1 + a.nob)) * a.NOP + (int64_t)(k0 & omask);
    __syncthreads();
    for (int64_t r0 = rb; r0 < re; r0 += WT_THREADS) {  // uniform over the workgroup
      const int64_t r = r0 + threadIdx.x;
      int64_t seg = -1;
      uint64_t v = 0;
      if (r < re) {
        const uint64_t ks = a.oev[2 * r], ke = a.oev[2 * r + 1];
        const int32_t p = (int32_t)(ks >> (a.wb1 + a.nob));
        const int64_t ts = a.W0 + (int64_t)((ks >> a.nob) & tmask);
        const int64_t tend = a.W0 + (int64_t)((ke >> a.nob) & tmask);
        seg = (int64_t)p * a.NOP + (int64_t)(ks & omask);
        v = (uint64_t)(idle_before(a, s_key, ns, S, cnt, p, tend) - idle_before(a, s_key, ns, S, cnt, p, ts));
      }
      // segmented inclusive sum (the runs of one name are consecutive)
      const int l = lane_id();
      for (int d = 1; d < WAVE; d <<= 1) {
        const uint64_t o = shfl_up(v, d);
        const int64_t os = shfl_up(seg, d);
        if (l >= d && os == seg) v += o;
      }
      const int64_t nxt = shfl_down(seg, 1);
      const bool last = seg >= 0 && (l == WAVE - 1 || nxt != seg);
      if (last && v) {
        const int64_t k = seg - seg0;  // (pid, op name) ascends along the runs
        if (k >= 0 && k < WT_ACC)
          atomicAdd((unsigned long long*)&s_acc[k], (unsigned long long)v);
        else
          atomicAdd((unsigned long long*)&a.op_idle[seg], (unsigned long long)v);
      }
    }
    __syncthreads();
    if (threadIdx.x < WT_ACC && s_acc[threadIdx.x])
      atomicAdd((unsigned long long*)&a.op_idle[seg0 + threadIdx.x], (unsigned long long)s_acc[threadIdx.x]);
  }
  if (a.dev_idle)
    for (int64_t p = (int64_t)blockIdx.x * WT_THREADS + threadIdx.x; p < a.P; p += nth)
      a.dev_idle[p] = idle_before(a, s_key, ns, S, cnt, (int32_t)p, a.W1) -
                      idle_before(a, s_key, ns, S, cnt, (int32_t)p, a.W0);
}

static WaitsArgs waits_args(Ctx& c) {
  WaitsArgs a;
  a.ds = c.ds;
  a.dg_pid = c.dg_pid;
  a.dg_begin = c.dg_begin;
  a.dg_end = c.dg_end;
  a.dg_pre = c.dg_pre;
  a.dg_key = c.dg_key;
  a.dg_status = c.dg_status;
  a.oev = c.oev;
  a.P = c.P;
  a.NOP = c.NOP;
  a.nob = c.nob;
  a.wb1 = c.wb1;
  a.W0 = c.W0;
  a.W1 = c.W1;
  a.dev_idle = c.o.dev_idle;
  a.op_idle = c.o.op_idle;
  return a;
}

void launch_dg_scan(Ctx& c) {
  const WaitsArgs a = waits_args(c);
  hipLaunchKernelGGL(k_dg_scan, dim3((unsigned)c.dg_tiles), dim3(DG_THREADS), 0, c.st, a);
}

void launch_waits(Ctx& c) {
  const WaitsArgs a = waits_args(c);
  // a grid of at most WT_BLOCKS workgroups: each stages the interval keys once
  const int64_t work = std::max<int64_t>(cdiv(c.oev_cap / 2, WT_THREADS), cdiv(c.P, WT_THREADS));
  hipLaunchKernelGGL(k_waits, dim3((unsigned)std::max<int64_t>(std::min<int64_t>(work, WT_BLOCKS), 1)),
                     dim3(WT_THREADS), 0, c.st, a);
}

}  // namespace hx
