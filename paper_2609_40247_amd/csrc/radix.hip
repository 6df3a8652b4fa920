// LSD radix sort of 64-bit keys (optionally with a 32-bit payload) for CDNA4.
//
// One launch per 8-bit digit, shared by the independent sorts of a call.  Each workgroup ranks a tile of 8192 keys with
// wave64 ballots (a 64-lane match of the digit built from 8 ballots gives the
// rank among equal digits in one step), publishes its 256 per-digit counts
// through a decoupled look-back (one chain per digit, four lanes per digit),
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
  int nd;
  int id;
};
struct HistJobs {
  HistJob j[N_SORTS];
  uint32_t* part;  // [N_SORTS][HIST_MAX_BLOCKS][8 * 256] per-workgroup counts
};

// Digit histograms of several sort inputs in one launch (blockIdx.y picks
// the sort).  Each workgroup counts a contiguous share of the keys in LDS
// and stores its table; the plan kernel that follows sums the tables.  No
// global atomics and no fences: counters shared by many workgroups serialise
// on their cache line, and a device-scope fence writes back the whole L2.
constexpr int HIST_THREADS = 1024;

// Adds one key's ND digits to the LDS table.  Digits 0 and 1 of these keys
// (nanoseconds, correlation ids) differ across a wave, so every lane adds;
// for higher digits, when the whole wave agrees, one lane adds the count.
template <int ND>
__device__ __forceinline__ void hist_add(uint32_t* h, uint64_t k) {
  const uint32_t lo = (uint32_t)k, hi = (uint32_t)(k >> 32);
  const uint64_t active = ballot(true);
  const bool leader = lane_id() == __ffsll((unsigned long long)active) - 1;
#pragma unroll
  for (int d = 0; d < ND; ++d) {
    const uint32_t dg = ((d < 4 ? lo : hi) >> (8 * (d & 3))) & 255u;
    if (d < 2) {
      atomicAdd(&h[d * 256 + dg], 1u);
    } else {
      const uint32_t d0 = __builtin_amdgcn_readfirstlane(dg);
      if (ballot(dg != d0) == 0) {
        if (leader) atomicAdd(&h[d * 256 + d0], (uint32_t)popc(active));
      } else {
        atomicAdd(&h[d * 256 + dg], 1u);
      }
    }
  }
}

template <int ND>
__device__ void hist_range(uint32_t* h, const uint64_t* __restrict__ keys, int64_t lo, int64_t hi) {
  constexpr int U = 8;  // loads in flight per thread
  int64_t i = lo + threadIdx.x;
  for (; i + (U - 1) * HIST_THREADS < hi; i += U * HIST_THREADS) {
    uint64_t k[U];
#pragma unroll
    for (int u = 0; u < U; ++u) k[u] = keys[i + u * HIST_THREADS];
#pragma unroll
    for (int u = 0; u < U; ++u) hist_add<ND>(h, k[u]);
  }
  for (; i < hi; i += HIST_THREADS) hist_add<ND>(h, keys[i]);
}

__global__ __launch_bounds__(HIST_THREADS) void k_digit_hist(HistJobs jobs, const DevState* ds) {
  const HistJob jb = jobs.j[blockIdx.y];
  if (jb.id == 1 && ds->join_direct) return;  // the correlation table replaces the join sort
  const int nd = jb.nd, nbins = nd * 256;
  __shared__ uint32_t h[8 * 256];
  const int64_t n = *jb.count;
  const int nblk = hist_blocks(n);
  const int blk = blockIdx.x;
  if (blk >= nblk) return;
  for (int i = threadIdx.x; i < 8 * 256; i += HIST_THREADS) h[i] = 0;
  __syncthreads();
  const int64_t per = cdiv(n, nblk);
  const int64_t lo = min<int64_t>(n, (int64_t)blk * per), hi = min<int64_t>(n, lo + per);
  switch (nd) {
    case 1: hist_range<1>(h, jb.keys, lo, hi); break;
    case 2: hist_range<2>(h, jb.keys, lo, hi); break;
    case 3: hist_range<3>(h, jb.keys, lo, hi); break;
    case 4: hist_range<4>(h, jb.keys, lo, hi); break;
    case 5: hist_range<5>(h, jb.keys, lo, hi); break;
    case 6: hist_range<6>(h, jb.keys, lo, hi); break;
    case 7: hist_range<7>(h, jb.keys, lo, hi); break;
    default: hist_range<8>(h, jb.keys, lo, hi); break;
  }
  __syncthreads();
  uint32_t* part = jobs.part + ((int64_t)jb.id * HIST_MAX_BLOCKS + blk) * 8 * 256;
  for (int j = threadIdx.x; j < nbins; j += HIST_THREADS) part[j] = h[j];
}

// Plan of one digit of one sort (blockIdx.x = digit, blockIdx.y = sort):
// the digit's counts summed over the workgroup tables, its trivial flag
// (one bin holds every key) and each bin's exclusive offset.
__global__ __launch_bounds__(256) void k_hist_plan(HistJobs jobs, DevState* ds) {
  __shared__ uint32_t s_scan[256 / WAVE + 1];
  const HistJob jb = jobs.j[blockIdx.y];
  const int d = blockIdx.x;
  if (d >= jb.nd || (jb.id == 1 && ds->join_direct)) return;
  const int64_t n = *jb.count;
  const int nblk = hist_blocks(n);
  const uint32_t* src = jobs.part + (int64_t)jb.id * HIST_MAX_BLOCKS * 8 * 256 + d * 256 + threadIdx.x;
  uint32_t c = 0;
  for (int b0 = 0; b0 < nblk; b0 += 16) {
    uint32_t v[16];
#pragma unroll
    for (int b = 0; b < 16; ++b) v[b] = b0 + b < nblk ? src[(int64_t)(b0 + b) * 8 * 256] : 0u;
#pragma unroll
    for (int b = 0; b < 16; ++b) c += v[b];
  }
  if (__syncthreads_or(c == (uint32_t)n) && threadIdx.x == 0) atomicOr(&ds->sort_trivial[jb.id], 1u << d);
  const uint32_t ex = block_excl_sum<256>(c, s_scan, nullptr);
  ds->hist[jb.id][d][threadIdx.x] = ex;
}

struct SortJob {
  uint64_t* k[2];
  uint32_t* v[2];
  const int32_t* count;
  uint32_t* status;  // [nd][tiles_max * 256]
  int64_t tiles_max;
  int nd, id;
};
struct SortJobs {
  SortJob j[N_SORTS];
};

// One digit pass of up to N_SORTS independent sorts (blockIdx.y picks one).
__global__ __launch_bounds__(RS_THREADS) void k_radix_pass(SortJobs jobs, DevState* ds, int d) {
  constexpr int NW = RS_THREADS / WAVE;     // waves per workgroup
  constexpr int NSL = RS_THREADS / 256;     // look-back slices per digit
  __shared__ uint64_t s_key[RS_TILE];
  __shared__ uint32_t s_val[RS_TILE];
  __shared__ uint32_t s_wh[NW][256];
  __shared__ uint32_t s_local[256];
  __shared__ uint32_t s_glob[256];
  __shared__ uint32_t s_scan[NW + 1];
  __shared__ uint32_t s_lb_sum[NSL][256];
  __shared__ uint8_t s_lb_state[NSL][256];
  __shared__ int s_tile;

  const SortJob& jb = jobs.j[blockIdx.y];
  if (d >= jb.nd) return;
  const int id = jb.id;
  const int tid = threadIdx.x, lane = lane_id(), wv = tid / WAVE;
  const int dgt = tid & 255, slice = tid >> 8;
  // The plan (trivial digits, offsets) was made by the histogram kernel.  A
  // digit is trivial iff one bin holds every key; the input buffer's parity
  // is the number of non-trivial digits below this one.  Workgroups with no
  // tile to sort leave before the ticket: the ticket counter is one address,
  // and every request to it is served in turn.  The first cdiv(n, tile)
  // workgroups stay, so they draw exactly the tickets of the real tiles.
  const uint32_t n = (uint32_t)*jb.count;
  const uint32_t triv = ds->sort_trivial[id];
  const uint32_t gexcl = ds->hist[id][d][dgt];
  // which buffer holds the result: parity of the digits that move data
  if (d == 0 && blockIdx.x == 0 && tid == 0)
    ds->sort_parity[id] = (uint32_t)(popc(~triv & ((jb.nd >= 32 ? 0u : 1u << jb.nd) - 1u)) & 1);
  if (((triv >> d) & 1) || (int64_t)blockIdx.x * RS_TILE >= (int64_t)n) return;
  if (tid == 0) s_tile = (int)atomicAdd(&ds->ticket[TK_RADIX + 8 * id + d], 1u);
  for (int i = tid; i < NW * 256; i += RS_THREADS) (&s_wh[0][0])[i] = 0;
  __syncthreads();
  const int parity = popc(~triv & ((1u << d) - 1u)) & 1;
  const uint64_t* kin = jb.k[parity];
  uint64_t* kout = jb.k[parity ^ 1];
  const uint32_t* vin = jb.v[parity];
  uint32_t* vout = jb.v[parity ^ 1];
  uint32_t* status = jb.status + (int64_t)d * jb.tiles_max * 256;
  const int tile = s_tile;
  const int64_t base = (int64_t)tile * RS_TILE;

  const int shift = 8 * d;
  uint64_t key[RS_ITEMS];
  uint32_t val[RS_ITEMS];
  uint32_t rank[RS_ITEMS];
  int dig[RS_ITEMS];
  // each wave owns RS_ITEMS * 64 consecutive keys, item j of lane l at j*64+l
  const int64_t wbase = base + (int64_t)wv * (RS_ITEMS * WAVE);
#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) {
    const int64_t idx = wbase + j * WAVE + lane;
    const bool ok = idx < (int64_t)n;
    key[j] = ok ? kin[idx] : 0ull;
    val[j] = ok ? vin[idx] : 0u;
  }
#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) {
    const int64_t idx = wbase + j * WAVE + lane;
    dig[j] = idx < (int64_t)n ? (int)((key[j] >> shift) & 255) : 256;
  }
  // Wave-private ranking in input order: items in order, lanes in order.
  const uint64_t lt = lanemask_lt();
#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) {
    const bool ok = dig[j] < 256;
    uint64_t peers = ballot(ok);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (dig[j] >> b) & 1;
      const uint64_t bb = ballot(bit);
      peers &= bit ? bb : ~bb;
    }
    const uint32_t before = ok ? s_wh[wv][dig[j]] : 0u;
    rank[j] = before + (uint32_t)popc(peers & lt);
    __builtin_amdgcn_wave_barrier();
    if (ok && (peers & lt) == 0) s_wh[wv][dig[j]] = before + (uint32_t)popc(peers);
    __builtin_amdgcn_wave_barrier();
  }
  __syncthreads();

  // Threads 0..255 own one digit each: tile count, per-wave exclusive offsets.
  uint32_t cnt = 0;
  if (tid < 256) {
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const uint32_t c = s_wh[w][tid];
      s_wh[w][tid] = cnt;
      cnt += c;
    }
  }
  uint32_t* st = status + (int64_t)tile * 256;
  if (tid < 256) st_agent(&st[tid], (tile == 0 ? RS_FLAG_P : RS_FLAG_A) | cnt);
  const uint32_t local_excl = block_excl_sum<RS_THREADS>(cnt, s_scan, nullptr);
  if (tid < 256) s_local[tid] = local_excl;

  // Look-back: every digit has NSL threads, each polling LB_WIN predecessors
  // per round trip (independent loads), so one round covers NSL * LB_WIN
  // tiles.  A round is used up to the nearest tile that published its
  // inclusive prefix; a round with an unpublished tile before that is
  // polled again.  The loop condition is uniform over the workgroup.
  uint32_t excl = 0;
  if (tile > 0) {
    constexpr int LB_WIN = 16;
    int pred = tile - 1;  // newest predecessor not yet counted
    bool done = false;
    uint32_t spins = 0;
    for (;;) {
      const int top = pred - slice * LB_WIN;
      uint32_t sum = 0;
      int state = 1;  // 0: not ready, 1: all aggregates, 2: reached a prefix
      if (!done) {
        uint32_t sv[LB_WIN];
#pragma unroll
        for (int i = 0; i < LB_WIN; ++i)
          sv[i] = top - i >= 0 ? ld_agent(&status[(int64_t)(top - i) * 256 + dgt]) : RS_FLAG_P;
#pragma unroll
        for (int i = 0; i < LB_WIN; ++i) {
          const uint32_t f = sv[i] >> 30;
          if (state == 1) {
            if (f == 0) {
              state = 0;
            } else {
              sum += sv[i] & RS_VAL;
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
          if (++spins > SPIN_LIMIT) {
            set_status(ds, DS_SPIN);
            done = true;
          } else {
            again = true;
          }
        } else {
          excl += add;
          pred -= NSL * LB_WIN;
          if (res == 2 || pred < 0) done = true;
        }
      }
      if (!__syncthreads_or(!done)) break;
      if (again) __builtin_amdgcn_s_sleep(1);
    }
    if (tid < 256) st_agent(&st[tid], RS_FLAG_P | ((excl + cnt) & RS_VAL));
  }
  if (tid < 256) s_glob[tid] = gexcl + excl;
  __syncthreads();

#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) {
    if (dig[j] < 256) {
      const uint32_t pos = s_local[dig[j]] + s_wh[wv][dig[j]] + rank[j];
      if (in_range(ds, pos, RS_TILE)) {
        s_key[pos] = key[j];
        s_val[pos] = val[j];
      }
    }
  }
  __syncthreads();

  const uint32_t tile_n = (uint32_t)min((int64_t)RS_TILE, (int64_t)n - base);
  for (uint32_t i = tid; i < tile_n; i += RS_THREADS) {
    const uint64_t kk = s_key[i];
    const int dg = (int)((kk >> shift) & 255);
    const uint32_t gpos = s_glob[dg] + (i - s_local[dg]);
    if (in_range(ds, gpos, n)) {
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
    jobs.j[m++] = HistJob{s[i]->k[0], count[i], s[i]->nd, s[i]->id};
    n_max = std::max<int64_t>(n_max, s[i]->n_max);
    nd = std::max(nd, s[i]->nd);
  }
  if (m == 0) return;
  const int64_t grid = std::min<int64_t>(cdiv(n_max, HIST_CHUNK), HIST_MAX_BLOCKS);
  hipLaunchKernelGGL(k_digit_hist, dim3((unsigned)grid, (unsigned)m), dim3(HIST_THREADS), 0, c.st, jobs, c.ds);
  hipLaunchKernelGGL(k_hist_plan, dim3((unsigned)nd, (unsigned)m), dim3(256), 0, c.st, jobs, c.ds);
}

void launch_sort_multi(Ctx& c, SortBufs* const* s, const int32_t* const* count, int k) {
  SortJobs jobs{};
  int64_t grid = 1;
  int nd = 0;
  for (int i = 0; i < k; ++i) {
    jobs.j[i] = SortJob{{s[i]->k[0], s[i]->k[1]}, {s[i]->v[0], s[i]->v[1]}, count[i], s[i]->status,
                        s[i]->tiles_max, s[i]->nd, s[i]->id};
    grid = std::max<int64_t>(grid, s[i]->tiles_max);
    nd = std::max(nd, s[i]->nd);
  }
  for (int d = 0; d < nd; ++d)
    hipLaunchKernelGGL(k_radix_pass, dim3((unsigned)grid, (unsigned)k), dim3(RS_THREADS), 0, c.st, jobs, c.ds, d);
}

}  // namespace hx
