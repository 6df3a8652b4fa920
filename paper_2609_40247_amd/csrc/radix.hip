// LSD radix sort of 64-bit keys (optionally with a 32-bit payload) for CDNA4.
//
// One launch per 8-bit digit.  Each workgroup ranks a tile of 4096 keys with
// wave64 ballots (a 64-lane match of the digit built from 8 ballots gives the
// rank among equal digits in one step), publishes its 256 per-digit counts
// through a decoupled look-back (one chain per digit, a lane per digit),
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

__global__ __launch_bounds__(256) void k_digit_hist(const uint64_t* __restrict__ keys, const int32_t* count,
                                                    int nd, uint32_t* __restrict__ hist) {
  __shared__ uint32_t h[8 * 256];
  for (int i = threadIdx.x; i < 8 * 256; i += 256) h[i] = 0;
  __syncthreads();
  const int64_t n = *count;
  const int lane = lane_id();
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const uint64_t k = keys[i];
    const uint64_t active = ballot(true);
    const int first = __ffsll((unsigned long long)active) - 1;
    for (int d = 0; d < nd; ++d) {
      const int dg = (int)((k >> (8 * d)) & 255);
      const int d0 = __shfl(dg, first, WAVE);
      if (ballot(dg != d0) == 0) {
        if (lane == first) atomicAdd(&h[d * 256 + d0], (uint32_t)popc(active));
      } else {
        atomicAdd(&h[d * 256 + dg], 1u);
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nd * 256; i += 256)
    if (h[i]) atomicAdd(&hist[i], h[i]);
}

template <bool VALS>
__global__ __launch_bounds__(RS_THREADS) void k_radix_pass(uint64_t* k0, uint64_t* k1, uint32_t* v0, uint32_t* v1,
                                                           const int32_t* count, DevState* ds, int id, int d,
                                                           uint32_t* status) {
  __shared__ uint64_t s_key[RS_TILE];
  __shared__ uint32_t s_val[VALS ? RS_TILE : 1];
  __shared__ uint32_t s_wh[RS_THREADS / WAVE][256];
  __shared__ uint32_t s_local[256];
  __shared__ uint32_t s_glob[256];
  __shared__ uint32_t s_scan[RS_THREADS / WAVE + 1];
  __shared__ int s_tile;

  const int tid = threadIdx.x, lane = lane_id(), wv = tid / WAVE;
  const uint32_t n = (uint32_t)*count;

  // Which buffer holds the input, and is this digit trivial?  A digit is
  // trivial iff one bin holds every key.  Every block decides identically.
  int parity = 0, trivial = 0;
  for (int dd = 0; dd <= d; ++dd) {
    const int full = ds->hist[id][dd][tid] == n;
    const int any = __syncthreads_or(full);
    if (dd < d)
      parity += any ? 0 : 1;
    else
      trivial = any;
  }
  if (trivial) {
    if (blockIdx.x == 0 && tid == 0) ds->sort_parity[id] = (uint32_t)(parity & 1);
    return;
  }
  if (blockIdx.x == 0 && tid == 0) ds->sort_parity[id] = (uint32_t)((parity + 1) & 1);
  const uint64_t* kin = (parity & 1) ? k1 : k0;
  uint64_t* kout = (parity & 1) ? k0 : k1;
  const uint32_t* vin = (parity & 1) ? v1 : v0;
  uint32_t* vout = (parity & 1) ? v0 : v1;

  const int tile = take_ticket(ds, TK_RADIX + 8 * id + d, &s_tile);
  const int64_t base = (int64_t)tile * RS_TILE;
  if (base >= (int64_t)n) return;

  for (int i = tid; i < (RS_THREADS / WAVE) * 256; i += RS_THREADS) (&s_wh[0][0])[i] = 0;
  __syncthreads();

  const int shift = 8 * d;
  uint64_t key[RS_ITEMS];
  uint32_t val[RS_ITEMS];
  uint32_t rank[RS_ITEMS];
  int dig[RS_ITEMS];
  const int64_t wbase = base + (int64_t)wv * (RS_ITEMS * WAVE);
#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) {
    const int64_t idx = wbase + j * WAVE + lane;
    const bool ok = idx < (int64_t)n;
    key[j] = ok ? kin[idx] : 0ull;
    if (VALS) val[j] = ok ? vin[idx] : 0u;
    dig[j] = ok ? (int)((key[j] >> shift) & 255) : 256;
  }
  // Wave-private ranking in input order: sub-tile of the wave, rounds in
  // order, lanes in order.
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

  // Thread t owns digit t: tile count, per-wave exclusive offsets.
  uint32_t cnt = 0;
#pragma unroll
  for (int w = 0; w < RS_THREADS / WAVE; ++w) {
    const uint32_t c = s_wh[w][tid];
    s_wh[w][tid] = cnt;
    cnt += c;
  }
  uint32_t* st = status + (int64_t)tile * 256;
  st_agent(&st[tid], (tile == 0 ? RS_FLAG_P : RS_FLAG_A) | cnt);
  const uint32_t local_excl = block_excl_sum<RS_THREADS>(cnt, s_scan, nullptr);
  s_local[tid] = local_excl;
  const uint32_t gexcl = block_excl_sum<RS_THREADS>(ds->hist[id][d][tid], s_scan, nullptr);

  uint32_t excl = 0;
  if (tile > 0) {
    int pred = tile - 1;
    uint32_t spins = 0;
    while (pred >= 0) {
      const uint32_t s = ld_agent(&status[(int64_t)pred * 256 + tid]);
      if ((s >> 30) == 0) {
        if (++spins > SPIN_LIMIT) {
          set_status(ds, DS_SPIN);
          break;
        }
        __builtin_amdgcn_s_sleep(1);
        continue;
      }
      excl += s & RS_VAL;
      if ((s >> 30) == 2) break;
      --pred;
    }
    st_agent(&st[tid], RS_FLAG_P | ((excl + cnt) & RS_VAL));
  }
  s_glob[tid] = gexcl + excl;
  __syncthreads();

#pragma unroll
  for (int j = 0; j < RS_ITEMS; ++j) {
    if (dig[j] < 256) {
      const uint32_t pos = s_local[dig[j]] + s_wh[wv][dig[j]] + rank[j];
      if (in_range(ds, pos, RS_TILE)) {
        s_key[pos] = key[j];
        if (VALS) s_val[pos] = val[j];
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
      if (VALS) vout[gpos] = s_val[i];
    }
  }
}

void launch_hist(Ctx& c, SortBufs& s, const int32_t* count) {
  if (s.nd == 0) return;
  const int64_t grid = std::min<int64_t>(std::max<int64_t>(cdiv(s.n_max, 8192), 1), 512);
  hipLaunchKernelGGL(k_digit_hist, dim3((unsigned)grid), dim3(256), 0, c.st, s.k[0], count, s.nd,
                     &c.ds->hist[s.id][0][0]);
}

void launch_sort(Ctx& c, SortBufs& s, const int32_t* count) {
  const int64_t grid = std::max<int64_t>(s.tiles_max, 1);
  for (int d = 0; d < s.nd; ++d) {
    uint32_t* status = s.status + (int64_t)d * s.tiles_max * 256;
    if (s.v[0])
      hipLaunchKernelGGL(k_radix_pass<true>, dim3((unsigned)grid), dim3(RS_THREADS), 0, c.st, s.k[0], s.k[1],
                         s.v[0], s.v[1], count, c.ds, s.id, d, status);
    else
      hipLaunchKernelGGL(k_radix_pass<false>, dim3((unsigned)grid), dim3(RS_THREADS), 0, c.st, s.k[0], s.k[1],
                         s.v[0], s.v[1], count, c.ds, s.id, d, status);
  }
}

}  // namespace hx
