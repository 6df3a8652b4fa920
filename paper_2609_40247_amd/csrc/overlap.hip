// Cross-stream overlap as interval coverage (Figure "Key performance
// observations", panel "Overlap and exposed work"; Section 6.1 separates
// communication hidden by computation from exposed time).
//
// Every coverage run of a stream contributes a start and an end event; with
// the events of a process sorted by time, the set of active streams between
// consecutive events is the XOR of all earlier events' stream bits.  Whole
// processes XOR to zero (every run closes), so a plain prefix XOR across the
// sorted list -- carried between tiles by a decoupled look-back on its two
// 32-bit halves -- gives each elementary interval's active mask.  Its length
// is added to every active pair, to the classes present and to "any".
#include "internal.hpp"

namespace hx {

constexpr int SW_THREADS = 256;
constexpr int SW_ITEMS = 16;
constexpr int SW_TILE = SW_THREADS * SW_ITEMS;

struct SweepArgs {
  const uint64_t* k[2];
  const uint8_t* cls;
  int P, S, sb, wb1;
  DevState* ds;
  int64_t* pair;
  int64_t* class_busy;
  int64_t* class_overlap;
  int64_t* any_busy;
  uint64_t* status;  // [2][tiles_max]
  int64_t tiles_max;
};

__device__ __forceinline__ void add_interval(const SweepArgs& a, uint64_t m, int64_t len, int pid, int pid0,
                                             const uint64_t* cmask, unsigned long long* s_pair,
                                             unsigned long long* s_cls) {
  if (len <= 0 || m == 0) return;
  const int S = a.S;
  const bool local = pid == pid0;
  int present[3];
  for (int c = 0; c < 3; ++c) present[c] = (m & cmask[c]) != 0;
  if (local) {
    atomicAdd(&s_cls[12], (unsigned long long)len);
    for (int c = 0; c < 3; ++c) {
      if (!present[c]) continue;
      atomicAdd(&s_cls[c], (unsigned long long)len);
      for (int c2 = 0; c2 < 3; ++c2)
        if (present[c2]) atomicAdd(&s_cls[3 + c * 3 + c2], (unsigned long long)len);
    }
  } else {
    atomicAdd((unsigned long long*)&a.any_busy[pid], (unsigned long long)len);
    for (int c = 0; c < 3; ++c) {
      if (!present[c]) continue;
      atomicAdd((unsigned long long*)&a.class_busy[pid * 3 + c], (unsigned long long)len);
      for (int c2 = 0; c2 < 3; ++c2)
        if (present[c2]) atomicAdd((unsigned long long*)&a.class_overlap[(pid * 3 + c) * 3 + c2], (unsigned long long)len);
    }
  }
  uint64_t mi = m;
  while (mi) {
    const int i = __ffsll((unsigned long long)mi) - 1;
    mi &= mi - 1;
    uint64_t mj = m;
    while (mj) {
      const int j = __ffsll((unsigned long long)mj) - 1;
      mj &= mj - 1;
      if (local)
        atomicAdd(&s_pair[i * S + j], (unsigned long long)len);
      else
        atomicAdd((unsigned long long*)&a.pair[((int64_t)pid * S + i) * S + j], (unsigned long long)len);
    }
  }
}

// Sums over one thread's intervals, kept in registers for up to SMAX streams
// (upper triangles of the symmetric pair and class matrices).
template <int SMAX>
struct SweepAcc {
  static constexpr int NP = SMAX * (SMAX + 1) / 2;
  uint64_t pair[NP];
  uint64_t co[6];  // class overlap upper triangle: 00 01 02 11 12 22
  uint64_t cb[3];
  uint64_t any;
  __device__ void zero() {
#pragma unroll
    for (int i = 0; i < NP; ++i) pair[i] = 0;
#pragma unroll
    for (int i = 0; i < 6; ++i) co[i] = 0;
    cb[0] = cb[1] = cb[2] = 0;
    any = 0;
  }
  __device__ void add(uint64_t m, uint64_t len, const uint64_t* cmask) {
    if (m == 0) return;
    any += len;
    const bool p0 = (m & cmask[0]) != 0, p1 = (m & cmask[1]) != 0, p2 = (m & cmask[2]) != 0;
    cb[0] += p0 ? len : 0;
    cb[1] += p1 ? len : 0;
    cb[2] += p2 ? len : 0;
    co[0] += p0 ? len : 0;
    co[1] += (p0 && p1) ? len : 0;
    co[2] += (p0 && p2) ? len : 0;
    co[3] += p1 ? len : 0;
    co[4] += (p1 && p2) ? len : 0;
    co[5] += p2 ? len : 0;
    int k = 0;
#pragma unroll
    for (int i = 0; i < SMAX; ++i) {
      const bool bi = (m >> i) & 1;
#pragma unroll
      for (int j = i; j < SMAX; ++j) {
        pair[k] += (bi && ((m >> j) & 1)) ? len : 0;
        ++k;
      }
    }
  }
};

template <int SMAX>
__global__ __launch_bounds__(SW_THREADS) void k_sweep(SweepArgs a) {
  __shared__ int s_tile;
  __shared__ unsigned long long s_pair[SMAX <= 8 ? SweepAcc<8>::NP : 64 * 64];
  __shared__ unsigned long long s_cls[13];  // class_busy[3], class_overlap[9], any
  __shared__ uint64_t s_cmask[3];
  __shared__ uint64_t s_wx[SW_THREADS / WAVE];
  __shared__ uint64_t s_tx;
  __shared__ uint64_t s_pre[2];
  const int tid = threadIdx.x, lane = lane_id(), wv = tid / WAVE;
  const int64_t n = a.ds->nEv;
  const int par = (int)a.ds->sort_parity[3];
  const uint64_t* keys = a.k[par];
  if ((int64_t)blockIdx.x * SW_TILE >= n) return;  // no tile: stay off the ticket counter
  const int tile = take_ticket(a.ds, TK_SWEEP, &s_tile);
  const int64_t base = (int64_t)tile * SW_TILE;
  const int S = a.S;
  constexpr int NPAIR = SMAX <= 8 ? SweepAcc<8>::NP : 64 * 64;
  for (int i = tid; i < NPAIR; i += SW_THREADS) s_pair[i] = 0;
  if (tid < 13) s_cls[tid] = 0;
  if (tid < 3) {
    uint64_t m = 0;
    for (int s = 0; s < S; ++s)
      if ((a.cls ? a.cls[s] : 0) == tid) m |= 1ull << s;
    s_cmask[tid] = m;
  }
  const uint64_t tmask = (1ull << a.wb1) - 1;
  const uint64_t smask = (1ull << a.sb) - 1;
  const int pshift = a.wb1 + a.sb;
  const int64_t i0 = base + (int64_t)tid * SW_ITEMS;
  uint64_t key[SW_ITEMS];
  uint64_t x = 0;
#pragma unroll
  for (int j = 0; j < SW_ITEMS; ++j) {
    key[j] = i0 + j < n ? keys[i0 + j] : 0;
    if (i0 + j < n) x ^= 1ull << (key[j] & smask);
  }
  // exclusive XOR over the block
  uint64_t inc = x;
  for (int d = 1; d < WAVE; d <<= 1) {
    const uint64_t o = shfl_up(inc, d);
    if (lane >= d) inc ^= o;
  }
  if (lane == WAVE - 1) s_wx[wv] = inc;
  __syncthreads();
  if (tid == 0) {
    uint64_t run = 0;
    for (int w = 0; w < SW_THREADS / WAVE; ++w) {
      const uint64_t t = s_wx[w];
      s_wx[w] = run;
      run ^= t;
    }
    s_tx = run;
  }
  __syncthreads();
  if (wv < 2) {
    const uint64_t half = wv == 0 ? (s_tx & 0xffffffffull) : (s_tx >> 32);
    const uint64_t ex = wave_lookback<OpXor32>(a.status + (int64_t)wv * a.tiles_max, tile, half, a.ds);
    if (lane == 0) s_pre[wv] = ex;
  }
  __syncthreads();
  uint64_t m = (s_pre[0] | (s_pre[1] << 32)) ^ s_wx[wv] ^ (inc ^ x);
  const uint64_t nextkey = i0 + SW_ITEMS < n ? keys[i0 + SW_ITEMS] : 0;
  const int pid0 = (int)(keys[base] >> pshift);
  uint64_t cm[3] = {s_cmask[0], s_cmask[1], s_cmask[2]};
  SweepAcc<SMAX <= 8 ? SMAX : 1> acc;
  acc.zero();
#pragma unroll
  for (int j = 0; j < SW_ITEMS; ++j) {
    if (i0 + j >= n) break;
    m ^= 1ull << (key[j] & smask);
    const bool has_next = i0 + j + 1 < n;
    const uint64_t nk = j + 1 < SW_ITEMS ? key[j + 1] : nextkey;
    const int pid = (int)(key[j] >> pshift);
    if (has_next && (int)(nk >> pshift) == pid) {
      const int64_t len = (int64_t)((nk >> a.sb) & tmask) - (int64_t)((key[j] >> a.sb) & tmask);
      if (SMAX <= 8 && pid == pid0)
        acc.add(m, (uint64_t)len, cm);
      else
        add_interval(a, m, len, pid, pid0, cm, s_pair, s_cls);
    }
  }
  if (SMAX <= 8) {
    // wave sums, then one LDS add per wave
    constexpr int NP = SweepAcc<SMAX <= 8 ? SMAX : 1>::NP;
#pragma unroll
    for (int k = 0; k < NP; ++k) {
      const uint64_t w = wave_sum_u64(acc.pair[k]);
      if (lane == 0 && w) atomicAdd(&s_pair[k], (unsigned long long)w);
    }
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      const uint64_t w = wave_sum_u64(acc.cb[c]);
      if (lane == 0 && w) atomicAdd(&s_cls[c], (unsigned long long)w);
    }
    const int co_idx[6] = {0, 1, 2, 4, 5, 8};
#pragma unroll
    for (int c = 0; c < 6; ++c) {
      const uint64_t w = wave_sum_u64(acc.co[c]);
      if (lane == 0 && w) atomicAdd(&s_cls[3 + co_idx[c]], (unsigned long long)w);
    }
    const uint64_t w = wave_sum_u64(acc.any);
    if (lane == 0 && w) atomicAdd(&s_cls[12], (unsigned long long)w);
  }
  __syncthreads();
  if (SMAX <= 8) {
    // upper triangles back to full symmetric matrices
    int k = 0;
    for (int i = 0; i < SMAX && i < S; ++i)
      for (int j = i; j < SMAX; ++j, ++k) {
        if (j >= S || tid != 0) continue;
        const unsigned long long v = s_pair[k];
        if (!v) continue;
        atomicAdd((unsigned long long*)&a.pair[((int64_t)pid0 * S + i) * S + j], v);
        if (j != i) atomicAdd((unsigned long long*)&a.pair[((int64_t)pid0 * S + j) * S + i], v);
      }
    if (tid < 3 && s_cls[tid]) atomicAdd((unsigned long long*)&a.class_busy[pid0 * 3 + tid], s_cls[tid]);
    if (tid >= 3 && tid < 12) {
      const int c1 = (tid - 3) / 3, c2 = (tid - 3) % 3;
      const unsigned long long v = c1 <= c2 ? s_cls[3 + c1 * 3 + c2] : s_cls[3 + c2 * 3 + c1];
      if (v) atomicAdd((unsigned long long*)&a.class_overlap[pid0 * 9 + (tid - 3)], v);
    }
    if (tid == 12 && s_cls[12]) atomicAdd((unsigned long long*)&a.any_busy[pid0], s_cls[12]);
  } else {
    for (int i = tid; i < S * S; i += SW_THREADS)
      if (s_pair[i]) atomicAdd((unsigned long long*)&a.pair[(int64_t)pid0 * S * S + i], s_pair[i]);
    if (tid < 3 && s_cls[tid]) atomicAdd((unsigned long long*)&a.class_busy[pid0 * 3 + tid], s_cls[tid]);
    if (tid >= 3 && tid < 12 && s_cls[tid])
      atomicAdd((unsigned long long*)&a.class_overlap[pid0 * 9 + (tid - 3)], s_cls[tid]);
    if (tid == 12 && s_cls[12]) atomicAdd((unsigned long long*)&a.any_busy[pid0], s_cls[12]);
  }
}

void launch_overlap(Ctx& c) {
  SweepArgs a;
  a.k[0] = c.sE.k[0];
  a.k[1] = c.sE.k[1];
  a.cls = c.p.stream_class;
  a.P = c.P;
  a.S = c.S;
  a.sb = c.sb;
  a.wb1 = c.wb1;
  a.ds = c.ds;
  a.pair = c.o.pair_overlap;
  a.class_busy = c.o.class_busy;
  a.class_overlap = c.o.class_overlap;
  a.any_busy = c.o.any_busy;
  a.status = c.sweep_status;
  a.tiles_max = c.sweep_tiles;
  launch_hist(c, c.sE, &c.ds->nEv);
  launch_sort(c, c.sE, &c.ds->nEv);
  const dim3 grid((unsigned)std::max<int64_t>(c.sweep_tiles, 1));
  if (c.S <= 4)
    hipLaunchKernelGGL(k_sweep<4>, grid, dim3(SW_THREADS), 0, c.st, a);
  else if (c.S <= 8)
    hipLaunchKernelGGL(k_sweep<8>, grid, dim3(SW_THREADS), 0, c.st, a);
  else
    hipLaunchKernelGGL(k_sweep<64>, grid, dim3(SW_THREADS), 0, c.st, a);
}

}  // namespace hx
