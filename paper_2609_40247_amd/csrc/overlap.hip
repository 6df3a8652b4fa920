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

__global__ __launch_bounds__(SW_THREADS) void k_sweep(SweepArgs a) {
  __shared__ int s_tile;
  __shared__ unsigned long long s_pair[64 * 64];
  __shared__ unsigned long long s_cls[13];  // class_busy[3], class_overlap[9], any
  __shared__ uint64_t s_cmask[3];
  __shared__ uint64_t s_wx[SW_THREADS / WAVE];
  __shared__ uint64_t s_tx;
  __shared__ uint64_t s_pre[2];
  const int tid = threadIdx.x, lane = lane_id(), wv = tid / WAVE;
  const int64_t n = a.ds->nEv;
  const int par = (int)a.ds->sort_parity[3];
  const uint64_t* keys = a.k[par];
  const int tile = take_ticket(a.ds, TK_SWEEP, &s_tile);
  const int64_t base = (int64_t)tile * SW_TILE;
  if (base >= n) return;
  const int S = a.S;
  for (int i = tid; i < S * S; i += SW_THREADS) s_pair[i] = 0;
  if (tid < 13) s_cls[tid] = 0;
  if (tid < 3) {
    uint64_t m = 0;
    for (int s = 0; s < S; ++s)
      if ((a.cls ? a.cls[s] : 0) == tid) m |= 1ull << s;
    s_cmask[tid] = m;
  }
  const uint64_t tmask = (1ull << a.wb1) - 1;
  const uint64_t smask = (1ull << a.sb) - 1;
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
  const int pid0 = (int)(keys[base] >> (a.wb1 + a.sb));
#pragma unroll
  for (int j = 0; j < SW_ITEMS; ++j) {
    if (i0 + j >= n) break;
    m ^= 1ull << (key[j] & smask);
    const bool has_next = i0 + j + 1 < n;
    const uint64_t nk = j + 1 < SW_ITEMS ? key[j + 1] : nextkey;
    const int pid = (int)(key[j] >> (a.wb1 + a.sb));
    if (has_next && (int)(nk >> (a.wb1 + a.sb)) == pid) {
      const int64_t len = (int64_t)((nk >> a.sb) & tmask) - (int64_t)((key[j] >> a.sb) & tmask);
      add_interval(a, m, len, pid, pid0, s_cmask, s_pair, s_cls);
    }
  }
  __syncthreads();
  for (int i = tid; i < S * S; i += SW_THREADS)
    if (s_pair[i]) atomicAdd((unsigned long long*)&a.pair[(int64_t)pid0 * S * S + i], s_pair[i]);
  if (tid < 3 && s_cls[tid]) atomicAdd((unsigned long long*)&a.class_busy[pid0 * 3 + tid], s_cls[tid]);
  if (tid >= 3 && tid < 12 && s_cls[tid])
    atomicAdd((unsigned long long*)&a.class_overlap[pid0 * 9 + (tid - 3)], s_cls[tid]);
  if (tid == 12 && s_cls[12]) atomicAdd((unsigned long long*)&a.any_busy[pid0], s_cls[12]);
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
  hipLaunchKernelGGL(k_sweep, dim3((unsigned)std::max<int64_t>(c.sweep_tiles, 1)), dim3(SW_THREADS), 0, c.st, a);
}

}  // namespace hx
