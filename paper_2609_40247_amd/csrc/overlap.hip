// Cross-stream overlap as interval coverage (Figure "Key performance
// observations", panel "Overlap and exposed work"; Section 6.1 separates
// communication hidden by computation from exposed time).
//
// Every coverage run of a stream contributes a start and an end event.  The
// timeline stage emits them grouped by (pid, stream) with strictly rising
// times inside a group, so starts and ends alternate.  Ordering a process's
// events by (time, stream) -- the order of the keys -- the elementary
// interval after event e ends at the first later event of any stream, and a
// stream is active in it iff an odd number of its events precede it.  Both
// follow from e's co-rank in each sibling group (how many of its events
// order before e), so the events are never merged into one sorted list.
// With up to 8 streams (and up to 256 groups) every tile lies inside one
// group; for each sibling it finds the stretch of that sibling's events its
// own events fall among (two wave searches), stages it in LDS and takes each
// co-rank by a binary search there.  More streams or groups: every event
// searches its sibling groups in memory.  The interval's length is added to
// every active pair, to the classes present and to "any".
#include "internal.hpp"

namespace hx {

constexpr int SW_THREADS = 512;
constexpr int SW_ITEMS = 8;
constexpr int SW_TILE = SW_THREADS * SW_ITEMS;
constexpr int SW_SMAX = 8;     // most streams summed per active-stream mask
constexpr int SB_CAP = 8192;   // sibling events staged in LDS per tile (64 KB)
constexpr int SW_GROUPS = 256; // most (pid, stream) groups for group-aligned tiles
static_assert(SW_SMAX <= 8 && SW_ITEMS <= 8, "a thread's active-stream masks are packed 8 bits each into 64");

struct SweepArgs {
  const uint64_t* ev;  // (pid << (wb1 + sb)) | (t << sb) | stream, grouped by (pid, stream)
  int32_t* seg_off;    // [P * S + 1] first event of each group
  const uint8_t* cls;
  int P, S, sb, wb1;
  DevState* ds;
  int64_t* pair;
  int64_t* class_busy;
  int64_t* class_overlap;
  int64_t* any_busy;
};

__device__ __attribute__((always_inline)) inline void add_interval(const SweepArgs& a, uint64_t m, int64_t len, int pid, int pid0,
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
    if (a.any_busy) atomicAdd((unsigned long long*)&a.any_busy[pid], (unsigned long long)len);
    for (int c = 0; c < 3; ++c) {
      if (!present[c]) continue;
      if (a.class_busy) atomicAdd((unsigned long long*)&a.class_busy[pid * 3 + c], (unsigned long long)len);
      if (a.class_overlap)
        for (int c2 = 0; c2 < 3; ++c2)
          if (present[c2])
            atomicAdd((unsigned long long*)&a.class_overlap[(pid * 3 + c) * 3 + c2], (unsigned long long)len);
    }
  }
  // separate loops for LDS and HBM, so that neither becomes a flat atomic
  if (local) {
    for (uint64_t mi = m; mi; mi &= mi - 1) {
      const int i = __ffsll((unsigned long long)mi) - 1;
      for (uint64_t mj = m; mj; mj &= mj - 1)
        atomicAdd(&s_pair[i * S + __ffsll((unsigned long long)mj) - 1], (unsigned long long)len);
    }
  } else if (a.pair) {
    for (uint64_t mi = m; mi; mi &= mi - 1) {
      const int i = __ffsll((unsigned long long)mi) - 1;
      for (uint64_t mj = m; mj; mj &= mj - 1)
        atomicAdd((unsigned long long*)&a.pair[((int64_t)pid * S + i) * S + __ffsll((unsigned long long)mj) - 1],
                  (unsigned long long)len);
    }
  }
}

// First event of every (pid, stream) group; entry P * S is the event count.
// One wave per group boundary searches the events 64-ary: each round every
// lane tests one point of the remaining stretch and a ballot keeps the part
// where the boundary lies (four rounds for a million events).
__global__ __launch_bounds__(256) void k_segoff(SweepArgs a) {
  const int32_t n = a.ds->nEv;
  const int nseg = a.P * a.S;
  const int pshift = a.wb1 + a.sb;
  const uint64_t smask = (1ull << a.sb) - 1;
  const int lane = lane_id();
  const int waves = gridDim.x * (256 / WAVE);
  for (int g = blockIdx.x * (256 / WAVE) + threadIdx.x / WAVE; g <= nseg; g += waves) {
    int32_t lo = 0, hi = n;  // the first event of group >= g lies in [lo, hi]
    while (lo < hi) {
      const int32_t step = (hi - lo + WAVE - 1) / WAVE;
      const int32_t x = lo + lane * step;
      bool below = false;
      if (x < hi) {
        const uint64_t k = a.ev[x];
        below = (int)(k >> pshift) * a.S + (int)(k & smask) < g;
      }
      const int c = popc(ballot(below));  // lanes 0..c-1 test points below the boundary
      const int32_t nlo = c > 0 ? lo + (c - 1) * step + 1 : lo;
      const int32_t xc = lo + c * step;
      hi = xc < hi ? xc : hi;
      lo = nlo;
    }
    if (lane == 0) a.seg_off[g] = lo;
  }
}

// First index in [lo, hi) whose key is not below `key` (hi if none), by a
// 64-ary search: every lane probes one point per round and a ballot keeps
// the stretch where the answer lies.  Called by a whole wave; every lane
// gets the answer.
__device__ int32_t wave_lower_bound(const uint64_t* __restrict__ ev, int32_t lo, int32_t hi, uint64_t key) {
  const int lane = lane_id();
  while (lo < hi) {  // answer in [lo, hi]
    const int32_t step = (hi - lo + WAVE - 1) / WAVE;
    const int32_t x = lo + lane * step;
    const bool below = x < hi && ev[x] < key;
    const int c = popc(ballot(below));  // lanes 0..c-1 probed below the key
    const int32_t nlo = c > 0 ? lo + (c - 1) * step + 1 : lo;
    const int32_t xc = lo + c * step;
    hi = xc < hi ? xc : hi;
    lo = nlo;
  }
  return lo;
}

// Copy the keys src[x * stride], x < cnt (cnt <= SB_CAP), into LDS, SW_STAGE
// loads in flight per thread (indices clamped to the last one, so every load
// is in bounds).
constexpr int SW_STAGE = 8;
__device__ __forceinline__ void stage_keys(const uint64_t* __restrict__ src, int32_t cnt, uint64_t* dst,
                                           int32_t stride = 1) {
  for (int32_t xb = 0; xb < cnt; xb += SW_STAGE * SW_THREADS) {
    uint64_t v[SW_STAGE];
#pragma unroll
    for (int u = 0; u < SW_STAGE; ++u) {
      const int32_t x = xb + u * SW_THREADS + (int32_t)threadIdx.x;
      v[u] = src[(int64_t)(x < cnt ? x : cnt - 1) * stride];
    }
#pragma unroll
    for (int u = 0; u < SW_STAGE; ++u) {
      const int32_t x = xb + u * SW_THREADS + (int32_t)threadIdx.x;
      if (x < cnt) dst[x] = v[u];
    }
  }
}

// Active-stream mask and next event time after event i (key `key`) from
// binary searches of its process's sibling groups in memory; the own stream
// is active after a start (even index in its group).
__device__ __forceinline__ void item_global(const SweepArgs& a, int64_t i, uint64_t key, uint64_t tmask,
                                            uint64_t smask, int pshift, uint64_t* m_out, uint64_t* tn_out) {
  const int S = a.S;
  const int pid = (int)(key >> pshift);
  const int st = (int)(key & smask);
  const int32_t* off = a.seg_off + (int64_t)pid * S;
  uint64_t m = 0, tn = ~0ull;
#pragma unroll 1
  for (int s = 0; s < S; ++s) {
    if (s == st) continue;
    const int32_t Lq = off[s], Rq = off[s + 1];
    int32_t lo = Lq, len = Rq - Lq;
    uint64_t nx = ~0ull;
    while (len > 0) {
      const int32_t half = len >> 1;
      const uint64_t v = a.ev[lo + half];
      if (v < key) {
        lo += half + 1;
        len -= half + 1;
      } else {
        nx = v;
        len = half;
      }
    }
    if ((lo - Lq) & 1) m |= 1ull << s;
    if (lo < Rq) {
      const uint64_t t2 = (nx >> a.sb) & tmask;
      tn = t2 < tn ? t2 : tn;
    }
  }
  const int32_t own_L = off[st], own_R = off[st + 1];
  if (((i - own_L) & 1) == 0) m |= 1ull << st;
  if (i + 1 < own_R) {
    const uint64_t t2 = (a.ev[i + 1] >> a.sb) & tmask;
    tn = t2 < tn ? t2 : tn;
  }
  *m_out = m;
  *tn_out = tn;
}

// Per-mask interval sums T[m] of one process (s_mlen, 256 entries, zero
// beyond 2^S) expanded into its pair matrix, class coverage and "any".  In
// S steps of 256 threads, s_mlen becomes the superset sums F[m] (the time at
// least the streams of m are active) and s_sub the subset sums G[m] (the
// time only streams of m are): pair (i, j) is F[{i, j}]; with the total
// T = G[all], a class's coverage is T - G[all but the class], and two
// classes' overlap T - G[not c1] - G[not c2] + G[neither].
__device__ __forceinline__ void flush_masks(const SweepArgs& a, int pid, unsigned long long* s_mlen,
                                            unsigned long long* s_sub, unsigned long long* s_cls, const uint64_t* cm) {
  const int tid = threadIdx.x, S = a.S;
  static_assert(SW_THREADS >= 256, "one thread per mask");
  if (tid < 256) s_sub[tid] = s_mlen[tid];
  for (int bit = 0; bit < S; ++bit) {
    __syncthreads();
    if (tid < 256) {
      const int m = 1 << bit;
      if (!(tid & m)) s_mlen[tid] += s_mlen[tid | m];  // entries with the bit are not written this step
      else s_sub[tid] += s_sub[tid ^ m];               // nor are those without it
    }
  }
  __syncthreads();
  const uint64_t all = (1ull << S) - 1;
  if (tid < S * S) {
    const int i = tid / S, jj = tid % S;
    const unsigned long long v = s_mlen[(1 << i) | (1 << jj)];
    if (v && a.pair) atomicAdd((unsigned long long*)&a.pair[((int64_t)pid * S + i) * S + jj], v);
  } else if (tid >= 64 && tid < 64 + 13) {
    const int e = tid - 64;  // 0..2 class busy, 3..11 class pairs, 12 any
    const unsigned long long T = s_sub[all];
    unsigned long long v;
    if (e < 3) {
      v = T - s_sub[all & ~cm[e]];
    } else if (e < 12) {
      const uint64_t c1 = cm[(e - 3) / 3], c2 = cm[(e - 3) % 3];
      v = T - s_sub[all & ~c1] - s_sub[all & ~c2] + s_sub[all & ~(c1 | c2)];
    } else {
      v = T;
    }
    s_cls[e] = v;
  }
  __syncthreads();
  if (a.class_busy && tid < 3 && s_cls[tid])
    atomicAdd((unsigned long long*)&a.class_busy[pid * 3 + tid], s_cls[tid]);
  if (a.class_overlap && tid >= 3 && tid < 12 && s_cls[tid])
    atomicAdd((unsigned long long*)&a.class_overlap[pid * 9 + (tid - 3)], s_cls[tid]);
  if (a.any_busy && tid == 12 && s_cls[12]) atomicAdd((unsigned long long*)&a.any_busy[pid], s_cls[12]);
}

__device__ __forceinline__ void class_masks(const SweepArgs& a, uint64_t* s_cmask) {
  if (threadIdx.x < 3) {
    uint64_t m = 0;
    for (int s = 0; s < a.S; ++s)
      if ((a.cls ? a.cls[s] : 0) == (int)threadIdx.x) m |= 1ull << s;
    s_cmask[threadIdx.x] = m;
  }
}

// Every valid item's co-rank in sibling s2, whose stretch of events
// cb .. cb + cnt - 1 (the item's lower bounds all lie in it or just past it)
// is read from src (LDS, or memory when it is too long to stage): a
// branchless binary search, the same steps for every item and the reads of
// a step issued together.  The sibling is active in the item's interval iff
// the co-rank (cb - L + position) is odd, and the event at the position is
// the sibling's next event.
__device__ __forceinline__ void sibling_search(const SweepArgs& a, const uint64_t* src, int32_t cnt, int32_t cb,
                                               int32_t L, int s2, const uint64_t* key, uint32_t valid, uint64_t& m8,
                                               uint64_t* tn) {
  if (!valid) return;
  const uint64_t tmask = (1ull << a.wb1) - 1;
  const int32_t cmax = cnt > 0 ? cnt - 1 : 0;
  constexpr int HB = SW_ITEMS / 2;  // two halves, to bound the registers in flight
#pragma unroll
  for (int hb = 0; hb < SW_ITEMS; hb += HB) {
    int32_t pos[HB];
#pragma unroll
    for (int u = 0; u < HB; ++u) pos[u] = 0;
    int32_t len = cnt;
    while (len > 1) {
      const int32_t half = len >> 1;
      uint64_t v[HB];
#pragma unroll
      for (int u = 0; u < HB; ++u) v[u] = src[pos[u] + half];
#pragma unroll
      for (int u = 0; u < HB; ++u) pos[u] = v[u] < key[hb + u] ? pos[u] + half : pos[u];
      len -= half;
    }
    uint64_t v[HB];
#pragma unroll
    for (int u = 0; u < HB; ++u) v[u] = src[pos[u]];
#pragma unroll
    for (int u = 0; u < HB; ++u) pos[u] += cnt > 0 && v[u] < key[hb + u];
#pragma unroll
    for (int u = 0; u < HB; ++u) v[u] = src[min(pos[u], cmax)];  // the head
#pragma unroll
    for (int u = 0; u < HB; ++u) {
      const int j = hb + u;
      const bool ok = (valid >> j) & 1;
      m8 |= ok && ((cb - L + pos[u]) & 1) ? (uint64_t)(1u << s2) << (8 * j) : 0ull;
      const uint64_t t2 = (v[u] >> a.sb) & tmask;
      tn[j] = ok && pos[u] < cnt && t2 < tn[j] ? t2 : tn[j];
    }
  }
}

// sibling_search for a stretch too long to stage: samp[x] holds the key at
// stretch position x * k (ns of them).  An item's first sample at or above
// it (a branchless search in LDS) brackets its lower bound within k
// positions, which a binary search in memory narrows.  Halves of the items
// with none valid in the lane are skipped.
__device__ __forceinline__ void sibling_search_sampled(const SweepArgs& a, const uint64_t* samp, int32_t ns, int32_t k,
                                                       const uint64_t* src, int32_t cnt, int32_t cb, int32_t L, int s2,
                                                       const uint64_t* key, uint32_t valid, uint64_t& m8,
                                                       uint64_t* tn) {
  const uint64_t tmask = (1ull << a.wb1) - 1;
  constexpr int HB = SW_ITEMS / 2;
#pragma unroll
  for (int hb = 0; hb < SW_ITEMS; hb += HB) {
    if (((valid >> hb) & ((1u << HB) - 1)) == 0) continue;
    int32_t idx[HB];
#pragma unroll
    for (int u = 0; u < HB; ++u) idx[u] = 0;
    int32_t len = ns;
    while (len > 1) {  // last sample below the key (or 0)
      const int32_t half = len >> 1;
      uint64_t v[HB];
#pragma unroll
      for (int u = 0; u < HB; ++u) v[u] = samp[idx[u] + half];
#pragma unroll
      for (int u = 0; u < HB; ++u) idx[u] = v[u] < key[hb + u] ? idx[u] + half : idx[u];
      len -= half;
    }
    // the lower bound lies in [lo, lo + w]: lo just past the last sample
    // below the key, w up to k - 1 further
    int32_t lo[HB], w[HB];
#pragma unroll
    for (int u = 0; u < HB; ++u) {
      const bool below = samp[idx[u]] < key[hb + u];
      lo[u] = below ? idx[u] * k + 1 : 0;
      const int32_t top = below ? min((idx[u] + 1) * k, cnt) : 0;
      w[u] = top - lo[u];
    }
    for (int32_t r = k; r > 0; r >>= 1) {  // at most log2(k) + 1 steps
      uint64_t v[HB];
#pragma unroll
      for (int u = 0; u < HB; ++u) v[u] = src[min(lo[u] + (w[u] >> 1), cnt - 1)];
#pragma unroll
      for (int u = 0; u < HB; ++u) {
        const int32_t h = w[u] >> 1;
        const bool b = w[u] > 0 && v[u] < key[hb + u];
        lo[u] = b ? lo[u] + h + 1 : lo[u];
        w[u] = w[u] > 0 ? (b ? w[u] - h - 1 : h) : 0;
      }
    }
#pragma unroll
    for (int u = 0; u < HB; ++u) {
      const int j = hb + u;
      const bool ok = (valid >> j) & 1;
      m8 |= ok && ((cb - L + lo[u]) & 1) ? (uint64_t)(1u << s2) << (8 * j) : 0ull;
      if (ok && lo[u] < cnt) {
        const uint64_t t2 = (src[lo[u]] >> a.sb) & tmask;
        tn[j] = t2 < tn[j] ? t2 : tn[j];
      }
    }
  }
}

// Up to 8 streams and SW_GROUPS (pid, stream) groups: tiles of SW_TILE
// events inside one group, numbered group after group (each workgroup
// finds its group from the groups' tile counts), items striped over the
// workgroup so that neighbouring lanes hold neighbouring events.  For each
// sibling the tile's events fall among a stretch of the sibling's events
// (its co-ranks of the tile's first and last events, by two wave searches),
// which is staged in LDS when it fits SB_CAP (else every k-th key of it is,
// and a short search in memory follows); every item takes its co-rank
// by a binary search there (the reads of a step issued together), the
// sibling is active in the item's interval iff the co-rank is odd, and the
// event at the co-rank is the sibling's next event.  Interval lengths are
// summed per active-stream mask in LDS and expanded at the end.
__global__ __launch_bounds__(SW_THREADS) void k_sweep_groups(SweepArgs a) {
  __shared__ uint64_t s_sib[SB_CAP];  // one chunk of a sibling's stretch
  __shared__ unsigned long long s_mlen[256];
  __shared__ unsigned long long s_sub[256];
  __shared__ unsigned long long s_cls[13];  // class_busy[3], class_overlap[9], any
  __shared__ uint64_t s_cmask[3];
  __shared__ int32_t s_goff[SW_GROUPS + 1];  // first event of each group
  __shared__ int32_t s_toff[SW_GROUPS + 1];  // first tile of each group
  __shared__ int32_t s_rng[2 * SW_SMAX];     // per sibling: its co-ranks of the tile's first and last events
  const int tid = threadIdx.x, wv = tid / WAVE, lane = lane_id();
  const int S = a.S, G = a.P * S;
  for (int g = tid; g <= G; g += SW_THREADS) s_goff[g] = a.seg_off[g];
  for (int i = tid; i < 256; i += SW_THREADS) s_mlen[i] = 0;
  if (tid < 13) s_cls[tid] = 0;
  class_masks(a, s_cmask);
  __syncthreads();
  if (wv == 0) {  // tiles per group, exclusive prefix over the groups
    int32_t run = 0;
    for (int g0 = 0; g0 <= G; g0 += WAVE) {  // uniform over the wave
      const int g = g0 + lane;
      const int32_t c = g < G ? (int32_t)cdiv((int64_t)(s_goff[g + 1] - s_goff[g]), (int64_t)SW_TILE) : 0;
      int32_t incl = c;
      for (int d = 1; d < WAVE; d <<= 1) {
        const int32_t o = shfl_up(incl, d);
        if (lane >= d) incl += o;
      }
      if (g <= G) s_toff[g] = run + incl - c;
      run += shfl(incl, WAVE - 1);
    }
  }
  __syncthreads();
  const int32_t b = (int32_t)blockIdx.x;
  if (b >= s_toff[G]) return;  // past the last tile (uniform over the workgroup)
  int glo = 0, ghi = G - 1;      // the last group whose tiles start at or before b
  while (glo < ghi) {
    const int mid = (glo + ghi + 1) >> 1;
    if (s_toff[mid] <= b)
      glo = mid;
    else
      ghi = mid - 1;
  }
  const int g = glo, pid = g / S, st = g - pid * S;
  const int32_t own_L = s_goff[g], own_R = s_goff[g + 1];
  const int64_t base = own_L + (int64_t)(b - s_toff[g]) * SW_TILE;
  const int64_t end = min<int64_t>(base + SW_TILE, own_R);
  const uint64_t tmask = (1ull << a.wb1) - 1;
  const uint64_t cm[3] = {s_cmask[0], s_cmask[1], s_cmask[2]};

  uint64_t key[SW_ITEMS], tn[SW_ITEMS];
  uint64_t m8 = 0;    // item j's active-stream mask in bits [8 j, 8 j + 8)
  uint32_t valid = 0;  // bit j: item j exists
#pragma unroll
  for (int j = 0; j < SW_ITEMS; ++j) {
    const int64_t i = base + (int64_t)j * SW_THREADS + tid;
    const bool ok = i < end;
    key[j] = ok ? a.ev[i] : ~0ull;
    // the own stream: the next event, and active after a start (even index)
    const uint64_t nk = ok && i + 1 < own_R ? a.ev[i + 1] : ~0ull;
    tn[j] = nk != ~0ull ? (nk >> a.sb) & tmask : ~0ull;
    m8 |= ok && ((i - own_L) & 1) == 0 ? (uint64_t)(1u << st) << (8 * j) : 0ull;
    valid |= ok ? 1u << j : 0u;
  }
  const uint64_t kf = a.ev[base], kl = a.ev[end - 1];
  for (int q = wv; q < 2 * S; q += SW_THREADS / WAVE) {
    const int s2 = q >> 1;
    if (s2 == st) continue;
    const int32_t c = wave_lower_bound(a.ev, s_goff[pid * S + s2], s_goff[pid * S + s2 + 1], (q & 1) ? kl : kf);
    if (lane == 0) s_rng[q] = c;
  }
  __syncthreads();
  for (int s2 = 0; s2 < S; ++s2) {  // uniform over the workgroup
    if (s2 == st) continue;
    // the tile's events fall among the sibling's events [c0, hi): up to the
    // last one's co-rank, and the head after it
    const int32_t L = s_goff[pid * S + s2], R = s_goff[pid * S + s2 + 1];
    const int32_t c0 = s_rng[2 * s2];
    const int32_t hi = min(s_rng[2 * s2 + 1] + 1, R);
    // a stretch that fits the LDS buffer is staged there; a longer one (a
    // sparse stream's tile over a dense sibling) is searched in memory
    const int32_t cnt = hi - c0;
    if (cnt <= SB_CAP) {
      stage_keys(a.ev + c0, cnt, s_sib);
      __syncthreads();
      sibling_search(a, s_sib, cnt, c0, L, s2, key, valid, m8, tn);
      __syncthreads();  // the next sibling's stretch overwrites this one
    } else {
      // every k-th key of the stretch in LDS: an item's lower bound lies
      // within k keys after the first staged key at or above it
      const int32_t k = (int32_t)cdiv((int64_t)cnt, (int64_t)SB_CAP), ns = (int32_t)cdiv((int64_t)cnt, (int64_t)k);
      stage_keys(a.ev + c0, ns, s_sib, k);
      __syncthreads();
      sibling_search_sampled(a, s_sib, ns, k, a.ev + c0, cnt, c0, L, s2, key, valid, m8, tn);
      __syncthreads();
    }
  }
  // a thread's intervals with one mask are summed before the atomic
  uint32_t cur_m = 0;
  int64_t cur_len = 0;
#pragma unroll
  for (int j = 0; j < SW_ITEMS; ++j) {
    const uint32_t mj = (uint32_t)(m8 >> (8 * j)) & 255;
    if (!((valid >> j) & 1) || mj == 0 || tn[j] == ~0ull) continue;
    const int64_t len = (int64_t)tn[j] - (int64_t)((key[j] >> a.sb) & tmask);
    if (len <= 0) continue;
    if (mj != cur_m) {
      if (cur_len) atomicAdd(&s_mlen[cur_m], (unsigned long long)cur_len);
      cur_m = mj;
      cur_len = 0;
    }
    cur_len += len;
  }
  if (cur_len) atomicAdd(&s_mlen[cur_m], (unsigned long long)cur_len);
  __syncthreads();
  flush_masks(a, pid, s_mlen, s_sub, s_cls, cm);
}

// Any number of streams and groups: tiles by position (several groups and
// processes in one), every item searching its siblings in memory, intervals
// added to the pair matrix of the workgroup's first process in LDS (others
// straight to the outputs).
__global__ __launch_bounds__(SW_THREADS) void k_sweep_global(SweepArgs a) {
  __shared__ unsigned long long s_pair[64 * 64];
  __shared__ unsigned long long s_cls[13];  // class_busy[3], class_overlap[9], any
  __shared__ uint64_t s_cmask[3];
  const int tid = threadIdx.x;
  const int32_t n = a.ds->nEv;
  const int64_t base = (int64_t)blockIdx.x * SW_TILE;
  if (base >= n) return;
  const int S = a.S;
  for (int i = tid; i < 64 * 64; i += SW_THREADS) s_pair[i] = 0;
  if (tid < 13) s_cls[tid] = 0;
  class_masks(a, s_cmask);
  const uint64_t tmask = (1ull << a.wb1) - 1;
  const uint64_t smask = (1ull << a.sb) - 1;
  const int pshift = a.wb1 + a.sb;
  const int pid0 = (int)(a.ev[base] >> pshift);
  __syncthreads();
  const uint64_t cm[3] = {s_cmask[0], s_cmask[1], s_cmask[2]};
  for (int jt = 0; jt < SW_ITEMS; ++jt) {
    const int64_t i = base + (int64_t)jt * SW_THREADS + tid;
    if (i >= n) break;
    const uint64_t key = a.ev[i];
    uint64_t m, tn;
    item_global(a, i, key, tmask, smask, pshift, &m, &tn);
    if (m == 0 || tn == ~0ull) continue;
    const int64_t len = (int64_t)tn - (int64_t)((key >> a.sb) & tmask);
    if (len <= 0) continue;
    add_interval(a, m, len, (int)(key >> pshift), pid0, cm, s_pair, s_cls);
  }
  __syncthreads();
  if (a.pair) {
    for (int i = tid; i < S * S; i += SW_THREADS)
      if (s_pair[i]) atomicAdd((unsigned long long*)&a.pair[(int64_t)pid0 * S * S + i], s_pair[i]);
  }
  if (a.class_busy && tid < 3 && s_cls[tid])
    atomicAdd((unsigned long long*)&a.class_busy[pid0 * 3 + tid], s_cls[tid]);
  if (a.class_overlap && tid >= 3 && tid < 12 && s_cls[tid])
    atomicAdd((unsigned long long*)&a.class_overlap[pid0 * 9 + (tid - 3)], s_cls[tid]);
  if (a.any_busy && tid == 12 && s_cls[12]) atomicAdd((unsigned long long*)&a.any_busy[pid0], s_cls[12]);
}

void launch_overlap(Ctx& c) {
  SweepArgs a;
  a.ev = c.ev_keys;
  a.seg_off = c.seg_off;
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
  const int64_t nseg = (int64_t)c.P * c.S + 1;
  hipLaunchKernelGGL(k_segoff, dim3((unsigned)std::min<int64_t>(cdiv(nseg, 256 / WAVE), 1024)), dim3(256), 0, c.st, a);
  const int64_t G = (int64_t)c.P * c.S;
  if (c.S <= SW_SMAX && G <= SW_GROUPS) {
    // at most one partial tile per group beyond the full ones
    hipLaunchKernelGGL(k_sweep_groups, dim3((unsigned)(cdiv(c.ev_cap, SW_TILE) + G)), dim3(SW_THREADS), 0, c.st, a);
  } else {
    hipLaunchKernelGGL(k_sweep_global, dim3((unsigned)std::max<int64_t>(cdiv(c.ev_cap, SW_TILE), 1)),
                       dim3(SW_THREADS), 0, c.st, a);
  }
}

}  // namespace hx
