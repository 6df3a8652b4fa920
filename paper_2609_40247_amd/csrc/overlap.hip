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
// With up to 8 streams the co-ranks come from a merge path over every pair
// of a process's groups (each thread takes a fixed number of merge steps,
// whatever the two groups' densities); with more, from binary searches.
// The interval's length is added to every active pair, to the classes
// present and to "any".
#include "internal.hpp"

namespace hx {

constexpr int SW_THREADS = 512;
constexpr int SW_ITEMS = 8;
constexpr int SW_TILE = SW_THREADS * SW_ITEMS;
constexpr int CR_STEPS = 8;  // merge-path steps per thread
constexpr int CR_SMAX = 8;    // most streams handled with pairwise merges

struct SweepArgs {
  const uint64_t* ev;  // (pid << (wb1 + sb)) | (t << sb) | stream, grouped by (pid, stream)
  int32_t* seg_off;    // [P * S + 1] first event of each group
  int32_t* corank;     // [S][ev_cap] co-rank of each event in each sibling group (S <= 8)
  int64_t ev_cap;
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

// Co-ranks by merge path.  For process p the pairs (s, s2), s < s2, of its
// groups are laid end to end; the merge of pair (s, s2) has n_s + n_s2
// steps, so p owns (S - 1) * n_p steps and the steps of all processes form
// one index space in process order.  A workgroup takes CR_TILE consecutive
// steps.  Inside one pair (the common case) it finds the merge positions of
// its two ends with 64-ary wave searches, stages the two key ranges in LDS,
// gives each thread CR_STEPS steps located by a binary search in LDS, and
// writes both co-rank ranges coalesced.  A workgroup whose steps straddle
// pairs lets every thread find its own position in global memory instead.
// Each merge step emits the co-rank of the smaller head in the other group
// (keys of different streams never tie).
constexpr int CR_THREADS = 512;
constexpr int CR_TILE = CR_THREADS * CR_STEPS;

struct PairPos {
  int p, s, s2;
  int32_t LA, nA, LB, nB;
  int64_t dl;  // steps into the pair's merge
};

// Pair and offset of global step d (d < (S - 1) * n).
__device__ PairPos locate_step(const SweepArgs& a, int64_t d) {
  const int32_t* off = a.seg_off;
  const int S = a.S;
  int lo = 0, hi = a.P - 1;  // the last process whose steps start at or before d
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((int64_t)(S - 1) * off[mid * S] <= d)
      lo = mid;
    else
      hi = mid - 1;
  }
  PairPos q;
  q.p = lo;
  q.s = 0;
  q.s2 = 1;
  q.dl = d - (int64_t)(S - 1) * off[lo * S];
  const int32_t* o = off + (int64_t)lo * S;
  q.LA = o[0];
  q.nA = o[1] - q.LA;
  q.LB = o[1];
  q.nB = o[2] - q.LB;
  while (q.dl >= (int64_t)q.nA + q.nB) {  // pairs wholly before d (all in process p)
    q.dl -= (int64_t)q.nA + q.nB;
    if (++q.s2 == S) {
      ++q.s;
      q.s2 = q.s + 1;
    }
    q.LA = o[q.s];
    q.nA = o[q.s + 1] - q.LA;
    q.LB = o[q.s2];
    q.nB = o[q.s2 + 1] - q.LB;
  }
  return q;
}

// Number of A keys among the first d merged keys of A = ev[LA, LA + nA) and
// B = ev[LB, LB + nB), by a 64-ary search of the diagonal: every lane probes
// one point per round and a ballot keeps the stretch where the answer lies.
// Called by a whole wave; every lane gets the answer.
__device__ int32_t wave_diag_search(const uint64_t* __restrict__ ev, int32_t LA, int32_t nA, int32_t LB, int32_t nB,
                                    int64_t d) {
  const int lane = lane_id();
  int32_t lo = (int32_t)max<int64_t>(0, d - nB), hi = (int32_t)min<int64_t>(d, nA);
  while (lo < hi) {  // answer in [lo, hi]; A[i] < B[d-1-i] holds exactly for i < answer
    const int32_t step = (hi - lo + WAVE - 1) / WAVE;
    const int32_t x = lo + lane * step;
    const bool probe = x < hi;
    const bool f = probe && ev[LA + x] < ev[LB + (int32_t)(d - 1 - x)];
    const uint64_t bf = ballot(f);
    const int k = popc(bf);  // lanes 0..k-1 probed true (monotone)
    const int32_t nlo = k > 0 ? lo + (k - 1) * step + 1 : lo;
    const int32_t xk = lo + k * step;
    hi = xk < hi ? xk : hi;
    lo = nlo;
  }
  return lo;
}

// Generic path: the thread locates its own first step and merges.
__device__ void corank_steps(const SweepArgs& a, int64_t d0, int64_t steps) {
  const int S = a.S;
  const int32_t* off = a.seg_off;
  PairPos q = locate_step(a, d0);
  int p = q.p, s = q.s, s2 = q.s2;
  int32_t LA = q.LA, nA = q.nA, LB = q.LB, nB = q.nB;
  const int64_t dl = q.dl;
  int32_t ilo = (int32_t)max<int64_t>(0, dl - nB), ihi = (int32_t)min<int64_t>(dl, nA);
  while (ilo < ihi) {
    const int32_t mid = (ilo + ihi) >> 1;
    if (a.ev[LA + mid] < a.ev[LB + (int32_t)dl - mid - 1])
      ilo = mid + 1;
    else
      ihi = mid;
  }
  int32_t i = ilo, j = (int32_t)dl - ilo;
  uint64_t va = i < nA ? a.ev[LA + i] : ~0ull;
  uint64_t vb = j < nB ? a.ev[LB + j] : ~0ull;
  while (steps > 0) {
    if (i == nA && j == nB) {  // next pair, or the first pair of the next process
      if (++s2 == S) {
        ++s;
        s2 = s + 1;
      }
      if (s >= S - 1) {
        ++p;
        s = 0;
        s2 = 1;
      }
      LA = off[p * S + s];
      nA = off[p * S + s + 1] - LA;
      LB = off[p * S + s2];
      nB = off[p * S + s2 + 1] - LB;
      i = j = 0;
      va = nA > 0 ? a.ev[LA] : ~0ull;
      vb = nB > 0 ? a.ev[LB] : ~0ull;
      continue;
    }
    if (va < vb) {
      a.corank[(int64_t)s2 * a.ev_cap + LA + i] = j;
      ++i;
      va = i < nA ? a.ev[LA + i] : ~0ull;
    } else {
      a.corank[(int64_t)s * a.ev_cap + LB + j] = i;
      ++j;
      vb = j < nB ? a.ev[LB + j] : ~0ull;
    }
    --steps;
  }
}

__global__ __launch_bounds__(CR_THREADS) void k_corank(SweepArgs a) {
  __shared__ uint64_t s_key[CR_TILE];  // A range, then B range
  __shared__ int32_t s_out[CR_TILE];   // co-ranks in the same layout
  __shared__ int32_t s_split[2];
  const int tid = threadIdx.x, wv = tid / WAVE;
  const int64_t n = a.ds->nEv;
  const int S = a.S;
  const int64_t total = (int64_t)(S - 1) * n;
  const int64_t D0 = (int64_t)blockIdx.x * CR_TILE;
  if (D0 >= total) return;
  const int64_t cnt = min<int64_t>(CR_TILE, total - D0);
  const PairPos q0 = locate_step(a, D0);
  const bool one_pair = q0.dl + cnt <= (int64_t)q0.nA + q0.nB;
  if (!one_pair) {
    const int64_t d0 = D0 + (int64_t)tid * CR_STEPS;
    if (d0 < total) corank_steps(a, d0, min<int64_t>(CR_STEPS, total - d0));
    return;
  }
  // merge positions of the tile's two ends
  if (wv < 2) {
    const int64_t d = q0.dl + (wv == 0 ? 0 : cnt);
    const int32_t i = wave_diag_search(a.ev, q0.LA, q0.nA, q0.LB, q0.nB, d);
    if (lane_id() == 0) s_split[wv] = i;
  }
  __syncthreads();
  const int32_t i0 = s_split[0], i1 = s_split[1];
  const int32_t j0 = (int32_t)q0.dl - i0, j1 = (int32_t)(q0.dl + cnt) - i1;
  const int32_t na = i1 - i0, nb = j1 - j0;  // na + nb == cnt
  for (int x = tid; x < na; x += CR_THREADS) s_key[x] = a.ev[q0.LA + i0 + x];
  for (int y = tid; y < nb; y += CR_THREADS) s_key[na + y] = a.ev[q0.LB + j0 + y];
  __syncthreads();
  const uint64_t* A = s_key;
  const uint64_t* B = s_key + na;
  const int32_t dd = tid * CR_STEPS;
  if (dd < cnt) {
    int32_t lo = max(0, dd - nb), hi = min(dd, na);
    while (lo < hi) {
      const int32_t mid = (lo + hi) >> 1;
      if (A[mid] < B[dd - 1 - mid])
        lo = mid + 1;
      else
        hi = mid;
    }
    int32_t i = lo, j = dd - lo;
    const int32_t steps = min<int32_t>(CR_STEPS, (int32_t)cnt - dd);
    for (int k = 0; k < steps; ++k) {
      const bool takeA = j >= nb || (i < na && A[i] < B[j]);
      if (takeA) {
        s_out[i] = j0 + j;
        ++i;
      } else {
        s_out[na + j] = i0 + i;
        ++j;
      }
    }
  }
  __syncthreads();
  int32_t* outA = a.corank + (int64_t)q0.s2 * a.ev_cap + q0.LA + i0;
  int32_t* outB = a.corank + (int64_t)q0.s * a.ev_cap + q0.LB + j0;
  for (int x = tid; x < na; x += CR_THREADS) outA[x] = s_out[x];
  for (int y = tid; y < nb; y += CR_THREADS) outB[y] = s_out[na + y];
}

// One event per thread and item (items striped over the workgroup).  With
// at most 8 streams a workgroup sums interval lengths per active-stream mask
// in LDS and expands the 2^S sums into pairs, classes and "any" at the end;
// with more streams every interval is added to the pair matrix in LDS
// directly.  Intervals of a process other than the workgroup's first go
// straight to the outputs.
template <int SMAX>
__global__ __launch_bounds__(SW_THREADS) void k_sweep(SweepArgs a) {
  constexpr bool SMALL = SMAX <= CR_SMAX;
  __shared__ unsigned long long s_mlen[SMALL ? 256 : 1];
  __shared__ unsigned long long s_pair[SMALL ? 1 : 64 * 64];
  __shared__ unsigned long long s_cls[13];  // class_busy[3], class_overlap[9], any
  __shared__ uint64_t s_cmask[3];
  __shared__ int32_t s_off0[SMAX + 1];  // group starts of the workgroup's first process
  const int tid = threadIdx.x;
  const int32_t n = a.ds->nEv;
  const int64_t base = (int64_t)blockIdx.x * SW_TILE;
  if (base >= n) return;
  const int S = a.S;
  if (SMALL) {
    for (int i = tid; i < 256; i += SW_THREADS) s_mlen[i] = 0;
  } else {
    for (int i = tid; i < 64 * 64; i += SW_THREADS) s_pair[i] = 0;
  }
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
  const int pid0 = (int)(a.ev[base] >> pshift);
  if (SMALL && tid <= S) s_off0[tid] = a.seg_off[pid0 * S + tid];
  __syncthreads();
  const uint64_t cm[3] = {s_cmask[0], s_cmask[1], s_cmask[2]};

  if constexpr (SMALL) {
    // Items in batches whose loads are issued together: keys, own successors
    // and co-ranks (addresses known up front), then the sibling heads.
    constexpr int BT = 32 / SMAX;
    for (int jb = 0; jb < SW_ITEMS; jb += BT) {
      uint64_t key[BT], nk[BT];
      int32_t cr[BT][SMAX];
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        const int64_t i = base + (int64_t)(jb + b) * SW_THREADS + tid;
        key[b] = i < n ? a.ev[i] : ~0ull;
        nk[b] = i + 1 < n ? a.ev[i + 1] : ~0ull;
        // the co-rank buffer exists only with two or more streams; the entry
        // of the event's own stream is loaded (it lies inside the buffer)
        // before the stream is known, and never used
#pragma unroll
        for (int s = 0; s < SMAX; ++s)
          cr[b][s] = S > 1 && i < n && s < S ? a.corank[(int64_t)s * a.ev_cap + i] : 0;
      }
#pragma unroll
      for (int b = 0; b < BT; ++b) {
        const int64_t i = base + (int64_t)(jb + b) * SW_THREADS + tid;
        if (i >= n) continue;
        const int pid = (int)(key[b] >> pshift);
        const int st = (int)(key[b] & smask);
        int32_t off[SMAX + 1];
#pragma unroll
        for (int s = 0; s <= SMAX; ++s)
          off[s] = s <= S ? (pid == pid0 ? s_off0[s] : a.seg_off[pid * S + s]) : 0;
        int32_t own_L = 0, own_R = 0;
#pragma unroll
        for (int s = 0; s < SMAX; ++s)
          if (s == st) {
            own_L = off[s];
            own_R = off[s + 1];
          }
        // its own stream is active after a start (even index in its group);
        // a sibling iff an odd number of its events precede this one
        uint64_t m = ((i - own_L) & 1) == 0 ? 1ull << st : 0ull;
        uint64_t tn = i + 1 < own_R ? (nk[b] >> a.sb) & tmask : ~0ull;
        uint64_t hv[SMAX];
#pragma unroll
        for (int s = 0; s < SMAX; ++s) {
          const bool sib = s < S && s != st;
          hv[s] = sib && (uint32_t)cr[b][s] < (uint32_t)(off[s + 1] - off[s]) ? a.ev[off[s] + cr[b][s]] : ~0ull;
        }
#pragma unroll
        for (int s = 0; s < SMAX; ++s) {
          if (s >= S || s == st) continue;
          if (cr[b][s] & 1) m |= 1ull << s;
          if (hv[s] != ~0ull) {
            const uint64_t t2 = (hv[s] >> a.sb) & tmask;
            tn = t2 < tn ? t2 : tn;
          }
        }
        if (m == 0 || tn == ~0ull) continue;
        const int64_t len = (int64_t)tn - (int64_t)((key[b] >> a.sb) & tmask);
        if (len <= 0) continue;
        if (pid == pid0)
          atomicAdd(&s_mlen[m], (unsigned long long)len);
        else
          add_interval(a, m, len, pid, pid0, cm, s_pair, s_cls);
      }
    }
  } else {
    for (int jt = 0; jt < SW_ITEMS; ++jt) {
      const int64_t i = base + (int64_t)jt * SW_THREADS + tid;
      if (i >= n) break;
      const uint64_t key = a.ev[i];
      const int pid = (int)(key >> pshift);
      const int st = (int)(key & smask);
      const int g = pid * S + st;
      uint64_t m = 0, tn = ~0ull;
      const int32_t own_L = a.seg_off[g], own_R = a.seg_off[g + 1];
      // many streams: one plain binary search per sibling
      for (int s = 0; s < S; ++s) {
        if (s == st) continue;
        const int32_t Lq = a.seg_off[pid * S + s], Rq = a.seg_off[pid * S + s + 1];
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
      // its own stream is active after a start (even index in its group)
      if (((i - own_L) & 1) == 0) m |= 1ull << st;
      if (i + 1 < own_R) {
        const uint64_t t2 = (a.ev[i + 1] >> a.sb) & tmask;
        tn = t2 < tn ? t2 : tn;
      }
      if (m == 0 || tn == ~0ull) continue;
      const int64_t len = (int64_t)tn - (int64_t)((key >> a.sb) & tmask);
      if (len <= 0) continue;
      add_interval(a, m, len, pid, pid0, cm, s_pair, s_cls);
    }
  }
  __syncthreads();
  if (SMALL) {
    // expand the per-mask sums: one thread per output entry
    const int nm = 1 << S;
    if (tid < S * S) {
      const int i = tid / S, jj = tid % S;
      const uint64_t need = (1ull << i) | (1ull << jj);
      unsigned long long v = 0;
      for (int mk = 1; mk < nm; ++mk)
        if (((uint64_t)mk & need) == need) v += s_mlen[mk];
      if (v && a.pair) atomicAdd((unsigned long long*)&a.pair[((int64_t)pid0 * S + i) * S + jj], v);
    } else if (tid >= 64 && tid < 64 + 13) {
      const int e = tid - 64;  // 0..2 class busy, 3..11 class pairs, 12 any
      unsigned long long v = 0;
      for (int mk = 1; mk < nm; ++mk) {
        const uint64_t mm = (uint64_t)mk;
        bool hit;
        if (e < 3)
          hit = (mm & cm[e]) != 0;
        else if (e < 12)
          hit = (mm & cm[(e - 3) / 3]) != 0 && (mm & cm[(e - 3) % 3]) != 0;
        else
          hit = true;
        if (hit) v += s_mlen[mk];
      }
      s_cls[e] = v;
    }
    __syncthreads();
  }
  if (!SMALL && a.pair) {
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
  a.corank = c.corank;
  a.ev_cap = c.ev_cap;
  const int64_t nseg = (int64_t)c.P * c.S + 1;
  hipLaunchKernelGGL(k_segoff, dim3((unsigned)std::min<int64_t>(cdiv(nseg, 256 / WAVE), 1024)), dim3(256), 0, c.st, a);
  const dim3 grid((unsigned)std::max<int64_t>(cdiv(c.ev_cap, SW_TILE), 1));
  if (c.S > 1 && c.S <= CR_SMAX) {
    const int64_t steps = (int64_t)(c.S - 1) * c.ev_cap;
    hipLaunchKernelGGL(k_corank, dim3((unsigned)std::max<int64_t>(cdiv(steps, CR_TILE), 1)), dim3(CR_THREADS), 0, c.st,
                       a);
  }
  if (c.S <= 4)
    hipLaunchKernelGGL(k_sweep<4>, grid, dim3(SW_THREADS), 0, c.st, a);
  else if (c.S <= CR_SMAX)
    hipLaunchKernelGGL(k_sweep<CR_SMAX>, grid, dim3(SW_THREADS), 0, c.st, a);
  else
    hipLaunchKernelGGL(k_sweep<64>, grid, dim3(SW_THREADS), 0, c.st, a);
}

}  // namespace hx
