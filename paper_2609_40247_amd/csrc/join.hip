// Launch <-> kernel join and cross-process waits.
//
// The correlation id associates a submission with its device activity
// (Section 5.2); kernel composition is recovered from these call-to-kernel
// links (Section 6.1), and a graph launch may own many kernels.  Launches and
// kernels are sorted by (pid, corr, is_kernel), so each id is one run with
// its launches first: a kernel's launch is the head of its run (the smallest
// row, the sort being stable), extra launches are duplicates.  Run bounds are
// found by galloping searches, which cost O(log run length).  The latency is
// the kernel start minus the launch start (the host submission time of the
// operator panel) binned by floor(log2)+1.  Dependency edges (panel
// "Cross-process blocking") are binary searches into the same sorted runs.
//
// When a call has at most JT_PROCS processes and their correlation ids span
// at most two slots per row (ids are dense per process: every API call takes
// the next one), a table indexed by (process, id) replaces the sort.  Bulk
// global atomics are slow on this GPU, so the table is built with plain
// stores and checked: launches store their rows (one writer wins), those
// that lost are the duplicates and put the smallest row in (atomics, rare);
// kernels store their rows in an owner word, and only kernels sharing a slot
// (graph replays) add to their launch's counts with atomics.  The decision
// is taken on the device right after prep, which finds each process's id
// range; the join sort's histogram and digit passes are then skipped.
#include "internal.hpp"

namespace hx {

struct JoinArgs {
  const uint64_t* k[2];
  const uint32_t* v[2];
  const int64_t* ts;
  const int64_t* te;
  const int64_t* off;
  DevState* ds;
  herschel_counters* cnt;
  int32_t* link;
  int32_t* aux;
  int64_t* lat_hist;
  int64_t* lk_first;
  int64_t* lk_last;
  int64_t* lk_sum;
  bool contain;
  const herschel_edge* edges;
  int64_t n_edges;
  int P;
  int64_t* edge_wait;
  int32_t* edge_status;
  // correlation table (processes <= JT_PROCS)
  uint32_t* tab;
  uint32_t* own;
  uint8_t* multi;
  int64_t* kmax;
  int64_t* kmin;
  int64_t cap;
  const uint32_t* k_rows;  // admitted kernels' rows (prep's list)
};

// Smallest index in [lo, hi) whose key is >= target (hi if none); galloping
// from lo.
__device__ int64_t gallop_ge(const uint64_t* keys, int64_t lo, int64_t hi, uint64_t target) {
  if (lo >= hi || keys[lo] >= target) return lo;
  int64_t a = lo, b = lo + 1, step = 1;
  while (b < hi && keys[b] < target) {
    a = b;
    step <<= 1;
    b = a + step;
  }
  if (b > hi) b = hi;
  while (b - a > 1) {
    const int64_t mid = a + (b - a) / 2;
    if (keys[mid] < target)
      a = mid;
    else
      b = mid;
  }
  return b;
}

// Smallest index <= i whose key is >= target, given keys[i] >= target;
// galloping backwards from i.
__device__ int64_t gallop_back_ge(const uint64_t* keys, int64_t i, uint64_t target) {
  if (i == 0 || keys[i - 1] < target) return i;
  int64_t b = i - 1, step = 1, a = b - 1;
  while (a >= 0 && keys[a] >= target) {
    b = a;
    step <<= 1;
    a = b - step;
  }
  if (a < -1) a = -1;
  while (b - a > 1) {
    const int64_t mid = a + (b - a) / 2;
    if (keys[mid] < target)
      a = mid;
    else
      b = mid;
  }
  return b;
}

// One sorted position per thread.  The neighbours i-2 .. i+2 are
// loaded with the position itself: they settle the usual groups (one launch
// and its kernel) without a search, and the gallops handle the rest.  Counts
// and latency bins go to one of JOIN_COPIES accumulator copies (spread so
// that few workgroups add to one address); the final kernel sums them.
__global__ __launch_bounds__(256) void k_join(JoinArgs a) {
  __shared__ unsigned long long s_c[JC_N];
  __shared__ unsigned long long s_h[64];
  const int tid = threadIdx.x;
  if (tid < JC_N) s_c[tid] = 0;
  if (tid < 64) s_h[tid] = 0;
  __syncthreads();
  if (a.ds->join_direct) return;  // the correlation table did the join
  const int64_t n = a.ds->nJ;
  const int par = (int)a.ds->sort_parity[1];
  const uint64_t* keys = a.k[par];
  const uint32_t* vals = a.v[par];
  const int64_t i = (int64_t)blockIdx.x * 256 + tid;
  uint32_t c[JC_N] = {};
  if (i < n) {
    const uint64_t key = keys[i];
    const uint32_t row = vals[i];
    const uint64_t kprev = i > 0 ? keys[i - 1] : ~0ull;
    const uint64_t kprev2 = i > 1 ? keys[i - 2] : ~0ull;
    const uint64_t knext = i + 1 < n ? keys[i + 1] : ~0ull;
    const uint64_t knext2 = i + 2 < n ? keys[i + 2] : ~0ull;
    const uint64_t g = key >> 1;
    if ((key & 1) == 0) {  // launch
      if ((kprev >> 1) != g) {  // the group's head
        int64_t fk, end;
        if (knext == ((g << 1) | 1)) {
          fk = i + 1;
          end = (knext2 >> 1) != g ? i + 2 : gallop_ge(keys, i + 2, n, (g + 1) << 1);
        } else if ((knext >> 1) != g) {
          fk = end = i + 1;
        } else {
          fk = gallop_ge(keys, i + 1, n, (g << 1) | 1);
          end = gallop_ge(keys, fk, n, (g + 1) << 1);
        }
        const int64_t nk = end - fk;
        a.aux[row] = (int32_t)nk;
        if (nk == 0) ++c[JC_UNM_L];
        if (a.contain && nk > 0) {
          const int64_t o = a.off ? a.off[(int32_t)(key >> 49)] : 0;
          int64_t first = I64MAX, last = I64MIN;
          uint64_t sum = 0;
          for (int64_t q = fk; q < end; ++q) {
            const uint32_t kr = vals[q];
            const int64_t s = a.ts[kr] - o, e = a.te[kr] - o;
            first = s < first ? s : first;
            last = e > last ? e : last;
            sum += (uint64_t)(e - s);
          }
          a.lk_first[row] = first;
          a.lk_last[row] = last;
          a.lk_sum[row] = (int64_t)sum;
        }
      } else {
        a.aux[row] = 0;
        ++c[JC_DUP];
        ++c[JC_UNM_L];
      }
    } else {  // kernel: the group's head decides
      // the first position of the group: i, i - 1 (one launch before), or
      // found by galloping back (several launches, or kernels before i)
      const int64_t f = (kprev >> 1) != g                          ? i
                        : (kprev & 1) == 0 && (kprev2 >> 1) != g ? i - 1
                                                                 : gallop_back_ge(keys, i, g << 1);
      const uint64_t kf = f == i ? key : f == i - 1 ? kprev : keys[f];
      if ((kf & 1) == 0) {
        const uint32_t lrow = vals[f];
        a.link[row] = (int32_t)lrow;
        ++c[JC_MATCHED];
        const int64_t x = a.ts[row] - a.ts[lrow];  // same process: the offset cancels
        if (x < 0) ++c[JC_NEG];
        const int bin = x <= 0 ? 0 : bits_of((uint64_t)x);
        atomicAdd(&s_h[bin], 1ull);
        a.aux[row] = -1;  // the kernel's op comes later (the name pass)
      } else {
        a.link[row] = -1;
        a.aux[row] = -1;
        ++c[JC_UNM_K];
      }
    }
  }
#pragma unroll
  for (int q = 0; q < JC_N; ++q) {
    const uint64_t w = wave_sum_u64(c[q]);
    if (lane_id() == 0 && w) atomicAdd(&s_c[q], (unsigned long long)w);
  }
  __syncthreads();
  unsigned long long* acc = &a.ds->join_acc[blockIdx.x % JOIN_COPIES][0];
  if (tid < JC_N && s_c[tid]) atomicAdd(&acc[tid], s_c[tid]);
  if (tid < 64 && s_h[tid]) atomicAdd(&acc[JC_N + tid], s_h[tid]);
}

// Correlation-table plan: each process's id range (from the key range prep
// found), slot bases by an exclusive scan, and the decision.  One wave, one
// lane per process.
__device__ __forceinline__ int64_t jt_slot(const DevState* ds, uint64_t key) {
  const int p = (int)(key >> 49);
  return ds->jt_base[p] + (int64_t)((key >> 1) & ((1ull << 48) - 1)) - ds->jt_cmin[p];
}

// Empty every slot in use (and the kernel-time tables when there are edges).
__global__ __launch_bounds__(256) void k_jt_clear(JoinArgs a) {
  if (!a.ds->join_direct) return;
  const int64_t R = a.ds->jt_slots;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < R; i += (int64_t)gridDim.x * 256) {
    a.tab[i] = ~0u;
    a.multi[i] = 0;
    if (a.kmax) {
      a.kmax[i] = I64MIN;
      a.kmin[i] = I64MAX;
    }
  }
}

__device__ __forceinline__ void jt_flush(const JoinArgs& a, uint32_t (&c)[JC_N], unsigned long long* s_c,
                                         unsigned long long* s_h) {
#pragma unroll
  for (int q = 0; q < JC_N; ++q) {
    const uint64_t w = wave_sum_u64(c[q]);
    if (lane_id() == 0 && w) atomicAdd(&s_c[q], (unsigned long long)w);
  }
  __syncthreads();
  unsigned long long* acc = &a.ds->join_acc[blockIdx.x % JOIN_COPIES][0];
  if (threadIdx.x < JC_N && s_c[threadIdx.x]) atomicAdd(&acc[threadIdx.x], s_c[threadIdx.x]);
  if (s_h && threadIdx.x < 64 && s_h[threadIdx.x]) atomicAdd(&acc[JC_N + threadIdx.x], s_h[threadIdx.x]);
}

// The table passes give each thread IT positions (striped over the
// workgroup) and issue each round of their loads together: a pass is a
// short chain of dependent loads, and batching positions per thread keeps
// the number of waves the chip must cycle through low.  The check and
// kernel passes, whose chains are longest, take 8 positions a thread; the
// store and fix passes 2 (each measured best).
constexpr int JT_IT_STORE = 2, JT_IT_CHECK = 8, JT_IT_FIX = 2, JT_IT_KERNEL = 8;

// Pass 1: every launch stores its row in its slot and every kernel in its
// slot's owner word, with plain stores (one writer of each wins).
template <int IT>
__global__ __launch_bounds__(256) void k_jt_store(JoinArgs a) {
  if (!a.ds->join_direct) return;
  const int64_t n = a.ds->nJ;
  const int64_t i0 = (int64_t)blockIdx.x * (256 * IT) + threadIdx.x;
  uint64_t key[IT];
  uint32_t row[IT];
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const int64_t i = i0 + u * 256;
    const int64_t ic = i < n ? i : (n > 0 ? n - 1 : 0);  // clamped: the loads stay in flight together
    key[u] = a.k[0][ic];  // unsorted: the join sort did not run
    row[u] = a.v[0][ic];
    if (i >= n) key[u] = ~0ull;
  }
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    if (key[u] == ~0ull) continue;
    const int64_t slot = jt_slot(a.ds, key[u]);
    if (!in_range(a.ds, slot, a.cap)) continue;
    if (key[u] & 1)
      a.own[slot] = row[u];
    else
      a.tab[slot] = row[u];
  }
}

// Pass 2: a launch that lost its slot is a duplicate; a kernel that lost its
// owner word marks the slot as holding several kernels.  Launches start with
// no kernels (their kernel aggregates are read only when they have some).
template <int IT>
__global__ __launch_bounds__(256) void k_jt_check(JoinArgs a) {
  __shared__ unsigned long long s_c[JC_N];
  const int tid = threadIdx.x;
  if (tid < JC_N) s_c[tid] = 0;
  __syncthreads();
  if (!a.ds->join_direct) return;
  const int64_t n = a.ds->nJ;
  const int64_t i0 = (int64_t)blockIdx.x * (256 * IT) + tid;
  uint32_t c[JC_N] = {};
  uint64_t key[IT];
  uint32_t row[IT], w[IT];
  int64_t slot[IT];
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const int64_t i = i0 + u * 256;
    const int64_t ic = i < n ? i : (n > 0 ? n - 1 : 0);
    key[u] = a.k[0][ic];
    row[u] = a.v[0][ic];
    if (i >= n) key[u] = ~0ull;
  }
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    slot[u] = key[u] != ~0ull ? jt_slot(a.ds, key[u]) : -1;
    const bool ok = slot[u] >= 0 && in_range(a.ds, slot[u], a.cap);
    const int64_t sc = ok ? slot[u] : 0;
    // one load: the owner word for a kernel, the slot for a launch
    const uint32_t ws = ((key[u] & 1) ? a.own : a.tab)[sc];
    w[u] = !ok ? row[u] : ws;
  }
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    if (key[u] == ~0ull) continue;
    if (key[u] & 1) {
      if (w[u] != row[u]) a.multi[slot[u]] = 1;
    } else {
      if (w[u] != row[u]) ++c[JC_DUP];
      a.aux[row[u]] = 0;
    }
  }
  jt_flush(a, c, s_c, nullptr);
}

// Pass 3: duplicates put the smallest row into their slot (rare: atomics),
// and the launches of slots with several kernels start their kernel
// aggregates at the identities (the kernels add to them with atomics; a
// launch with one kernel gets plain stores).
template <int IT>
__global__ __launch_bounds__(256) void k_jt_fix(JoinArgs a) {
  if (!a.ds->join_direct) return;
  const int64_t n = a.ds->nJ;
  const int64_t i0 = (int64_t)blockIdx.x * (256 * IT) + threadIdx.x;
  uint64_t key[IT];
  uint32_t row[IT];
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const int64_t i = i0 + u * 256;
    const int64_t ic = i < n ? i : (n > 0 ? n - 1 : 0);
    key[u] = a.k[0][ic];
    row[u] = a.v[0][ic];
    if (i >= n) key[u] = 1ull;  // past the end: treated as a kernel
  }
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    if (key[u] & 1) continue;
    const int64_t slot = jt_slot(a.ds, key[u]);
    if (!in_range(a.ds, slot, a.cap)) continue;
    const uint32_t t = a.tab[slot];
    const uint8_t mu = a.multi[slot];
    if (t != row[u]) atomicMin(&a.tab[slot], row[u]);
    if (a.contain && mu) {
      a.lk_first[row[u]] = I64MAX;
      a.lk_last[row[u]] = I64MIN;
      a.lk_sum[row[u]] = 0;
    }
  }
}

// Pass 4: each kernel reads its launch, records the latency, and adds itself
// to the launch's counts: with plain stores when it is its slot's only kernel
// (the usual case), with atomics otherwise.
template <int IT>
__global__ __launch_bounds__(256) void k_jt_kernel(JoinArgs a) {
  __shared__ unsigned long long s_c[JC_N];
  __shared__ unsigned long long s_h[64];
  const int tid = threadIdx.x;
  if (tid < JC_N) s_c[tid] = 0;
  if (tid < 64) s_h[tid] = 0;
  __syncthreads();
  if (!a.ds->join_direct) return;
  const int64_t n = a.ds->nJ;
  // Positions past the end take the last entry's row (clamped loads); with
  // no entry there is no row to take, and nothing to do.
  if (n == 0) return;
  const int64_t i0 = (int64_t)blockIdx.x * (256 * IT) + tid;
  uint32_t c[JC_N] = {};
  uint64_t key[IT];
  uint32_t row[IT];
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const int64_t i = i0 + u * 256;
    const int64_t ic = i < n ? i : n - 1;
    key[u] = a.k[0][ic];
    row[u] = a.v[0][ic];
    if (i >= n) key[u] = 0ull;  // past the end: treated as a launch (skipped)
  }
  // round 2: the slot's launch and kernel count, the kernel's times
  int64_t slot[IT], ts[IT], te[IT];
  uint32_t l[IT];
  bool single[IT];
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const bool kern = (key[u] & 1) != 0;
    slot[u] = kern ? jt_slot(a.ds, key[u]) : -1;
    const bool ok = slot[u] >= 0 && in_range(a.ds, slot[u], a.cap);
    const int64_t sc = ok ? slot[u] : 0;
    const uint32_t lt = a.tab[sc];
    const uint8_t mu = a.multi[sc];
    const int64_t t0 = a.ts[row[u]], t1 = a.te[row[u]];
    l[u] = ok ? lt : ~0u;
    single[u] = ok && mu == 0;
    ts[u] = kern ? t0 : 0;
    te[u] = kern ? t1 : 0;
  }
  // round 3: the launch's start
  int64_t lts[IT];
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const bool has = (key[u] & 1) && l[u] != ~0u;
    const int64_t t = a.ts[has ? l[u] : 0u];
    lts[u] = has ? t : 0;
  }
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    if (!(key[u] & 1)) continue;
    const int64_t o = a.off ? a.off[(int32_t)(key[u] >> 49)] : 0;
    if (a.kmax && slot[u] >= 0) {
      if (single[u]) {
        a.kmax[slot[u]] = te[u] - o;
        a.kmin[slot[u]] = ts[u] - o;
      } else {
        atomicMax((long long*)&a.kmax[slot[u]], (long long)(te[u] - o));
        atomicMin((long long*)&a.kmin[slot[u]], (long long)(ts[u] - o));
      }
    }
    if (l[u] != ~0u) {
      a.link[row[u]] = (int32_t)l[u];
      ++c[JC_MATCHED];
      const int64_t x = ts[u] - lts[u];  // same process: the offset cancels
      if (x < 0) ++c[JC_NEG];
      atomicAdd(&s_h[x <= 0 ? 0 : bits_of((uint64_t)x)], 1ull);
      a.aux[row[u]] = -1;  // the kernel's op comes later (the name pass)
      if (single[u]) {
        a.aux[l[u]] = 1;
        ++c[JC_MLAUNCH];
        if (a.contain) {
          a.lk_first[l[u]] = ts[u] - o;
          a.lk_last[l[u]] = te[u] - o;
          a.lk_sum[l[u]] = te[u] - ts[u];
        }
      } else {
        if (atomicAdd(&a.aux[l[u]], 1) == 0) ++c[JC_MLAUNCH];
        if (a.contain) {
          atomicMin((long long*)&a.lk_first[l[u]], (long long)(ts[u] - o));
          atomicMax((long long*)&a.lk_last[l[u]], (long long)(te[u] - o));
          atomicAdd((unsigned long long*)&a.lk_sum[l[u]], (unsigned long long)(te[u] - ts[u]));
        }
      }
    } else {
      a.link[row[u]] = -1;
      a.aux[row[u]] = -1;
      ++c[JC_UNM_K];
    }
  }
  jt_flush(a, c, s_c, s_h);
}

__global__ __launch_bounds__(256) void k_edges(JoinArgs a) {
  if (a.ds->join_direct) {
    // table path: the kernels' latest end and earliest start per slot
    for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < a.n_edges; e += (int64_t)gridDim.x * 256) {
      const herschel_edge ed = a.edges[e];
      int found[2] = {0, 0};
      int64_t prod_end = I64MIN, cons_start = I64MAX;
      for (int side = 0; side < 2; ++side) {
        const int32_t pid = side == 0 ? ed.prod_pid : ed.cons_pid;
        const int64_t corr = side == 0 ? ed.prod_corr : ed.cons_corr;
        if (pid < 0 || pid >= a.P || corr < 0 || corr >= HERSCHEL_CORR_LIMIT) continue;
        const int64_t rel = corr - a.ds->jt_cmin[pid];
        const int64_t lim = (pid + 1 < a.P ? a.ds->jt_base[pid + 1] : a.ds->jt_slots) - a.ds->jt_base[pid];
        if (rel < 0 || rel >= lim) continue;
        const int64_t slot = a.ds->jt_base[pid] + rel;
        if (side == 0 && a.kmax[slot] != I64MIN) {
          found[0] = 1;
          prod_end = a.kmax[slot];
        }
        if (side == 1 && a.kmin[slot] != I64MAX) {
          found[1] = 1;
          cons_start = a.kmin[slot];
        }
      }
      a.edge_status[e] = (found[0] ? 0 : 1) | (found[1] ? 0 : 2);
      a.edge_wait[e] = (found[0] && found[1]) ? (int64_t)((uint64_t)cons_start - (uint64_t)prod_end) : I64MIN;
    }
    return;
  }
  const int64_t n = a.ds->nJ;
  const int par = (int)a.ds->sort_parity[1];
  const uint64_t* keys = a.k[par];
  const uint32_t* vals = a.v[par];
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < a.n_edges; e += (int64_t)gridDim.x * 256) {
    const herschel_edge ed = a.edges[e];
    int found[2] = {0, 0};
    int64_t prod_end = I64MIN, cons_start = I64MAX;
    for (int side = 0; side < 2; ++side) {
      const int32_t pid = side == 0 ? ed.prod_pid : ed.cons_pid;
      const int64_t corr = side == 0 ? ed.prod_corr : ed.cons_corr;
      if (pid < 0 || pid >= a.P || corr < 0 || corr >= HERSCHEL_CORR_LIMIT) continue;
      const uint64_t target = ((uint64_t)pid << 49) | ((uint64_t)corr << 1) | 1;
      int64_t lo = 0, hi = n;
      while (lo < hi) {
        const int64_t mid = lo + (hi - lo) / 2;
        if (keys[mid] < target)
          lo = mid + 1;
        else
          hi = mid;
      }
      const int64_t o = a.off ? a.off[pid] : 0;
      for (int64_t q = lo; q < n && keys[q] == target; ++q) {
        const uint32_t r = vals[q];
        found[side] = 1;
        if (side == 0) {
          const int64_t t = a.te[r] - o;
          prod_end = t > prod_end ? t : prod_end;
        } else {
          const int64_t t = a.ts[r] - o;
          cons_start = t < cons_start ? t : cons_start;
        }
      }
    }
    a.edge_status[e] = (found[0] ? 0 : 1) | (found[1] ? 0 : 2);
    a.edge_wait[e] = (found[0] && found[1]) ? (int64_t)((uint64_t)cons_start - (uint64_t)prod_end) : I64MIN;
  }
}

static JoinArgs join_args(Ctx& c) {
  JoinArgs a;
  a.k[0] = c.sJ.k[0];
  a.k[1] = c.sJ.k[1];
  a.v[0] = c.sJ.v[0];
  a.v[1] = c.sJ.v[1];
  a.ts = c.ev.ts;
  a.te = c.ev.te;
  a.off = c.p.clock_offset;
  a.ds = c.ds;
  a.cnt = c.o.counters;
  a.link = c.o.link;
  a.aux = c.o.aux;
  a.lat_hist = c.o.lat_hist;
  a.lk_first = c.lk_first;
  a.lk_last = c.lk_last;
  a.lk_sum = c.lk_sum;
  a.contain = c.contain;
  a.edges = c.p.edges;
  a.n_edges = c.p.n_edges;
  a.P = c.P;
  a.edge_wait = c.o.edge_wait;
  a.edge_status = c.o.edge_status;
  a.tab = c.jt_tab;
  a.own = c.jt_own;
  a.multi = c.jt_multi;
  a.kmax = c.jt_kmax;
  a.kmin = c.jt_kmin;
  a.cap = c.jt_cap;
  a.k_rows = c.k_rows;
  return a;
}

// The correlation-table join (no-ops unless the plan chose it); it needs only
// prep's lists, so it can run beside the sorts.
void launch_join_table(Ctx& c) {
  if (c.P > JT_PROCS) return;
  JoinArgs a = join_args(c);
  const int64_t cgrid = std::min<int64_t>(std::max<int64_t>(cdiv(c.jt_cap, 256 * 8), 1), 4096);
  auto tgrid = [&](int it) { return dim3((unsigned)std::max<int64_t>(cdiv(c.sJ.n_max, 256 * it), 1)); };
  hipLaunchKernelGGL(k_jt_clear, dim3((unsigned)cgrid), dim3(256), 0, c.st, a);
  hipLaunchKernelGGL(k_jt_store<JT_IT_STORE>, tgrid(JT_IT_STORE), dim3(256), 0, c.st, a);
  hipLaunchKernelGGL(k_jt_check<JT_IT_CHECK>, tgrid(JT_IT_CHECK), dim3(256), 0, c.st, a);
  hipLaunchKernelGGL(k_jt_fix<JT_IT_FIX>, tgrid(JT_IT_FIX), dim3(256), 0, c.st, a);
  hipLaunchKernelGGL(k_jt_kernel<JT_IT_KERNEL>, tgrid(JT_IT_KERNEL), dim3(256), 0, c.st, a);
}

// The sort-merge join (a no-op when the table did the join); after the sorts.
void launch_join(Ctx& c) {
  JoinArgs a = join_args(c);
  const int64_t grid = std::max<int64_t>(cdiv(c.sJ.n_max, 256), 1);
  hipLaunchKernelGGL(k_join, dim3((unsigned)grid), dim3(256), 0, c.st, a);
}


void launch_edges(Ctx& c) {
  if (c.p.n_edges <= 0) return;
  JoinArgs a = join_args(c);
  const int grid = (int)std::min<int64_t>(cdiv(c.p.n_edges, 256), 1024);
  hipLaunchKernelGGL(k_edges, dim3(grid), dim3(256), 0, c.st, a);
}

}  // namespace hx
