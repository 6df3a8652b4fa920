// Launch <-> kernel join and cross-process waits.
//
// The correlation id associates a submission with its device activity
// (Section 5.2); kernel composition is recovered from these call-to-kernel
// links (Section 6.1), and a graph launch may own many kernels.  A kernel
// joins the admitted launch with its (pid, corr) and the smallest row;
// further launches with that id are duplicates.  The latency is the kernel
// start minus the launch start (the host submission time of the operator
// panel) binned by floor(log2)+1.  Dependency edges (panel "Cross-process
// blocking") look their two ids up in the same table.
//
// The join is a table of (pid, corr) slots, each with a launch word and a
// kernel word, built with plain stores: bulk global atomics are slow on this
// GPU, and in real traces nearly every id has one launch and one kernel.
// Slots are dense (process base + id - the process's smallest id) when the
// call has at most JT_PROCS processes whose ids span at most two slots per
// row, as ids that every API call takes in turn do; otherwise hashed, by
// linear probing over a power-of-two table in which the first row of a key
// claims the slot with a compare-and-swap.  The table is emptied by the
// histogram kernel, which takes the plan.
//
//   store:   every launch writes its row to its slot's launch word, every
//            kernel to the kernel word (one writer of each wins);
//   resolve: a launch that won its word is the slot's launch for now; it
//            joins the kernel that won the kernel word (the usual case: one
//            launch, one kernel, all plain stores).  A launch that lost is a
//            duplicate, a kernel that lost shares its slot with others: both
//            go to a short fix-up list;
//   dups:    duplicates put the smallest row into the launch word (atomics);
//   fix:     a duplicate that ends up in the word takes the slot's kernel
//            over from the launch that held it, and every kernel of the
//            list joins the final launch with atomics.
// The fix-up passes are short grids that leave at once when the list is
// empty.
#include "internal.hpp"

namespace hx {

struct JoinArgs {
  const uint64_t* jkey;  // prep's join list: launches and kernels in row order
  const uint32_t* jrow;
  uint32_t* jslot;       // [n] each entry's slot (hashed slots only)
  const int64_t* ts;
  const int64_t* te;
  const int64_t* corr;
  const int32_t* pid;
  const int64_t* off;
  DevState* ds;
  int32_t* link;  // may be NULL (no containment, output not wanted)
  int32_t* aux;   // may be NULL (likewise)
  int64_t* lk_first;
  int64_t* lk_last;
  int64_t* lk_sum;
  bool contain;
  const herschel_edge* edges;
  int64_t n_edges;
  int P;
  int64_t* edge_wait;
  int32_t* edge_status;
  uint32_t* L;     // [cap] launch word per slot
  uint32_t* K;     // [cap] kernel word per slot
  uint32_t* C;     // [cap] claiming row per slot (hashed slots)
  int64_t* kmax;   // [cap] latest kernel end per slot (edges only)
  int64_t* kmin;   // [cap] earliest kernel start per slot (edges only)
  uint64_t hmask;  // hashed table size - 1 (a power of two)
  uint32_t* fix;   // [fix_cap][3]: slot, row | FIX_DUP, launch row seen by the resolve pass
  int64_t fix_cap;
};

constexpr uint32_t FIX_DUP = 1u << 31;  // the entry is a duplicate launch (else a kernel sharing its slot)

// Hashed slot of (key, pid, corr): probe from the key's hash; an empty slot
// is claimed with a compare-and-swap (a claimed slot never changes within a
// call, so a stale read of an empty slot only sends the thread to the
// compare-and-swap, which returns the current claimer); a claimed slot is
// this key's when its claiming row has the same process and id.
__device__ __forceinline__ int64_t jt_claim(const JoinArgs& a, uint64_t key, uint32_t row, int32_t pid,
                                            int64_t corr) {
  uint64_t s = jt_hash(key) & a.hmask;
  for (uint64_t probe = 0; probe <= a.hmask; ++probe) {
    uint32_t c = a.C[s];
    if (c == JT_EMPTY) {
      c = atomicCAS(&a.C[s], JT_EMPTY, row);
      if (c == JT_EMPTY) return (int64_t)s;
    }
    if (a.pid[c] == pid && a.corr[c] == corr) return (int64_t)s;
    s = (s + 1) & a.hmask;
  }
  set_status(a.ds, DS_CAPACITY);  // unreachable: the table has twice the rows' slots
  return -1;
}

// Slot of (pid, corr) without claiming; -1 when no admitted launch or kernel
// has that id.
__device__ __forceinline__ int64_t jt_find(const JoinArgs& a, int32_t pid, int64_t corr) {
  if (pid < 0 || pid >= a.P) return -1;
  const uint64_t key = ((uint64_t)pid << JK_PID_SHIFT) | (((uint64_t)corr & JK_CORR_MASK) << 1);
  if (a.ds->join_direct) {
    if (!((a.ds->jt_present >> pid) & 1)) return -1;
    const uint64_t rel = (uint64_t)corr - (uint64_t)a.ds->jt_cmin[pid];
    const int64_t lim = (pid + 1 < a.P ? a.ds->jt_base[pid + 1] : a.ds->jt_slots) - a.ds->jt_base[pid];
    if (rel >= (uint64_t)lim) return -1;
    return a.ds->jt_base[pid] + (int64_t)rel;
  }
  uint64_t s = jt_hash(key) & a.hmask;
  for (uint64_t probe = 0; probe <= a.hmask; ++probe) {
    const uint32_t c = a.C[s];
    if (c == JT_EMPTY) return -1;
    if (a.pid[c] == pid && a.corr[c] == corr) return (int64_t)s;
    s = (s + 1) & a.hmask;
  }
  return -1;
}

// Adds each thread's counts (signed: the fix-up moves latencies between
// bins) to the workgroup's and then to one of the accumulator copies.
__device__ __forceinline__ void jt_flush(const JoinArgs& a, int64_t (&c)[JC_N], unsigned long long* s_c,
                                         unsigned long long* s_h) {
#pragma unroll
  for (int q = 0; q < JC_N; ++q) {
    const uint64_t w = wave_sum_u64((uint64_t)c[q]);
    if (lane_id() == 0 && w) atomicAdd(&s_c[q], (unsigned long long)w);
  }
  __syncthreads();
  unsigned long long* acc = &a.ds->join_acc[blockIdx.x % JOIN_COPIES][0];
  if (threadIdx.x < JC_N && s_c[threadIdx.x]) atomicAdd(&acc[threadIdx.x], s_c[threadIdx.x]);
  if (s_h && threadIdx.x < 64 && s_h[threadIdx.x]) atomicAdd(&acc[JC_N + threadIdx.x], s_h[threadIdx.x]);
}

__device__ __forceinline__ int lat_bin(int64_t x) { return x <= 0 ? 0 : bits_of((uint64_t)x); }

// The passes give each thread IT entries (striped over the workgroup) and
// issue each round of their loads together: a pass is a short chain of
// dependent loads, and batching entries per thread keeps the number of waves
// the chip must cycle through low.
constexpr int JT_IT_STORE = 4, JT_IT_RESOLVE = 6;

// Pass 1: every launch writes its row to its slot's launch word, every kernel
// to the kernel word (plain stores; one writer of each wins).
template <int IT>
__global__ __launch_bounds__(256) void k_jt_store(JoinArgs a) {
  const int64_t n = a.ds->nJ;
  if (n == 0) return;
  const bool dense = a.ds->join_direct != 0;
  const int64_t cap = a.ds->jt_slots;
  const int64_t i0 = (int64_t)blockIdx.x * (256 * IT) + threadIdx.x;
  uint64_t key[IT];
  uint32_t row[IT];
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const int64_t i = i0 + u * 256;
    const int64_t ic = i < n ? i : n - 1;  // clamped: the loads stay in flight together
    key[u] = a.jkey[ic];
    row[u] = a.jrow[ic];
  }
  if (dense) {
#pragma unroll
    for (int u = 0; u < IT; ++u) {
      if (i0 + u * 256 >= n) continue;
      const int64_t slot = jt_dense_slot(a.ds, key[u]);
      if (!in_bounds(a.ds, slot, cap)) continue;
      ((key[u] & 1) ? a.K : a.L)[slot] = row[u];
    }
    return;
  }
  // hashed: the entries' own process and full id, then the probes
  int32_t pd[IT];
  int64_t cr[IT];
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    pd[u] = a.pid[row[u]];
    cr[u] = a.corr[row[u]];
  }
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const int64_t i = i0 + u * 256;
    if (i >= n) continue;
    const int64_t slot = jt_claim(a, key[u], row[u], pd[u], cr[u]);
    if (slot < 0) continue;
    a.jslot[i] = (uint32_t)slot;
    ((key[u] & 1) ? a.K : a.L)[slot] = row[u];
  }
}

// Appends (slot, row | flag, w) to the fix-up list: one atomic per wave.
__device__ __forceinline__ void fix_append(const JoinArgs& a, bool want, int64_t slot, uint32_t rowf, uint32_t w) {
  const uint64_t b = ballot(want);
  if (!b) return;
  const int leader = __ffsll((unsigned long long)b) - 1;
  uint32_t base = 0;
  if (lane_id() == leader) base = atomicAdd(&a.ds->jt_nfix, (uint32_t)popc(b));
  base = __shfl(base, leader, WAVE);
  if (!want) return;
  const int64_t at = (int64_t)base + popc(b & lanemask_lt());
  if (!in_bounds(a.ds, at, a.fix_cap)) return;
  a.fix[3 * at + 0] = (uint32_t)slot;
  a.fix[3 * at + 1] = rowf;
  a.fix[3 * at + 2] = w;
}

// Pass 2.  A launch that holds its slot's launch word joins the kernel that
// holds the kernel word: it writes the kernel's link, the latency, its own
// kernel count (1) and kernel aggregates.  A launch that lost is a duplicate
// (count 0; listed).  A kernel that holds the kernel word records its times
// for the edges, or, with no launch in the slot, is unmatched; a kernel that
// lost shares the slot (listed).
template <int IT>
__global__ __launch_bounds__(256) void k_jt_resolve(JoinArgs a) {
  __shared__ unsigned long long s_c[JC_N];
  __shared__ unsigned long long s_h[64];
  const int tid = threadIdx.x;
  if (tid < JC_N) s_c[tid] = 0;
  if (tid < 64) s_h[tid] = 0;
  __syncthreads();
  const int64_t n = a.ds->nJ;
  if (n == 0) return;
  const bool dense = a.ds->join_direct != 0;
  const int64_t cap = a.ds->jt_slots;
  const int64_t i0 = (int64_t)blockIdx.x * (256 * IT) + tid;
  int64_t c[JC_N] = {};
  // round 1: the entries
  uint64_t key[IT];
  uint32_t row[IT], hs[IT];
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const int64_t i = i0 + u * 256;
    const int64_t ic = i < n ? i : n - 1;
    key[u] = a.jkey[ic];
    row[u] = a.jrow[ic];
    hs[u] = dense ? 0u : a.jslot[ic];
  }
  // round 2: the slot's words
  int64_t slot[IT];
  uint32_t lw[IT], kw[IT];
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const bool live = i0 + u * 256 < n;
    slot[u] = dense ? jt_dense_slot(a.ds, key[u]) : (int64_t)hs[u];
    if (!live || !in_bounds(a.ds, slot[u], cap)) slot[u] = -1;
    const int64_t sc = slot[u] >= 0 ? slot[u] : 0;
    lw[u] = a.L[sc];
    kw[u] = a.K[sc];
  }
  // round 3: times (a launch that joins a kernel: the kernel's start and end
  // and its own start; a kernel with edges: its start and end)
  int64_t t0[IT], t1[IT], t2[IT];
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const bool kern = (key[u] & 1) != 0;
    const bool joins = !kern && slot[u] >= 0 && lw[u] == row[u] && kw[u] != JT_EMPTY;
    const uint32_t kr = kern ? row[u] : joins ? kw[u] : 0u;
    t0[u] = a.ts[kr];
    t1[u] = a.te[kr];
    t2[u] = a.ts[joins ? row[u] : 0u];
  }
#pragma unroll
  for (int u = 0; u < IT; ++u) {
    const bool kern = (key[u] & 1) != 0;
    const bool live = slot[u] >= 0;
    const int64_t o = a.off ? a.off[(int32_t)(key[u] >> JK_PID_SHIFT)] : 0;
    if (live && !kern) {
      if (lw[u] != row[u]) {  // a duplicate: no kernels (unless the fix-up hands it the slot's)
        if (a.aux) a.aux[row[u]] = 0;
        ++c[JC_DUP];
      } else if (kw[u] == JT_EMPTY) {
        if (a.aux) a.aux[row[u]] = 0;
      } else {
        const uint32_t kr = kw[u];
        if (a.link) a.link[kr] = (int32_t)row[u];
        if (a.aux) {
          a.aux[kr] = -1;  // the kernel's op comes later (the name pass)
          a.aux[row[u]] = 1;
        }
        ++c[JC_MATCHED];
        ++c[JC_MLAUNCH];
        const int64_t x = t0[u] - t2[u];  // same process: the offset cancels
        if (x < 0) ++c[JC_NEG];
        atomicAdd(&s_h[lat_bin(x)], 1ull);
        if (a.contain) {
          a.lk_first[row[u]] = t0[u] - o;
          a.lk_last[row[u]] = t1[u] - o;
          a.lk_sum[row[u]] = t1[u] - t0[u];
        }
      }
    }
    if (live && kern && kw[u] == row[u]) {
      if (a.kmax) {
        a.kmax[slot[u]] = t1[u] - o;
        a.kmin[slot[u]] = t0[u] - o;
      }
      if (lw[u] == JT_EMPTY) {
        if (a.link) a.link[row[u]] = -1;
        if (a.aux) a.aux[row[u]] = -1;
        ++c[JC_UNM_K];
      }
    }
    const bool dup = live && !kern && lw[u] != row[u];
    const bool shared = live && kern && kw[u] != row[u];
    fix_append(a, dup || shared, slot[u], row[u] | (dup ? FIX_DUP : 0u), lw[u]);
  }
  jt_flush(a, c, s_c, s_h);
}

constexpr int JT_FIX_BLOCKS = 256;

// Fix-up 1: duplicates put the smallest row into the launch word, and start
// their kernel aggregates at the identities (the one that ends up in the
// word receives its kernels with atomics).
__global__ __launch_bounds__(256) void k_jt_dups(JoinArgs a) {
  const int64_t nf = min((int64_t)a.ds->jt_nfix, a.fix_cap);
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nf; i += (int64_t)gridDim.x * 256) {
    const uint32_t rf = a.fix[3 * i + 1];
    if (!(rf & FIX_DUP)) continue;
    const uint32_t slot = a.fix[3 * i], row = rf & ~FIX_DUP;
    atomicMin(&a.L[slot], row);
    if (a.contain) {
      a.lk_first[row] = I64MAX;
      a.lk_last[row] = I64MIN;
      a.lk_sum[row] = 0;
    }
  }
}

// Fix-up 2: the duplicate now in its slot's launch word takes over the slot's
// kernel from the launch that joined it in the resolve pass (link, latency
// bin, kernel count and aggregates move); every kernel that shares a slot
// joins the slot's final launch with atomics (or is unmatched) and adds its
// times to the slot's edge extremes.
__global__ __launch_bounds__(256) void k_jt_fix(JoinArgs a) {
  __shared__ unsigned long long s_c[JC_N];
  __shared__ unsigned long long s_h[64];
  const int tid = threadIdx.x;
  if (tid < JC_N) s_c[tid] = 0;
  if (tid < 64) s_h[tid] = 0;
  __syncthreads();
  const int64_t nf = min((int64_t)a.ds->jt_nfix, a.fix_cap);
  if ((int64_t)blockIdx.x * 256 >= nf) return;  // uniform: no entry for this workgroup
  int64_t c[JC_N] = {};
  for (int64_t i = (int64_t)blockIdx.x * 256 + tid; i < nf; i += (int64_t)gridDim.x * 256) {
    const uint32_t slot = a.fix[3 * i], rf = a.fix[3 * i + 1], w = a.fix[3 * i + 2];
    const uint32_t row = rf & ~FIX_DUP;
    const uint32_t l = a.L[slot];
    if (rf & FIX_DUP) {
      const uint32_t kr = a.K[slot];
      if (l != row || kr == JT_EMPTY) continue;
      // row < w: the kernel of the resolve pass moves from launch w to row
      const int64_t o = a.off ? a.off[a.pid[row]] : 0;
      const int64_t ks = a.ts[kr], ke = a.te[kr];
      const int64_t x_old = ks - a.ts[w], x_new = ks - a.ts[row];
      if (a.link) a.link[kr] = (int32_t)row;
      if (a.aux) {
        a.aux[w] = 0;
        atomicAdd(&a.aux[row], 1);
      }
      atomicAdd(&s_h[lat_bin(x_old)], ~0ull);  // minus one
      atomicAdd(&s_h[lat_bin(x_new)], 1ull);
      c[JC_NEG] += (x_new < 0 ? 1 : 0) - (x_old < 0 ? 1 : 0);
      if (a.contain) {
        atomicMin((long long*)&a.lk_first[row], (long long)(ks - o));
        atomicMax((long long*)&a.lk_last[row], (long long)(ke - o));
        atomicAdd((unsigned long long*)&a.lk_sum[row], (unsigned long long)(ke - ks));
      }
      continue;
    }
    // a kernel that shares its slot
    const int64_t o = a.off ? a.off[a.pid[row]] : 0;
    const int64_t ks = a.ts[row], ke = a.te[row];
    if (a.kmax) {
      atomicMax((long long*)&a.kmax[slot], (long long)(ke - o));
      atomicMin((long long*)&a.kmin[slot], (long long)(ks - o));
    }
    if (l == JT_EMPTY) {
      if (a.link) a.link[row] = -1;
      if (a.aux) a.aux[row] = -1;
      ++c[JC_UNM_K];
      continue;
    }
    if (a.link) a.link[row] = (int32_t)l;
    if (a.aux) {
      a.aux[row] = -1;
      atomicAdd(&a.aux[l], 1);
    }
    ++c[JC_MATCHED];
    const int64_t x = ks - a.ts[l];
    if (x < 0) ++c[JC_NEG];
    atomicAdd(&s_h[lat_bin(x)], 1ull);
    if (a.contain) {
      atomicMin((long long*)&a.lk_first[l], (long long)(ks - o));
      atomicMax((long long*)&a.lk_last[l], (long long)(ke - o));
      atomicAdd((unsigned long long*)&a.lk_sum[l], (unsigned long long)(ke - ks));
    }
  }
  jt_flush(a, c, s_c, s_h);
}

// Dependency waits: each edge's producer and consumer ids looked up in the
// table; the slot's kernel extremes give the producer's last end and the
// consumer's first start.
__global__ __launch_bounds__(256) void k_edges(JoinArgs a) {
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < a.n_edges; e += (int64_t)gridDim.x * 256) {
    const herschel_edge ed = a.edges[e];
    int found[2] = {0, 0};
    int64_t prod_end = I64MIN, cons_start = I64MAX;
    for (int side = 0; side < 2; ++side) {
      const int64_t slot = side == 0 ? jt_find(a, ed.prod_pid, ed.prod_corr) : jt_find(a, ed.cons_pid, ed.cons_corr);
      if (slot < 0 || a.K[slot] == JT_EMPTY) continue;
      found[side] = 1;
      if (side == 0)
        prod_end = a.kmax[slot];
      else
        cons_start = a.kmin[slot];
    }
    if (a.edge_status) a.edge_status[e] = (found[0] ? 0 : 1) | (found[1] ? 0 : 2);
    if (a.edge_wait)
      a.edge_wait[e] = (found[0] && found[1]) ? (int64_t)((uint64_t)cons_start - (uint64_t)prod_end) : I64MIN;
  }
}

static JoinArgs join_args(Ctx& c) {
  JoinArgs a;
  a.jkey = c.jkey;
  a.jrow = c.jrow;
  a.jslot = c.jslot;
  a.ts = c.ev.ts;
  a.te = c.ev.te;
  a.corr = c.ev.corr;
  a.pid = c.ev.pid;
  a.off = c.p.clock_offset;
  a.ds = c.ds;
  a.link = c.o.link;
  a.aux = c.o.aux;
  a.lk_first = c.lk_first;
  a.lk_last = c.lk_last;
  a.lk_sum = c.lk_sum;
  a.contain = c.contain;
  a.edges = c.p.edges;
  a.n_edges = c.p.n_edges;
  a.P = c.P;
  a.edge_wait = c.o.edge_wait;
  a.edge_status = c.o.edge_status;
  a.L = c.jt_L;
  a.K = c.jt_K;
  a.C = c.jt_C;
  a.kmax = c.jt_kmax;
  a.kmin = c.jt_kmin;
  a.hmask = (uint64_t)c.jt_hsize - 1;
  a.fix = c.jt_fix;
  a.fix_cap = c.jt_fix_cap;
  return a;
}

// The join after the plan and the emptied table (both from the histogram
// kernel): store, resolve and the two fix-up passes.
void launch_join_table(Ctx& c) {
  if (c.n == 0) return;
  JoinArgs a = join_args(c);
  auto grid = [&](int it) { return dim3((unsigned)std::max<int64_t>(cdiv(c.n, 256 * it), 1)); };
  hipLaunchKernelGGL(k_jt_store<JT_IT_STORE>, grid(JT_IT_STORE), dim3(256), 0, c.st, a);
  hipLaunchKernelGGL(k_jt_resolve<JT_IT_RESOLVE>, grid(JT_IT_RESOLVE), dim3(256), 0, c.st, a);
  const unsigned fb = (unsigned)std::min<int64_t>(std::max<int64_t>(cdiv(c.n, 256), 1), JT_FIX_BLOCKS);
  hipLaunchKernelGGL(k_jt_dups, dim3(fb), dim3(256), 0, c.st, a);
  hipLaunchKernelGGL(k_jt_fix, dim3(fb), dim3(256), 0, c.st, a);
}

void launch_edges(Ctx& c) {
  if (c.p.n_edges <= 0) return;
  JoinArgs a = join_args(c);
  const int grid = (int)std::min<int64_t>(cdiv(c.p.n_edges, 256), 1024);
  hipLaunchKernelGGL(k_edges, dim3(grid), dim3(256), 0, c.st, a);
}

}  // namespace hx
