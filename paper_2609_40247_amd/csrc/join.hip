// Launch <-> kernel join and cross-process waits.
//
// The correlation id associates a submission with its device activity
// (Section 5.2); kernel composition is recovered from these call-to-kernel
// links (Section 6.1), and a graph launch may own many kernels.  Launches and
// kernels are sorted by (pid, corr, is_kernel), so each id is one run with
// its launches first: a kernel's launch is the head of its run (the smallest
// row, the sort being stable), extra launches are duplicates.  Run bounds are
// found by galloping searches, which cost O(log run length).  The latency is
// the kernel start minus the launch start (the "CPU submission time" of the
// operator figure) binned by floor(log2)+1.  Dependency edges (panel
// "Cross-process blocking") are binary searches into the same sorted runs.
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
  const int64_t n = a.ds->nJ;
  const int par = (int)a.ds->sort_parity[1];
  const uint64_t* keys = a.k[par];
  const uint32_t* vals = a.v[par];
  const int64_t i = (int64_t)blockIdx.x * 256 + tid;
  uint32_t c[JC_N] = {0, 0, 0, 0, 0, 0};
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
        if (a.contain) {
          const int32_t op = a.link[lrow];
          a.aux[row] = op;
          if (op < 0) ++c[JC_UNATTR];
        } else {
          a.aux[row] = -1;
        }
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

__global__ __launch_bounds__(256) void k_edges(JoinArgs a) {
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
  return a;
}

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
