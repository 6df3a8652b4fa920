// Graph replay separation (Section 6.1, "Operator execution and
// efficiency": replaying a captured graph hides the operator calls; graph
// identities and launch correlations separate the replays).
//
// A replay is an admitted launch and the kernels the join gave it; its span
// (first kernel start, last kernel end) is the join's per-launch aggregate,
// reported for every admitted launch.  Each kernel's graph node (the
// caller's dense id of a node of a captured graph) names the same operator
// in every replay: per node, over admitted kernels joined to a launch, the
// count, sum, minimum and maximum of the duration, and the summed offset of
// the kernel's start from its replay's first start.
//
// One pass over the admitted kernels (row order) keeps a private table of
// all nodes per workgroup in LDS (40 bytes a node) and writes it out whole;
// a second kernel folds the tables node by node into the outputs.  More
// nodes than LDS holds go to the outputs by global atomics.  The same first
// pass also writes the launches' spans from the join list.
#include "internal.hpp"

namespace hx {

constexpr int GR_THREADS = 512;
constexpr int GR_LDS_NODES = 1024;  // 40 KB of LDS
constexpr int GR_STATS = 5;         // count, sum, min, max, offset
constexpr int GR_MAX_BLOCKS = 256;
constexpr int GF_ROWS = 16;         // rows of the fold's grid

struct GraphArgs {
  DevState* ds;
  const uint32_t* k_rows;  // admitted kernels, row order
  const uint64_t* jkey;    // join list: admitted launches and kernels, row order
  const uint32_t* jrow;
  const int32_t* node;
  const int32_t* link;
  const int32_t* aux;
  const int32_t* pid;
  const int64_t* ts;
  const int64_t* te;
  const int64_t* off;
  const int64_t* lk_first;
  const int64_t* lk_last;
  int NG;
  bool lds;
  uint64_t* part;  // [blocks][NG][GR_STATS]
  int blocks;
  int64_t* o_first;
  int64_t* o_last;
  int64_t* o_count;
  int64_t* o_sum;
  int64_t* o_min;
  int64_t* o_max;
  int64_t* o_off;
};

__global__ __launch_bounds__(GR_THREADS) void k_graph(GraphArgs a) {
  extern __shared__ unsigned long long gtab[];  // [NG][GR_STATS]
  const int tid = threadIdx.x;
  if (a.lds) {
    for (int q = tid; q < a.NG; q += GR_THREADS) {
      gtab[q * GR_STATS + 0] = 0;
      gtab[q * GR_STATS + 1] = 0;
      gtab[q * GR_STATS + 2] = (unsigned long long)I64MAX;
      gtab[q * GR_STATS + 3] = (unsigned long long)I64MIN;
      gtab[q * GR_STATS + 4] = 0;
    }
    __syncthreads();
  }
  const int64_t stride = (int64_t)gridDim.x * GR_THREADS;
  const int64_t nk = a.ds->nK;
  for (int64_t i = (int64_t)blockIdx.x * GR_THREADS + tid; i < nk; i += stride) {
    const uint32_t r = a.k_rows[i];
    const int32_t q = a.node[r];
    const int32_t L = a.link[r];
    if (q < 0 || L < 0) continue;
    const int64_t o = a.off ? a.off[a.pid[r]] : 0;
    const int64_t s = a.ts[r] - o;
    const int64_t d = a.te[r] - a.ts[r];
    const int64_t rel = s - a.lk_first[L];
    if (a.lds) {
      atomicAdd(&gtab[q * GR_STATS + 0], 1ull);
      atomicAdd(&gtab[q * GR_STATS + 1], (unsigned long long)d);
      atomicMin((long long*)&gtab[q * GR_STATS + 2], (long long)d);
      atomicMax((long long*)&gtab[q * GR_STATS + 3], (long long)d);
      atomicAdd(&gtab[q * GR_STATS + 4], (unsigned long long)rel);
    } else {
      if (a.o_count) atomicAdd((unsigned long long*)&a.o_count[q], 1ull);
      if (a.o_sum) atomicAdd((unsigned long long*)&a.o_sum[q], (unsigned long long)d);
      if (a.o_min) atomicMin((long long*)&a.o_min[q], (long long)d);
      if (a.o_max) atomicMax((long long*)&a.o_max[q], (long long)d);
      if (a.o_off) atomicAdd((unsigned long long*)&a.o_off[q], (unsigned long long)rel);
    }
  }
  // the launches' spans
  const int64_t nj = a.ds->nJ;
  if (a.o_first || a.o_last)
    for (int64_t i = (int64_t)blockIdx.x * GR_THREADS + tid; i < nj; i += stride) {
      if (a.jkey[i] & 1) continue;  // a kernel
      const uint32_t r = a.jrow[i];
      const bool any = a.aux[r] > 0;
      if (a.o_first) a.o_first[r] = any ? a.lk_first[r] : I64MAX;
      if (a.o_last) a.o_last[r] = any ? a.lk_last[r] : I64MIN;
    }
  if (!a.lds) return;
  __syncthreads();
  uint64_t* out = a.part + (int64_t)blockIdx.x * a.NG * GR_STATS;
  for (int i = tid; i < a.NG * GR_STATS; i += GR_THREADS) out[i] = gtab[i];
}

// One thread per (node, statistic) and row of the grid: row g folds the
// tables g, g + rows, ... (16 loads in flight) and combines its result into
// the output with one atomic (the outputs start as the identities).
__global__ __launch_bounds__(256) void k_graph_fold(GraphArgs a) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t nv = (int64_t)a.NG * GR_STATS;
  if (t >= nv) return;
  const int q = (int)(t / GR_STATS), st = (int)(t % GR_STATS);
  int64_t* const dst[GR_STATS] = {a.o_count, a.o_sum, a.o_min, a.o_max, a.o_off};
  if (!dst[st]) return;
  uint64_t acc = st == 2 ? (uint64_t)I64MAX : st == 3 ? (uint64_t)I64MIN : 0;
  for (int b0 = blockIdx.y; b0 < a.blocks; b0 += 16 * (int)gridDim.y) {
    uint64_t v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int b = b0 + i * (int)gridDim.y;
      v[i] = a.part[(int64_t)(b < a.blocks ? b : blockIdx.y) * nv + t];
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (b0 + i * (int)gridDim.y >= a.blocks) break;
      if (st == 2)
        acc = (int64_t)v[i] < (int64_t)acc ? v[i] : acc;
      else if (st == 3)
        acc = (int64_t)v[i] > (int64_t)acc ? v[i] : acc;
      else
        acc += v[i];
    }
  }
  if (st == 2) {
    if ((int64_t)acc != I64MAX) atomicMin((long long*)&dst[st][q], (long long)acc);
  } else if (st == 3) {
    if ((int64_t)acc != I64MIN) atomicMax((long long*)&dst[st][q], (long long)acc);
  } else if (acc) {
    atomicAdd((unsigned long long*)&dst[st][q], (unsigned long long)acc);
  }
}

bool graph_uses_tables(int NG) { return NG <= GR_LDS_NODES; }

int graph_block_count(int64_t n_max, int NG) {
  if (!graph_uses_tables(NG)) return (int)std::min<int64_t>(std::max<int64_t>(cdiv(n_max, 4096), 1), 1024);
  return (int)std::min<int64_t>(std::max<int64_t>(cdiv(n_max, 8192), 1), GR_MAX_BLOCKS);
}

static GraphArgs graph_args(Ctx& c) {
  GraphArgs a;
  a.ds = c.ds;
  a.k_rows = c.k_rows;
  a.jkey = c.jkey;
  a.jrow = c.jrow;
  a.node = c.ev.graph_node;
  a.link = c.o.link;
  a.aux = c.o.aux;
  a.pid = c.ev.pid;
  a.ts = c.ev.ts;
  a.te = c.ev.te;
  a.off = c.p.clock_offset;
  a.lk_first = c.lk_first;
  a.lk_last = c.lk_last;
  a.NG = c.NG;
  a.lds = graph_uses_tables(c.NG);
  a.part = c.graph_part;
  a.blocks = c.graph_blocks;
  a.o_first = c.o.launch_first;
  a.o_last = c.o.launch_last;
  a.o_count = c.o.gn_count;
  a.o_sum = c.o.gn_sum;
  a.o_min = c.o.gn_min;
  a.o_max = c.o.gn_max;
  a.o_off = c.o.gn_offset;
  return a;
}

void launch_graph(Ctx& c) {
  GraphArgs a = graph_args(c);
  const size_t lds = a.lds ? (size_t)c.NG * GR_STATS * 8 : 0;
  hipLaunchKernelGGL(k_graph, dim3((unsigned)c.graph_blocks), dim3(GR_THREADS), lds, c.st, a);
  if (a.lds) {
    const unsigned gy = (unsigned)std::min(GF_ROWS, std::max(c.graph_blocks, 1));
    hipLaunchKernelGGL(k_graph_fold, dim3((unsigned)cdiv((int64_t)c.NG * GR_STATS, 256), gy), dim3(256), 0, c.st,
                       a);
  }
}

}  // namespace hx
