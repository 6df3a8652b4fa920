// Per kernel-name aggregates: count, sum, min and max of the unclipped
// kernel duration over all admitted kernels (Section 6.1 measures kernel
// durations; grouping by kernel name is the per-name view of the same
// records).  With containment a separate pass gives each matched kernel the
// op of its launch (kernel composition, Section 6.1) and counts the matched
// kernels whose launch has no op: it needs the launches' ops, the tables do
// not, so the tables are built while the containment query still runs.
//
// Each workgroup keeps a private table of all names in LDS (32 bytes per
// name) while it streams a slice of the admitted kernels, then writes the
// table out whole; a second kernel folds the tables name by name.  No global
// atomics touch the hot names of a Zipf-distributed name mix.  Name counts
// beyond the LDS budget fall back to global atomics.
#include "internal.hpp"

namespace hx {

constexpr int NM_THREADS = 512;
constexpr int NM_LDS_NAMES = 4096;  // 128 KB of LDS
constexpr int NM_BATCH = 8;
static_assert(NM_LDS_NAMES * 32 <= 160 * 1024, "the per-block name table must fit the LDS of a CU");

struct NamesArgs {
  const uint32_t* rows;  // admitted kernels' rows (prep's own copy: the sorts reuse their buffers)
  const int32_t* name;
  const int64_t* ts;
  const int64_t* te;
  DevState* ds;
  int NN;
  uint64_t* part;  // [blocks][NN][4]
  int blocks;
  int64_t* count;
  int64_t* sum;
  int64_t* mn;
  int64_t* mx;
  bool tables;  // some name output is wanted
  // kernel -> op (with containment): the op of the kernel's launch
  const int32_t* link;
  int32_t* aux;
};

__global__ __launch_bounds__(NM_THREADS) void k_names_partial(NamesArgs a) {
  extern __shared__ unsigned long long tab[];  // [NN][4]: count, sum, min, max
  const int tid = threadIdx.x;
  const bool lds = a.tables && a.NN <= NM_LDS_NAMES;
  if (lds) {
    for (int q = tid; q < a.NN; q += NM_THREADS) {
      tab[q * 4 + 0] = 0;
      tab[q * 4 + 1] = 0;
      tab[q * 4 + 2] = (unsigned long long)I64MAX;
      tab[q * 4 + 3] = (unsigned long long)I64MIN;
    }
    __syncthreads();
  }
  const int64_t n = a.ds->nK;
  const uint32_t* rows = a.rows;
  // NM_BATCH kernels per thread and round, each round of loads issued
  // together (positions past the end take the last kernel: clamped, not
  // branched on, and then skipped)
  const int64_t stride = (int64_t)gridDim.x * NM_THREADS;
  for (int64_t i0 = (int64_t)blockIdx.x * NM_THREADS + tid; i0 < n; i0 += NM_BATCH * stride) {
    uint32_t r[NM_BATCH];
#pragma unroll
    for (int u = 0; u < NM_BATCH; ++u) r[u] = rows[i0 + u * stride < n ? i0 + u * stride : n - 1];
    int32_t q[NM_BATCH];
    int64_t d[NM_BATCH];
#pragma unroll
    for (int u = 0; u < NM_BATCH; ++u) {
      const int32_t nm = a.name[r[u]];
      const int64_t e = a.te[r[u]], s = a.ts[r[u]];
      q[u] = i0 + u * stride < n ? nm : -1;
      d[u] = e - s;
    }
#pragma unroll
    for (int u = 0; u < NM_BATCH; ++u) {
      if (q[u] < 0) continue;
      if (lds) {
        atomicAdd(&tab[q[u] * 4 + 0], 1ull);
        atomicAdd(&tab[q[u] * 4 + 1], (unsigned long long)d[u]);
        atomicMin((long long*)&tab[q[u] * 4 + 2], (long long)d[u]);
        atomicMax((long long*)&tab[q[u] * 4 + 3], (long long)d[u]);
      } else {
        if (a.count) atomicAdd((unsigned long long*)&a.count[q[u]], 1ull);
        if (a.sum) atomicAdd((unsigned long long*)&a.sum[q[u]], (unsigned long long)d[u]);
        if (a.mn) atomicMin((long long*)&a.mn[q[u]], (long long)d[u]);
        if (a.mx) atomicMax((long long*)&a.mx[q[u]], (long long)d[u]);
      }
    }
  }
  if (!lds) return;
  __syncthreads();
  uint64_t* out = a.part + (int64_t)blockIdx.x * a.NN * 4;
  for (int i = tid; i < a.NN * 4; i += NM_THREADS) out[i] = tab[i];
}

// Kernel -> op: each matched kernel takes the op of its launch (the join
// gave the kernel its launch, the containment query the launch its op;
// unmatched kernels keep the join's -1).  KO_ITEMS kernels per thread, each
// round of loads issued together.
constexpr int KO_THREADS = 256;
constexpr int KO_ITEMS = 8;

__global__ __launch_bounds__(KO_THREADS) void k_kernel_ops(NamesArgs a) {
  const int64_t n = a.ds->nK;
  if (n == 0) return;
  const int64_t p0 = (int64_t)blockIdx.x * KO_THREADS * KO_ITEMS + threadIdx.x;
  if (p0 >= n) return;
  uint32_t r[KO_ITEMS];
#pragma unroll
  for (int u = 0; u < KO_ITEMS; ++u) {
    const int64_t p = p0 + u * KO_THREADS;
    r[u] = a.rows[p < n ? p : n - 1];
  }
  int32_t l[KO_ITEMS];
#pragma unroll
  for (int u = 0; u < KO_ITEMS; ++u) l[u] = a.link[r[u]];
  int32_t op[KO_ITEMS];
#pragma unroll
  for (int u = 0; u < KO_ITEMS; ++u) op[u] = a.link[l[u] >= 0 ? l[u] : 0];
  uint32_t unattr = 0;  // matched kernels whose launch has no op
#pragma unroll
  for (int u = 0; u < KO_ITEMS; ++u) {
    if (p0 + u * KO_THREADS >= n || l[u] < 0) continue;
    a.aux[r[u]] = op[u];
    if (op[u] < 0) ++unattr;
  }
  const uint64_t w = wave_sum_u64(unattr);
  if (lane_id() == 0 && w) atomicAdd(&a.ds->join_acc[blockIdx.x % JOIN_COPIES][JC_UNATTR], (unsigned long long)w);
}

// One thread per (name, statistic) and group of tables: group g folds the
// tables g, g + NR_GROUPS, ... with independent, coalesced loads
// (consecutive threads read consecutive words), 16 in flight, and combines
// its result into the output with one atomic (the outputs start as the
// identities, set by the init kernel).
constexpr int NR_GROUPS = 16;

__global__ __launch_bounds__(256) void k_names_reduce(NamesArgs a) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= (int64_t)a.NN * 4) return;
  const int q = (int)(t >> 2), stat = (int)(t & 3);
  int64_t* const dst[4] = {a.count, a.sum, a.mn, a.mx};
  if (!dst[stat]) return;  // that output is not wanted
  const int64_t stride = (int64_t)a.NN * 4;
  uint64_t acc = stat == 2 ? (uint64_t)I64MAX : stat == 3 ? (uint64_t)I64MIN : 0;
  for (int b0 = blockIdx.y; b0 < a.blocks; b0 += 16 * NR_GROUPS) {
    uint64_t v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int b = b0 + i * NR_GROUPS;
      v[i] = a.part[(int64_t)(b < a.blocks ? b : blockIdx.y) * stride + t];
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (b0 + i * NR_GROUPS >= a.blocks) break;
      if (stat < 2) acc += v[i];
      else if (stat == 2) acc = (int64_t)v[i] < (int64_t)acc ? v[i] : acc;
      else acc = (int64_t)v[i] > (int64_t)acc ? v[i] : acc;
    }
  }
  if (stat == 0) {
    if (acc) atomicAdd((unsigned long long*)&a.count[q], (unsigned long long)acc);
  } else if (stat == 1) {
    if (acc) atomicAdd((unsigned long long*)&a.sum[q], (unsigned long long)acc);
  } else if (stat == 2) {
    if ((int64_t)acc != I64MAX) atomicMin((long long*)&a.mn[q], (long long)acc);
  } else {
    if ((int64_t)acc != I64MIN) atomicMax((long long*)&a.mx[q], (long long)acc);
  }
}

static NamesArgs names_args(Ctx& c) {
  NamesArgs a;
  a.rows = c.k_rows;
  a.name = c.ev.name;
  a.ts = c.ev.ts;
  a.te = c.ev.te;
  a.ds = c.ds;
  a.NN = c.NN;
  a.part = c.name_part;
  a.blocks = c.name_blocks;
  a.count = c.o.name_count;
  a.sum = c.o.name_sum;
  a.mn = c.o.name_min;
  a.mx = c.o.name_max;
  a.tables = c.o.name_count || c.o.name_sum || c.o.name_min || c.o.name_max;
  a.link = c.o.link;
  a.aux = c.o.aux;
  return a;
}

int names_block_count(int64_t n_max, int NN) {
  if (NN > NM_LDS_NAMES) return (int)std::min<int64_t>(std::max<int64_t>(cdiv(n_max, 4096), 1), 1024);
  return (int)std::min<int64_t>(std::max<int64_t>(cdiv(n_max, 8192), 1), 256);
}

static bool names_tables(const Ctx& c) {
  return c.o.name_count || c.o.name_sum || c.o.name_min || c.o.name_max;
}

void launch_names(Ctx& c) {
  if (!names_tables(c)) return;
  NamesArgs a = names_args(c);
  const size_t lds = c.NN <= NM_LDS_NAMES ? (size_t)c.NN * 32 : 0;
  hipLaunchKernelGGL(k_names_partial, dim3(c.name_blocks), dim3(NM_THREADS), lds, c.st, a);
}

// after the join and the containment query
void launch_kernel_ops(Ctx& c) {
  if (!c.contain) return;
  NamesArgs a = names_args(c);
  const int64_t grid = std::max<int64_t>(cdiv(c.n, (int64_t)KO_THREADS * KO_ITEMS), 1);
  hipLaunchKernelGGL(k_kernel_ops, dim3((unsigned)grid), dim3(KO_THREADS), 0, c.st, a);
}

void launch_names_reduce(Ctx& c) {
  if (c.NN > NM_LDS_NAMES || !names_tables(c)) return;
  NamesArgs a = names_args(c);
  const int groups = std::min(NR_GROUPS, std::max(c.name_blocks, 1));
  hipLaunchKernelGGL(k_names_reduce, dim3((unsigned)cdiv((int64_t)c.NN * 4, 256), (unsigned)groups), dim3(256), 0, c.st,
                     a);
}

// ---------------------------------------------------------------- op names
// The same reductions per op name over the admitted CPU ops (the per-op-name
// variant), from the containment list (prep's compacted ops and launches,
// sorted with containment, in row order without it): a private LDS table per
// workgroup, written out whole and folded by a second kernel; more op names
// than the LDS budget go to the outputs by global atomics.
constexpr int ON_THREADS = 512;
constexpr int ON_LDS_NAMES = 2048;  // 64 KB of LDS, the default dynamic limit
constexpr int ON_MAX_BLOCKS = 512;
constexpr int ON_BATCH = 8;

struct OpNamesArgs {
  const uint64_t* keys[2];
  const uint32_t* vals[2];
  bool sorted;  // the containment list was sorted (its buffer is given by the parity)
  DevState* ds;
  const int32_t* name;
  const int64_t* ts;
  const int64_t* te;
  int NOP;
  bool lds;
  uint64_t* part;  // [blocks][NOP][4]
  int blocks;
  int64_t* out[4];  // count, sum, min, max (each may be NULL)
};

__global__ __launch_bounds__(ON_THREADS) void k_opnames_partial(OpNamesArgs a) {
  extern __shared__ unsigned long long otab[];  // [NOP][4]
  const int tid = threadIdx.x;
  if (a.lds) {
    for (int q = tid; q < a.NOP; q += ON_THREADS) {
      otab[q * 4 + 0] = 0;
      otab[q * 4 + 1] = 0;
      otab[q * 4 + 2] = (unsigned long long)I64MAX;
      otab[q * 4 + 3] = (unsigned long long)I64MIN;
    }
    __syncthreads();
  }
  const int par = a.sorted ? (int)a.ds->sort_parity[SORT_C] : 0;
  const uint64_t* keys = a.keys[par];
  const uint32_t* vals = a.vals[par];
  const int64_t n = a.ds->nCL;
  // ON_BATCH entries per thread and round, each round of loads issued
  // together (positions past the end take the last entry and are skipped)
  const int64_t stride = (int64_t)gridDim.x * ON_THREADS;
  for (int64_t i0 = (int64_t)blockIdx.x * ON_THREADS + tid; i0 < n; i0 += ON_BATCH * stride) {
    uint32_t rr[ON_BATCH];
    bool op[ON_BATCH];
#pragma unroll
    for (int u = 0; u < ON_BATCH; ++u) {
      const int64_t i = i0 + u * stride;
      const int64_t ic = i < n ? i : n - 1;
      op[u] = i < n && (keys[ic] & 1) == 0;
      rr[u] = vals[ic];
    }
    int qq[ON_BATCH];
    int64_t dd[ON_BATCH];
#pragma unroll
    for (int u = 0; u < ON_BATCH; ++u) {
      qq[u] = a.name[rr[u]];
      dd[u] = a.te[rr[u]] - a.ts[rr[u]];
    }
#pragma unroll
    for (int u = 0; u < ON_BATCH; ++u) {
    if (!op[u]) continue;
    const int q = qq[u];
    const int64_t d = dd[u];
    if (a.lds) {
      atomicAdd(&otab[q * 4 + 0], 1ull);
      atomicAdd(&otab[q * 4 + 1], (unsigned long long)d);
      atomicMin((long long*)&otab[q * 4 + 2], (long long)d);
      atomicMax((long long*)&otab[q * 4 + 3], (long long)d);
    } else {
      if (a.out[0]) atomicAdd((unsigned long long*)&a.out[0][q], 1ull);
      if (a.out[1]) atomicAdd((unsigned long long*)&a.out[1][q], (unsigned long long)d);
      if (a.out[2]) atomicMin((long long*)&a.out[2][q], (long long)d);
      if (a.out[3]) atomicMax((long long*)&a.out[3][q], (long long)d);
    }
    }
  }
  if (!a.lds) return;
  __syncthreads();
  uint64_t* o = a.part + (int64_t)blockIdx.x * a.NOP * 4;
  for (int i = tid; i < a.NOP * 4; i += ON_THREADS) o[i] = otab[i];
}

// One thread per (op name, statistic) and row of the grid; one atomic each
// into the outputs, which start as the identities.
__global__ __launch_bounds__(256) void k_opnames_fold(OpNamesArgs a) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t nv = (int64_t)a.NOP * 4;
  if (t >= nv) return;
  const int q = (int)(t >> 2), st = (int)(t & 3);
  int64_t* const dst = a.out[st];
  if (!dst) return;
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
      if (st < 2)
        acc += v[i];
      else if (st == 2)
        acc = (int64_t)v[i] < (int64_t)acc ? v[i] : acc;
      else
        acc = (int64_t)v[i] > (int64_t)acc ? v[i] : acc;
    }
  }
  if (st < 2) {
    if (acc) atomicAdd((unsigned long long*)&dst[q], (unsigned long long)acc);
  } else if (st == 2) {
    if ((int64_t)acc != I64MAX) atomicMin((long long*)&dst[q], (long long)acc);
  } else if ((int64_t)acc != I64MIN) {
    atomicMax((long long*)&dst[q], (long long)acc);
  }
}

bool opnames_wanted(const Ctx& c) {
  return c.o.opname_count || c.o.opname_sum || c.o.opname_min || c.o.opname_max;
}
bool opnames_use_tables(int NOP) { return NOP <= ON_LDS_NAMES; }
// one workgroup per 4096 entries, capped at ON_MAX_BLOCKS and so that the
// per-workgroup tables (NOP * 32 bytes each) stay within 4 MB
int opnames_block_count(int64_t n_max, int NOP) {
  const int64_t cap = std::max<int64_t>((int64_t)(4 << 20) / ((int64_t)std::max(NOP, 1) * 32), 1);
  return (int)std::min<int64_t>({std::max<int64_t>(cdiv(n_max, 4096), 1), (int64_t)ON_MAX_BLOCKS, cap});
}

void launch_opnames(Ctx& c) {
  if (!opnames_wanted(c)) return;
  OpNamesArgs a;
  for (int b = 0; b < 2; ++b) {
    a.keys[b] = c.sC.k[b];
    a.vals[b] = c.sC.v[b];
  }
  a.sorted = c.contain;
  a.ds = c.ds;
  a.name = c.ev.name;
  a.ts = c.ev.ts;
  a.te = c.ev.te;
  a.NOP = c.NOP;
  a.lds = opnames_use_tables(c.NOP);
  a.part = c.opn_part;
  a.blocks = c.opn_blocks;
  a.out[0] = c.o.opname_count;
  a.out[1] = c.o.opname_sum;
  a.out[2] = c.o.opname_min;
  a.out[3] = c.o.opname_max;
  hipLaunchKernelGGL(k_opnames_partial, dim3((unsigned)c.opn_blocks), dim3(ON_THREADS),
                     a.lds ? (size_t)c.NOP * 32 : 0, c.st, a);
  if (a.lds) {
    const unsigned gy = (unsigned)std::min(32, c.opn_blocks);  // 16 tables or fewer per thread: one round of loads
    hipLaunchKernelGGL(k_opnames_fold, dim3((unsigned)cdiv((int64_t)c.NOP * 4, 256), gy), dim3(256), 0, c.st, a);
  }
}

int names_lds_limit() { return NM_LDS_NAMES; }

void names_set_lds_attr() {
  (void)hipFuncSetAttribute((const void*)k_names_partial, hipFuncAttributeMaxDynamicSharedMemorySize,
                            NM_LDS_NAMES * 32);
}

}  // namespace hx
