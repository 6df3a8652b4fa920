// Per kernel-name aggregates: count, sum, min and max of the unclipped
// kernel duration over all admitted kernels (Section 6.1 measures kernel
// durations; grouping by kernel name is the per-name view of the same
// records).  With containment the same pass over the kernels also gives each
// matched kernel the op of its launch (kernel composition, Section 6.1) and
// counts the matched kernels whose launch has no op.
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
  // kernel -> op (with containment): the op of the kernel's launch
  bool kernel_ops;
  bool tables;  // some name output is wanted
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
  uint32_t unattr = 0;  // matched kernels whose launch has no op
  // NM_BATCH kernels per thread and round, each round of loads issued
  // together (positions past the end take the last kernel: clamped, not
  // branched on, and then skipped)
  const int64_t stride = (int64_t)gridDim.x * NM_THREADS;
  for (int64_t i0 = (int64_t)blockIdx.x * NM_THREADS + tid; i0 < n; i0 += NM_BATCH * stride) {
    uint32_t r[NM_BATCH];
#pragma unroll
    for (int u = 0; u < NM_BATCH; ++u) r[u] = rows[i0 + u * stride < n ? i0 + u * stride : n - 1];
    int32_t q[NM_BATCH], l[NM_BATCH];
    int64_t d[NM_BATCH];
#pragma unroll
    for (int u = 0; u < NM_BATCH; ++u) {
      const int32_t nm = a.name[r[u]];
      const int64_t e = a.te[r[u]], s = a.ts[r[u]];
      l[u] = a.kernel_ops ? a.link[r[u]] : -1;
      q[u] = i0 + u * stride < n ? nm : -1;
      d[u] = e - s;
    }
    if (a.kernel_ops) {
      // the op of each matched kernel's launch (one more round of gathers)
      int32_t op[NM_BATCH];
#pragma unroll
      for (int u = 0; u < NM_BATCH; ++u) op[u] = a.link[l[u] >= 0 ? l[u] : 0];
#pragma unroll
      for (int u = 0; u < NM_BATCH; ++u) {
        if (q[u] < 0 || l[u] < 0) continue;
        a.aux[r[u]] = op[u];
        if (op[u] < 0) ++unattr;
      }
    }
#pragma unroll
    for (int u = 0; u < NM_BATCH; ++u) {
      if (q[u] < 0 || !a.tables) continue;
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
  if (a.kernel_ops) {
    const uint64_t w = wave_sum_u64(unattr);
    if (lane_id() == 0 && w) atomicAdd(&a.ds->join_acc[blockIdx.x % JOIN_COPIES][JC_UNATTR], (unsigned long long)w);
  }
  if (!lds) return;
  __syncthreads();
  uint64_t* out = a.part + (int64_t)blockIdx.x * a.NN * 4;
  for (int i = tid; i < a.NN * 4; i += NM_THREADS) out[i] = tab[i];
}

// One thread per (name, statistic) and group of tables: group g folds the
// tables g, g + NR_GROUPS, ... with independent, coalesced loads
// (consecutive threads read consecutive words), 16 in flight, and combines
// its result into the output with one atomic (the outputs start as the
// identities, set by the init kernel).
constexpr int NR_GROUPS = 8;

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
  a.kernel_ops = c.contain;
  a.tables = c.o.name_count || c.o.name_sum || c.o.name_min || c.o.name_max;
  a.link = c.o.link;
  a.aux = c.o.aux;
  return a;
}

int names_block_count(int64_t n_max, int NN) {
  if (NN > NM_LDS_NAMES) return (int)std::min<int64_t>(std::max<int64_t>(cdiv(n_max, 4096), 1), 1024);
  return (int)std::min<int64_t>(std::max<int64_t>(cdiv(n_max, 8192), 1), 256);
}

// Names are wanted, or the pass gives kernels their ops (containment).
static bool names_needed(const Ctx& c) {
  return c.contain || c.o.name_count || c.o.name_sum || c.o.name_min || c.o.name_max;
}
static bool names_tables(const Ctx& c) {
  return c.o.name_count || c.o.name_sum || c.o.name_min || c.o.name_max;
}

void launch_names(Ctx& c) {
  if (!names_needed(c)) return;
  NamesArgs a = names_args(c);
  const size_t lds = a.tables && c.NN <= NM_LDS_NAMES ? (size_t)c.NN * 32 : 0;
  hipLaunchKernelGGL(k_names_partial, dim3(c.name_blocks), dim3(NM_THREADS), lds, c.st, a);
}

void launch_names_reduce(Ctx& c) {
  if (c.NN > NM_LDS_NAMES || !names_tables(c)) return;
  NamesArgs a = names_args(c);
  const int groups = std::min(NR_GROUPS, std::max(c.name_blocks, 1));
  hipLaunchKernelGGL(k_names_reduce, dim3((unsigned)cdiv((int64_t)c.NN * 4, 256), (unsigned)groups), dim3(256), 0, c.st,
                     a);
}

int names_lds_limit() { return NM_LDS_NAMES; }

void names_set_lds_attr() {
  (void)hipFuncSetAttribute((const void*)k_names_partial, hipFuncAttributeMaxDynamicSharedMemorySize,
                            NM_LDS_NAMES * 32);
}

}  // namespace hx
