// Per kernel-name aggregates: count, sum, min and max of the unclipped
// kernel duration over all admitted kernels (Section 6.1 measures kernel
// durations; grouping by kernel name is the per-name view of the same
// records).
//
// Each workgroup keeps a private table of all names in LDS (32 bytes per
// name) while it streams a slice of the admitted kernels, then writes the
// table out whole; a second kernel folds the tables name by name.  No global
// atomics touch the hot names of a Zipf-distributed name mix.  Name counts
// beyond the LDS budget fall back to global atomics.
#include "internal.hpp"

namespace hx {

constexpr int NM_THREADS = 256;
constexpr int NM_LDS_NAMES = 4096;  // 128 KB of LDS

struct NamesArgs {
  const uint32_t* rows;  // admitted kernels (any order)
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
};

__global__ __launch_bounds__(NM_THREADS) void k_names_partial(NamesArgs a) {
  extern __shared__ unsigned long long tab[];  // [NN][4]: count, sum, min, max
  const int tid = threadIdx.x;
  const bool lds = a.NN <= NM_LDS_NAMES;
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
  for (int64_t i = (int64_t)blockIdx.x * NM_THREADS + tid; i < n; i += (int64_t)gridDim.x * NM_THREADS) {
    const uint32_t r = a.rows[i];
    const int32_t q = a.name[r];
    const int64_t d = a.te[r] - a.ts[r];
    if (lds) {
      atomicAdd(&tab[q * 4 + 0], 1ull);
      atomicAdd(&tab[q * 4 + 1], (unsigned long long)d);
      atomicMin((long long*)&tab[q * 4 + 2], (long long)d);
      atomicMax((long long*)&tab[q * 4 + 3], (long long)d);
    } else {
      atomicAdd((unsigned long long*)&a.count[q], 1ull);
      atomicAdd((unsigned long long*)&a.sum[q], (unsigned long long)d);
      atomicMin((long long*)&a.mn[q], (long long)d);
      atomicMax((long long*)&a.mx[q], (long long)d);
    }
  }
  if (!lds) return;
  __syncthreads();
  uint64_t* out = a.part + (int64_t)blockIdx.x * a.NN * 4;
  for (int i = tid; i < a.NN * 4; i += NM_THREADS) out[i] = tab[i];
}

__global__ __launch_bounds__(256) void k_names_reduce(NamesArgs a) {
  const int q = blockIdx.x * 256 + threadIdx.x;
  if (q >= a.NN) return;
  uint64_t c = 0, s = 0;
  int64_t mn = I64MAX, mx = I64MIN;
  for (int b = 0; b < a.blocks; ++b) {
    const uint64_t* t = a.part + ((int64_t)b * a.NN + q) * 4;
    c += t[0];
    s += t[1];
    mn = (int64_t)t[2] < mn ? (int64_t)t[2] : mn;
    mx = (int64_t)t[3] > mx ? (int64_t)t[3] : mx;
  }
  a.count[q] = (int64_t)c;
  a.sum[q] = (int64_t)s;
  a.mn[q] = mn;
  a.mx[q] = mx;
}

static NamesArgs names_args(Ctx& c) {
  NamesArgs a;
  a.rows = c.sK.v[0];
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
  return a;
}

int names_block_count(int64_t n_max, int NN) {
  if (NN > NM_LDS_NAMES) return (int)std::min<int64_t>(std::max<int64_t>(cdiv(n_max, 4096), 1), 1024);
  return (int)std::min<int64_t>(std::max<int64_t>(cdiv(n_max, 16384), 1), 128);
}

void launch_names(Ctx& c) {
  NamesArgs a = names_args(c);
  const size_t lds = c.NN <= NM_LDS_NAMES ? (size_t)c.NN * 32 : 0;
  hipLaunchKernelGGL(k_names_partial, dim3(c.name_blocks), dim3(NM_THREADS), lds, c.st, a);
}

void launch_names_reduce(Ctx& c) {
  if (c.NN > NM_LDS_NAMES) return;
  NamesArgs a = names_args(c);
  hipLaunchKernelGGL(k_names_reduce, dim3((unsigned)cdiv(c.NN, 256)), dim3(256), 0, c.st, a);
}

int names_lds_limit() { return NM_LDS_NAMES; }

void names_set_lds_attr() {
  (void)hipFuncSetAttribute((const void*)k_names_partial, hipFuncAttributeMaxDynamicSharedMemorySize,
                            NM_LDS_NAMES * 32);
}

}  // namespace hx
