// Operator efficiency (Section 6.1, "Operator execution and efficiency").
// A measured op's MFU and MBU are its operation count F and its logical
// bytes B over its span T_op (first kernel start to last kernel end, from
// the inclusive per-op aggregates) and the device's peaks, in parts per
// million; its SOL is the larger of the two.  Per op name: the sums of F, B
// and T_op over the measured ops, the SOL of those sums, and the hotness,
// the time the name's ops below the name's reference SOL would save by
// reaching it, sum of floor(T_op (ref - SOL) / ref) (Section 6.2 ranks the
// distance to a reference by the time it costs).
//
// Exactness: 10^15 F and T_op * peak take up to 127 bits.  A quotient below
// 2^50 (every realistic ppm) is estimated in double precision, which puts
// it within one of the exact value, and corrected by exact 128-bit
// multiplication; larger ones take a binary long division over the
// quotient's own bits; results saturate at INT64_MAX.
//
// One pass over the rows, after the per-op aggregates are final, each
// workgroup keeping a private table of all op names in LDS (32 bytes a
// name); a second kernel folds the tables into totals and a third writes
// the per-name outputs.
#include "internal.hpp"

namespace hx {

constexpr int SOL_THREADS = 512;
constexpr int SOL_BATCH = 4;
constexpr int SOL_LDS_NAMES = 2048;  // 64 KB of LDS, the default dynamic limit
constexpr int SOL_MAX_BLOCKS = 1024;
constexpr int64_t SOL_PART_BYTES = 8 << 20;  // bound on the per-workgroup tables written per call
constexpr int SF_ROWS = 64;  // rows of the fold's grid: each thread folds SOL_MAX_BLOCKS / SF_ROWS tables

typedef unsigned __int128 u128;

__device__ __forceinline__ int bitlen128(u128 x) {
  const uint64_t hi = (uint64_t)(x >> 64), lo = (uint64_t)x;
  return hi ? 128 - __clzll((long long)hi) : lo ? 64 - __clzll((long long)lo) : 0;
}

__device__ __forceinline__ double u128_to_double(u128 x) {
  return (double)(uint64_t)(x >> 64) * 18446744073709551616.0 + (double)(uint64_t)x;
}

// min(floor(num / den), INT64_MAX) for den > 0.
__device__ __forceinline__ int64_t udiv_sat(u128 num, u128 den) {
  if ((num >> 63) >= den) return I64MAX;  // the quotient is at least 2^63
  // Both conversions and the division round to nearest: the estimate's
  // relative error is below 5 * 2^-53 < 2^-50, so under 2^50 it lies within
  // one of num/den.
  const double qd = u128_to_double(num) / u128_to_double(den);
  if (qd < 1125899906842624.0) {
    uint64_t q = (uint64_t)qd;
    // q * den stays below 2^128: q is at most one above the quotient, the
    // quotient times den is at most num, and num and den are below 2^127
    u128 prod = (u128)q * den;
    while (prod > num) {
      --q;
      prod -= den;
    }
    while (num - prod >= den) {
      ++q;
      prod += den;
    }
    return (int64_t)q;
  }
  int k = bitlen128(num) - bitlen128(den);
  if (k < 0) return 0;
  // the quotient is below 2^(k+1) and below 2^63; den << k is below
  // 2^bitlen(num), so no shift overflows
  uint64_t q = 0;
  for (; k >= 0; --k) {
    const u128 d = den << k;
    if (num >= d) {
      num -= d;
      q |= 1ull << k;
    }
  }
  return (int64_t)q;
}

// floor(10^15 x / (t peak)) in ppm: x an unsigned count, t > 0 ns, peak > 0 per second.
__device__ __forceinline__ int64_t ppm(uint64_t x, uint64_t t, uint64_t peak) {
  return udiv_sat((u128)x * 1000000000000000ull, (u128)t * peak);
}

struct SolArgs {
  int64_t n;
  const uint8_t* kind;
  const int32_t* link;  // -2 at rows outside the window (a workspace array when the output is NULL)
  DevState* ds;
  const int32_t* name;
  const int64_t* flops;
  const int64_t* bytes;
  const int32_t* nkern;
  const int64_t* first;
  const int64_t* last;
  const int64_t* ref;  // [NOP] or NULL
  uint64_t PF, PB;
  int NOP;
  bool lds;       // per-workgroup tables in LDS folded in two levels, else atomics on the totals
  int64_t* mfu;
  int64_t* mbu;
  int64_t* sol;
  uint64_t* part;   // [blocks][NOP * 4] each workgroup's table
  uint64_t* tot;    // [NOP * 4]: F, B, T_op, hotness (atomics; cleared by the init kernel)
  int64_t* o_flops;
  int64_t* o_bytes;
  int64_t* o_time;
  int64_t* o_sol;
  int64_t* o_hot;
};

// Writes the per-name outputs from the totals (F, B, T_op, hotness) of op
// name o, and flags a negative reference.
__device__ __forceinline__ bool sol_name_out(const SolArgs& a, int o, uint64_t F, uint64_t B, uint64_t T, uint64_t H) {
  if (a.o_flops) a.o_flops[o] = (int64_t)F;
  if (a.o_bytes) a.o_bytes[o] = (int64_t)B;
  if (a.o_time) a.o_time[o] = (int64_t)T;
  if (a.o_hot) a.o_hot[o] = (int64_t)H;
  if (a.o_sol) {
    int64_t s = -1;
    if (T != 0) {
      const int64_t mf = ppm(F, T, a.PF), mb = ppm(B, T, a.PB);
      s = mf > mb ? mf : mb;
    }
    a.o_sol[o] = s;
  }
  return a.ref && a.ref[o] < 0;
}

// Rows in row order, SOL_BATCH per thread and round (consecutive threads on
// consecutive rows, so the op columns are read where the ops lie, and a
// trace that delivers records of one kind together reads them contiguously).
// A row is a measured op when it is an admitted CPU op with kernels and
// T_op > 0.  Per-name sums go to the workgroup's LDS table, written out
// whole at the end (or, with more names than LDS holds, to the totals by
// global atomics).  Tables are handed to the next kernel, not to a last
// workgroup of this one: on this chip a workgroup's stores reach another
// XCD only after a device-scope release, which writes back the whole L2.
__global__ __launch_bounds__(SOL_THREADS) void k_sol(SolArgs a) {
  extern __shared__ unsigned long long tab[];  // [NOP * 4]
  const int tid = threadIdx.x;
  const int nv = a.NOP * 4;
  if (a.lds) {
    for (int q = tid; q < nv; q += SOL_THREADS) tab[q] = 0;
    __syncthreads();
  }
  const int64_t n = a.n;
  const int64_t stride = (int64_t)gridDim.x * SOL_THREADS;
  for (int64_t r0 = (int64_t)blockIdx.x * SOL_THREADS + tid; r0 < n; r0 += SOL_BATCH * stride) {
    // each round of loads is issued for the whole batch (rows past the end
    // load the last row and are skipped)
    bool op[SOL_BATCH];
#pragma unroll
    for (int u = 0; u < SOL_BATCH; ++u) {
      const int64_t r = r0 + u * stride;
      const int64_t rc = r < n ? r : n - 1;
      const int k = a.kind[rc];
      const int32_t l = a.link[rc];
      op[u] = r < n && k == HERSCHEL_CPU_OP && l != -2;
    }
    int32_t nk[SOL_BATCH], nm[SOL_BATCH];
    int64_t f[SOL_BATCH], l[SOL_BATCH], F[SOL_BATCH], B[SOL_BATCH];
#pragma unroll
    for (int u = 0; u < SOL_BATCH; ++u) {
      nk[u] = 0;
      if (!op[u]) continue;
      const int64_t r = r0 + u * stride;
      nk[u] = a.nkern[r];
      f[u] = a.first[r];
      l[u] = a.last[r];
      F[u] = a.flops[r];
      B[u] = a.bytes[r];
      nm[u] = a.name[r];
    }
    int64_t ref[SOL_BATCH];
#pragma unroll
    for (int u = 0; u < SOL_BATCH; ++u) ref[u] = a.ref && op[u] && nk[u] > 0 ? a.ref[nm[u]] : 0;
#pragma unroll
    for (int u = 0; u < SOL_BATCH; ++u) {
      if (!op[u]) continue;
      const int64_t r = r0 + u * stride;
      const int64_t T = nk[u] > 0 ? (int64_t)((uint64_t)l[u] - (uint64_t)f[u]) : 0;
      if (T <= 0) {  // unmeasured: no kernels, or kernels that span no time
        if (a.mfu) a.mfu[r] = -1;
        if (a.mbu) a.mbu[r] = -1;
        if (a.sol) a.sol[r] = -1;
        continue;
      }
      const int64_t mf = ppm((uint64_t)F[u], (uint64_t)T, a.PF);
      const int64_t mb = ppm((uint64_t)B[u], (uint64_t)T, a.PB);
      const int64_t s = mf > mb ? mf : mb;
      if (a.mfu) a.mfu[r] = mf;
      if (a.mbu) a.mbu[r] = mb;
      if (a.sol) a.sol[r] = s;
      const int64_t rf = ref[u];
      const uint64_t hot =
          rf > 0 && s < rf ? (uint64_t)udiv_sat((u128)(uint64_t)T * (uint64_t)(rf - s), (u128)(uint64_t)rf) : 0;
      const int q = nm[u];
      if (a.lds) {
        atomicAdd(&tab[q * 4 + 0], (unsigned long long)F[u]);
        atomicAdd(&tab[q * 4 + 1], (unsigned long long)B[u]);
        atomicAdd(&tab[q * 4 + 2], (unsigned long long)T);
        if (hot) atomicAdd(&tab[q * 4 + 3], (unsigned long long)hot);
      } else {
        atomicAdd((unsigned long long*)&a.tot[q * 4 + 0], (unsigned long long)F[u]);
        atomicAdd((unsigned long long*)&a.tot[q * 4 + 1], (unsigned long long)B[u]);
        atomicAdd((unsigned long long*)&a.tot[q * 4 + 2], (unsigned long long)T);
        if (hot) atomicAdd((unsigned long long*)&a.tot[q * 4 + 3], (unsigned long long)hot);
      }
    }
  }
  if (!a.lds) return;
  __syncthreads();
  for (int i = tid; i < nv; i += SOL_THREADS) a.part[(int64_t)blockIdx.x * nv + i] = tab[i];
}

// One thread per (name, statistic) and row of the grid: row g folds the
// tables g, g + rows, ... (16 independent, coalesced loads in flight) and
// adds its sum into the totals, which the init kernel has cleared.
__global__ __launch_bounds__(256) void k_sol_fold(SolArgs a, int blocks) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t nv = (int64_t)a.NOP * 4;
  if (t >= nv) return;
  uint64_t acc = 0;
  for (int b0 = blockIdx.y; b0 < blocks; b0 += 16 * (int)gridDim.y) {
    uint64_t v[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int b = b0 + i * (int)gridDim.y;
      v[i] = b < blocks ? a.part[(int64_t)b * nv + t] : 0;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) acc += v[i];
  }
  if (acc) atomicAdd((unsigned long long*)&a.tot[t], (unsigned long long)acc);
}

// One thread per op name: the per-name outputs from the totals.
__global__ __launch_bounds__(256) void k_sol_names(SolArgs a) {
  const int o = blockIdx.x * 256 + threadIdx.x;
  bool bad = false;
  if (o < a.NOP) bad = sol_name_out(a, o, a.tot[4 * o], a.tot[4 * o + 1], a.tot[4 * o + 2], a.tot[4 * o + 3]);
  if (ballot(bad) && lane_id() == 0) set_status(a.ds, DS_PARAM);
}

static SolArgs sol_args(Ctx& c) {
  SolArgs a;
  a.n = c.n;
  a.kind = c.ev.kind;
  a.link = c.o.link;
  a.ds = c.ds;
  a.name = c.ev.name;
  a.flops = c.ev.flops;
  a.bytes = c.ev.bytes;
  a.nkern = c.o.op_nkern;
  a.first = c.o.op_first;
  a.last = c.o.op_last;
  a.ref = c.p.ref_sol_ppm;
  a.PF = (uint64_t)c.p.peak_flops;
  a.PB = (uint64_t)c.p.peak_bytes;
  a.NOP = c.NOP;
  a.lds = sol_uses_tables(c.NOP);
  a.mfu = c.o.op_mfu;
  a.mbu = c.o.op_mbu;
  a.sol = c.o.op_sol;
  a.part = c.sol_part;
  a.tot = c.sol_tot;
  a.o_flops = c.o.opn_flops;
  a.o_bytes = c.o.opn_bytes;
  a.o_time = c.o.opn_time;
  a.o_sol = c.o.opn_sol;
  a.o_hot = c.o.opn_hot;
  return a;
}

// Workgroups of the op pass: about 2048 rows each, at most SOL_MAX_BLOCKS,
// and with name tables no more than SOL_PART_BYTES of them.
int sol_block_count(int64_t n_max, int NOP) {
  int64_t b = std::min<int64_t>(cdiv(n_max, 2048), SOL_MAX_BLOCKS);
  if (sol_uses_tables(NOP)) b = std::min<int64_t>(b, SOL_PART_BYTES / ((int64_t)NOP * 32));
  return (int)std::max<int64_t>(b, 1);
}

bool sol_uses_tables(int NOP) { return NOP <= SOL_LDS_NAMES; }

void launch_sol(Ctx& c) {
  SolArgs a = sol_args(c);
  const size_t lds = a.lds ? (size_t)c.NOP * 32 : 0;
  hipLaunchKernelGGL(k_sol, dim3((unsigned)c.sol_blocks), dim3(SOL_THREADS), lds, c.st, a);
  if (a.lds) {
    const unsigned gx = (unsigned)cdiv((int64_t)c.NOP * 4, 256);
    const unsigned gy = (unsigned)std::min(SF_ROWS, c.sol_blocks);
    hipLaunchKernelGGL(k_sol_fold, dim3(gx, gy), dim3(256), 0, c.st, a, c.sol_blocks);
  }
  hipLaunchKernelGGL(k_sol_names, dim3((unsigned)cdiv(c.NOP, 256)), dim3(256), 0, c.st, a);
}

}  // namespace hx
