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
// Exactness: 10^15 F and T_op * peak take up to 127 bits; the quotient comes
// from a binary long division over the quotient's own bits only (about 20
// for a ppm), saturating at INT64_MAX.
//
// One pass streams the containment list (ops and launches in sorted order;
// an op's aggregates are final once the aggregate pass has run), each
// workgroup keeping a private table of all op names in LDS (32 bytes a
// name) that it writes out whole; a second kernel folds the tables into
// totals, and its last workgroup to finish writes the per-name outputs.
#include "internal.hpp"

namespace hx {

constexpr int SOL_THREADS = 512;
constexpr int SOL_BATCH = 4;
constexpr int SOL_LDS_NAMES = 2048;  // 64 KB of LDS, the default dynamic limit
constexpr int SOL_MAX_BLOCKS = 256;
constexpr int SR_GROUPS = 8;  // workgroup rows of the fold, each folding every SR_GROUPS-th table

typedef unsigned __int128 u128;

__device__ __forceinline__ int bitlen128(u128 x) {
  const uint64_t hi = (uint64_t)(x >> 64), lo = (uint64_t)x;
  return hi ? 128 - __clzll((long long)hi) : lo ? 64 - __clzll((long long)lo) : 0;
}

// min(floor(num / den), INT64_MAX) for den > 0.
__device__ __forceinline__ int64_t udiv_sat(u128 num, u128 den) {
  if ((num >> 63) >= den) return I64MAX;  // the quotient is at least 2^63
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
  const uint64_t* keys[2];
  const uint32_t* vals[2];
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
  bool lds;  // per-workgroup tables in LDS, else atomics on the totals
  int64_t* mfu;
  int64_t* mbu;
  int64_t* sol;
  uint64_t* part;  // [blocks][NOP][4]
  int blocks;
  uint64_t* tot;  // [NOP][4]: F, B, T_op, hotness (cleared by the init kernel)
  int64_t* o_flops;
  int64_t* o_bytes;
  int64_t* o_time;
  int64_t* o_sol;
  int64_t* o_hot;
};

__global__ __launch_bounds__(SOL_THREADS) void k_sol_partial(SolArgs a) {
  extern __shared__ unsigned long long tab[];  // [NOP][4]
  const int tid = threadIdx.x;
  if (a.lds) {
    for (int q = tid; q < a.NOP * 4; q += SOL_THREADS) tab[q] = 0;
    __syncthreads();
  }
  const int64_t n = a.ds->nCL;
  const int par = (int)a.ds->sort_parity[1];
  const uint64_t* keys = a.keys[par];
  const uint32_t* vals = a.vals[par];
  const int64_t stride = (int64_t)gridDim.x * SOL_THREADS;
  for (int64_t i0 = (int64_t)blockIdx.x * SOL_THREADS + tid; i0 < n; i0 += SOL_BATCH * stride) {
    // each round of loads is issued for the whole batch (positions past the
    // end take the last entry and are skipped)
    uint32_t r[SOL_BATCH];
    bool op[SOL_BATCH];
#pragma unroll
    for (int u = 0; u < SOL_BATCH; ++u) {
      const int64_t i = i0 + u * stride;
      const int64_t ic = i < n ? i : n - 1;
      op[u] = i < n && (keys[ic] & 1) == 0;
      r[u] = vals[ic];
    }
    int32_t nk[SOL_BATCH], nm[SOL_BATCH];
    int64_t f[SOL_BATCH], l[SOL_BATCH], F[SOL_BATCH], B[SOL_BATCH];
#pragma unroll
    for (int u = 0; u < SOL_BATCH; ++u) {
      nk[u] = 0;
      if (!op[u]) continue;
      const uint32_t rr = r[u];
      nk[u] = a.nkern[rr];
      f[u] = a.first[rr];
      l[u] = a.last[rr];
      F[u] = a.flops[rr];
      B[u] = a.bytes[rr];
      nm[u] = a.name[rr];
    }
    int64_t ref[SOL_BATCH];
#pragma unroll
    for (int u = 0; u < SOL_BATCH; ++u) ref[u] = a.ref && op[u] && nk[u] > 0 ? a.ref[nm[u]] : 0;
#pragma unroll
    for (int u = 0; u < SOL_BATCH; ++u) {
      if (!op[u]) continue;
      const uint32_t rr = r[u];
      const int64_t T = nk[u] > 0 ? (int64_t)((uint64_t)l[u] - (uint64_t)f[u]) : 0;
      if (T <= 0) {  // unmeasured: no kernels, or kernels that span no time
        if (a.mfu) a.mfu[rr] = -1;
        if (a.mbu) a.mbu[rr] = -1;
        if (a.sol) a.sol[rr] = -1;
        continue;
      }
      const int64_t mf = ppm((uint64_t)F[u], (uint64_t)T, a.PF);
      const int64_t mb = ppm((uint64_t)B[u], (uint64_t)T, a.PB);
      const int64_t s = mf > mb ? mf : mb;
      if (a.mfu) a.mfu[rr] = mf;
      if (a.mbu) a.mbu[rr] = mb;
      if (a.sol) a.sol[rr] = s;
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
  uint64_t* out = a.part + (int64_t)blockIdx.x * a.NOP * 4;
  for (int i = tid; i < a.NOP * 4; i += SOL_THREADS) out[i] = tab[i];
}

// One thread per (name, statistic) and workgroup row: row g folds the
// tables g, g + rows, ... with 16 independent, coalesced loads in flight and
// adds its sum into the totals.  The last workgroup to finish (a counter in
// the state, cleared by the init kernel) writes the per-name outputs and
// checks the reference table.
__global__ __launch_bounds__(256) void k_sol_reduce(SolArgs a) {
  __shared__ int s_last;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t stride = (int64_t)a.NOP * 4;
  if (a.lds && t < stride) {
    uint64_t acc = 0;
    for (int b0 = blockIdx.y; b0 < a.blocks; b0 += 16 * (int)gridDim.y) {
      uint64_t v[16];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int b = b0 + i * (int)gridDim.y;
        v[i] = a.part[(int64_t)(b < a.blocks ? b : blockIdx.y) * stride + t];
      }
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (b0 + i * (int)gridDim.y < a.blocks) acc += v[i];
    }
    if (acc) atomicAdd((unsigned long long*)&a.tot[t], (unsigned long long)acc);
  }
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) s_last = atomicAdd(&a.ds->sol_done, 1u) == gridDim.x * gridDim.y - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  bool bad = false;
  for (int o = threadIdx.x; o < a.NOP; o += 256) {
    const uint64_t F = ld_agent(&a.tot[4 * o + 0]), B = ld_agent(&a.tot[4 * o + 1]);
    const uint64_t T = ld_agent(&a.tot[4 * o + 2]), H = ld_agent(&a.tot[4 * o + 3]);
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
    if (a.ref && a.ref[o] < 0) bad = true;
  }
  if (bad) set_status(a.ds, DS_PARAM);
}

static SolArgs sol_args(Ctx& c) {
  SolArgs a;
  a.keys[0] = c.sC.k[0];
  a.keys[1] = c.sC.k[1];
  a.vals[0] = c.sC.v[0];
  a.vals[1] = c.sC.v[1];
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
  a.lds = c.NOP <= SOL_LDS_NAMES;
  a.mfu = c.o.op_mfu;
  a.mbu = c.o.op_mbu;
  a.sol = c.o.op_sol;
  a.part = c.sol_part;
  a.blocks = c.sol_blocks;
  a.tot = c.sol_tot;
  a.o_flops = c.o.opn_flops;
  a.o_bytes = c.o.opn_bytes;
  a.o_time = c.o.opn_time;
  a.o_sol = c.o.opn_sol;
  a.o_hot = c.o.opn_hot;
  return a;
}

int sol_block_count(int64_t n_max, int NOP) {
  const int64_t b = std::min<int64_t>(std::max<int64_t>(cdiv(n_max, 8192), 1), SOL_MAX_BLOCKS);
  if (NOP > SOL_LDS_NAMES) return (int)std::min<int64_t>(std::max<int64_t>(cdiv(n_max, 4096), 1), 1024);
  return (int)b;
}

bool sol_uses_tables(int NOP) { return NOP <= SOL_LDS_NAMES; }

void launch_sol(Ctx& c) {
  SolArgs a = sol_args(c);
  const size_t lds = a.lds ? (size_t)c.NOP * 32 : 0;
  hipLaunchKernelGGL(k_sol_partial, dim3((unsigned)c.sol_blocks), dim3(SOL_THREADS), lds, c.st, a);
  const unsigned gx = a.lds ? (unsigned)cdiv((int64_t)c.NOP * 4, 256) : 1u;
  const unsigned gy = a.lds ? (unsigned)std::min(SR_GROUPS, std::max(c.sol_blocks, 1)) : 1u;
  hipLaunchKernelGGL(k_sol_reduce, dim3(gx, gy), dim3(256), 0, c.st, a);
}

}  // namespace hx
