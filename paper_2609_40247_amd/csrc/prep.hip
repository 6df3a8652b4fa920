// Prep: one pass over the raw records (37 bytes per row).
//
// Validates each row (record schema of Section 5.2), moves it onto the
// common clock, admits it by its start time (Section 5.2, session transitions), marks rows outside the window, and compacts the admitted rows, in
// row order, into the inputs of the three sorts:
//   timeline    (pid, stream, ts'-W0)            kernels
//   containment (pid, thread, ts'-W0, is_launch) ops and launches
//   join        (pid, corr mod 2^51, is_kernel)   launches and kernels (not sorted: the
//                                                 correlation table takes them in row order)
// and, with the idle-coincidence outputs, the op-name list
//   (pid, op name, ts'-W0) of the CPU ops, and for every kernel at its
//   timeline position the device-lane key (pid, ts'-W0).
// Compaction offsets come from a decoupled look-back per list; the last
// tile's prefixes are the admitted counts.
#include "internal.hpp"

namespace hx {

constexpr int PREP_THREADS = 512;
constexpr int PREP_ITEMS = 8;
constexpr int PREP_TILE = PREP_THREADS * PREP_ITEMS;

struct PrepArgs {
  herschel_events ev;
  int64_t n;
  const int64_t* off;
  int64_t W0, W1;
  int P, S, T, NN, NOP;
  int sb, tb, wb;
  int64_t n_tiles;
  bool jt_range;  // find each process's id range (at most JT_PROCS processes)
  bool waits;     // the op-name list and device-lane keys (idle coincidence)
  int nob;        // bits of an op name
  bool sol;       // ops carry operation counts and bytes (operator efficiency), which must be >= 0
  int NG;         // kernels carry a graph node in [-1, NG) (graph replay separation), 0: not read
  DevState* ds;
  herschel_counters* cnt;
  int32_t* link;
  int32_t* aux;
  uint64_t* status;  // [4][n_tiles]
  uint64_t* kK;
  uint32_t* vK;
  uint32_t* kRows;  // the admitted kernels' rows again, for the per-name tables (not sorted)
  uint64_t* kC;
  uint32_t* vC;
  uint64_t* kJ;
  uint32_t* vJ;
  uint64_t* kD;  // device-lane keys at the timeline positions
  uint32_t* vD;
  uint64_t* kO;  // op-name list
  uint32_t* vO;
};
constexpr int PREP_LISTS = 4;  // timeline, containment, join, op names

// Rows are loaded PREP_BATCH per thread at a time, every column of every row
// of a batch in flight together: no load waits for another (the correlation
// id is loaded for every kind, the clock offsets are read from LDS).
constexpr int PREP_BATCH = 2;
constexpr int PREP_OFF_LDS = 512;  // processes whose clock offsets are staged in LDS
// the four list flags of every item are packed into one 32-bit word
static_assert(PREP_LISTS * PREP_ITEMS <= 32, "list flags of all items must fit the 32-bit flag word");
static_assert(PREP_LISTS <= PREP_THREADS / WAVE, "one wave per list's look-back");
static_assert(PREP_ITEMS % PREP_BATCH == 0, "items are loaded in whole batches");
static_assert(PREP_THREADS % WAVE == 0 && 2 * JT_PROCS <= PREP_THREADS, "one thread per id-range word");

// Tiles are taken by workgroup index: a tile's look-back waits only for
// tiles of lower index, whose workgroups the dispatcher started first.
__global__ __launch_bounds__(PREP_THREADS) void k_prep(PrepArgs a) {
  __shared__ uint64_t s_bal[PREP_ITEMS][PREP_THREADS / WAVE][PREP_LISTS];
  __shared__ uint32_t s_off[PREP_ITEMS][PREP_THREADS / WAVE][PREP_LISTS];
  __shared__ uint32_t s_tot[PREP_LISTS];
  __shared__ uint64_t s_base[PREP_LISTS];
  __shared__ unsigned long long s_bad;
  __shared__ unsigned long long s_jr[2 * JT_PROCS];  // per process: max of ~u, max of u (u = corr ^ 2^63)
  __shared__ unsigned long long s_jp;                 // processes with an admitted launch or kernel
  __shared__ int64_t s_clk[PREP_OFF_LDS];

  const int tid = threadIdx.x, lane = lane_id(), wv = tid / WAVE;
  const int tile = blockIdx.x;
  const int64_t base = (int64_t)tile * PREP_TILE;
  const bool clk_lds = a.off && a.P <= PREP_OFF_LDS;
  if (tid == 0) {
    s_bad = ~0ull;
    s_jp = 0;
  }
  if (tid < 2 * JT_PROCS) s_jr[tid] = 0;
  if (clk_lds)
    for (int i = tid; i < a.P; i += PREP_THREADS) s_clk[i] = a.off[i];
  __syncthreads();

  uint64_t kA[PREP_ITEMS], kB[PREP_ITEMS];  // kA: timeline or containment key, kB: join key
  uint32_t fl = 0;                          // per item: bit 4j list K, 4j+1 C, 4j+2 J, 4j+3 O
  uint64_t bad = ~0ull;
  // id range of the thread's current process (the join items of a thread
  // mostly share one): tp the process, ulo / uhi the max of ~u and of u
  int tp = -1;
  uint64_t ulo = 0, uhi = 0;
  const uint64_t lt = lanemask_lt();
#pragma unroll
  for (int j0 = 0; j0 < PREP_ITEMS; j0 += PREP_BATCH) {
    // rows past the end load the last row (clamped index) and are ignored
    int kind_[PREP_BATCH];
    int32_t pid_[PREP_BATCH], lane_[PREP_BATCH], name_[PREP_BATCH];
    int64_t ts_[PREP_BATCH], te_[PREP_BATCH], corr_[PREP_BATCH], cost_[PREP_BATCH];
    int32_t node_[PREP_BATCH];
#pragma unroll
    for (int u = 0; u < PREP_BATCH; ++u) {
      const int64_t r = base + (int64_t)(j0 + u) * PREP_THREADS + tid;
      const int64_t rc = r < a.n ? r : a.n - 1;
      kind_[u] = a.ev.kind[rc];
      pid_[u] = a.ev.pid[rc];
      lane_[u] = a.ev.lane[rc];
      name_[u] = a.ev.name[rc];
      ts_[u] = a.ev.ts[rc];
      te_[u] = a.ev.te[rc];
      corr_[u] = a.ev.corr[rc];
      // an op's counts: negative iff either is (loaded for every kind)
      cost_[u] = a.sol ? a.ev.flops[rc] | a.ev.bytes[rc] : 0;
      node_[u] = a.NG ? a.ev.graph_node[rc] : -1;
    }
#pragma unroll
    for (int u = 0; u < PREP_BATCH; ++u) {
      const int j = j0 + u;
      const int64_t r = base + (int64_t)j * PREP_THREADS + tid;
      bool fK = false, fC = false, fJ = false, fO = false;
      kA[j] = 0;
      kB[j] = 0;
      if (r < a.n) {
        const int kind = kind_[u];
        const int32_t pid = pid_[u], ln = lane_[u], name = name_[u];
        const int64_t ts = ts_[u], te = te_[u];
        const int64_t corr = kind != HERSCHEL_CPU_OP ? corr_[u] : 0;
        constexpr int64_t LIM = HERSCHEL_MAX_ABS_TIME;
        bool ok = kind <= 2 && pid >= 0 && pid < a.P;
        if (kind == HERSCHEL_KERNEL)
          ok = ok && ln >= 0 && ln < a.S && name >= 0 && name < a.NN && node_[u] >= -1 &&
               (a.NG == 0 || node_[u] < a.NG);
        else
          ok = ok && ln >= 0 && ln < a.T && name >= 0 &&
               (kind != HERSCHEL_CPU_OP || (name < a.NOP && cost_[u] >= 0));
        ok = ok && ts > -LIM && ts < LIM && te > -LIM && te < LIM && te >= ts;
        bool adm = false;
        int64_t rel = 0;
        if (ok) {
          const int64_t o = !a.off ? 0 : clk_lds ? s_clk[pid] : a.off[pid];
          const int64_t tsc = ts - o;
          adm = tsc >= a.W0 && tsc < a.W1;
          rel = tsc - a.W0;
        } else {
          bad = (uint64_t)r < bad ? (uint64_t)r : bad;
        }
        if (!adm) {
          if (a.link) a.link[r] = -2;
          if (a.aux) a.aux[r] = -2;
        } else {
          fK = kind == HERSCHEL_KERNEL;
          fC = !fK;
          fJ = kind != HERSCHEL_CPU_OP;
          if (fK)
            kA[j] = ((uint64_t)pid << (a.sb + a.wb)) | ((uint64_t)ln << a.wb) | (uint64_t)rel;
          else
            kA[j] = ((uint64_t)pid << (a.tb + a.wb + 1)) | ((uint64_t)ln << (a.wb + 1)) | ((uint64_t)rel << 1) |
                    (uint64_t)(kind == HERSCHEL_LAUNCH);
          kB[j] = ((uint64_t)pid << JK_PID_SHIFT) | (((uint64_t)corr & JK_CORR_MASK) << 1) |
                  (uint64_t)(kind == HERSCHEL_KERNEL);
          fO = a.waits && kind == HERSCHEL_CPU_OP;
          if (fO)  // an op takes no join key: its slot holds the op-name key
            kB[j] = ((uint64_t)pid << (a.nob + a.wb)) | ((uint64_t)name << a.wb) | (uint64_t)rel;
          if (a.jt_range && fJ) {
            const uint64_t u = (uint64_t)corr ^ SIGN64;  // unsigned order = signed order of the ids
            if (pid != tp) {
              if (tp >= 0) {
                atomicMax(&s_jr[2 * tp], (unsigned long long)ulo);
                atomicMax(&s_jr[2 * tp + 1], (unsigned long long)uhi);
                atomicOr(&s_jp, 1ull << tp);
              }
              tp = pid;
              ulo = ~u;
              uhi = u;
            } else {
              ulo = ~u > ulo ? ~u : ulo;
              uhi = u > uhi ? u : uhi;
            }
          }
        }
      }
      fl |= (fK ? 1u : 0u) << (4 * j) | (fC ? 1u : 0u) << (4 * j + 1) | (fJ ? 1u : 0u) << (4 * j + 2) |
            (fO ? 1u : 0u) << (4 * j + 3);
      const uint64_t b0 = ballot(fK), b1 = ballot(fC), b2 = ballot(fJ), b3 = ballot(fO);
      if (lane == 0) {
        s_bal[j][wv][0] = b0;
        s_bal[j][wv][1] = b1;
        s_bal[j][wv][2] = b2;
        s_bal[j][wv][3] = b3;
      }
    }
  }
  if (bad != ~0ull) atomicMin(&s_bad, (unsigned long long)bad);
  __syncthreads();
  if (a.jt_range) {
    // each process's smallest and largest id: a wave whose items all belong
    // to one process combines them by shuffles, others add per thread
    int pm = tp;
    for (int d = 1; d < WAVE; d <<= 1) {
      const int o = __shfl_xor(pm, d, WAVE);
      pm = o > pm ? o : pm;
    }
    if (pm >= 0 && ballot(tp >= 0 && tp != pm) == 0) {
      for (int d = 1; d < WAVE; d <<= 1) {
        const uint64_t ol = shfl_xor(ulo, d), oh = shfl_xor(uhi, d);
        ulo = ol > ulo ? ol : ulo;
        uhi = oh > uhi ? oh : uhi;
      }
      if (lane == 0) {
        atomicMax(&s_jr[2 * pm], (unsigned long long)ulo);
        atomicMax(&s_jr[2 * pm + 1], (unsigned long long)uhi);
        atomicOr(&s_jp, 1ull << pm);
      }
    } else if (tp >= 0) {
      atomicMax(&s_jr[2 * tp], (unsigned long long)ulo);
      atomicMax(&s_jr[2 * tp + 1], (unsigned long long)uhi);
      atomicOr(&s_jp, 1ull << tp);
    }
  }
  const int nlists = a.waits ? PREP_LISTS : PREP_LISTS - 1;  // the op-name list only with its outputs
  if (tid < nlists) {
    uint32_t run = 0;
    for (int j = 0; j < PREP_ITEMS; ++j)
      for (int w = 0; w < PREP_THREADS / WAVE; ++w) {
        s_off[j][w][tid] = run;
        run += (uint32_t)popc(s_bal[j][w][tid]);
      }
    s_tot[tid] = run;
  }
  if (tid == 0 && s_bad != ~0ull) atomicMin((unsigned long long*)&a.ds->first_invalid, s_bad);
  __syncthreads();
  if (a.jt_range && tid < 2 * JT_PROCS && ((s_jp >> (tid >> 1)) & 1)) {
    unsigned long long* dst = (unsigned long long*)(tid & 1 ? &a.ds->jt_hi[tid >> 1] : &a.ds->jt_lo[tid >> 1]);
    atomicMax(dst, s_jr[tid]);
  }
  if (a.jt_range && tid == 0 && s_jp) atomicOr((unsigned long long*)&a.ds->jt_present, s_jp);
  if (wv < nlists) {
    const uint64_t ex = wave_lookback<OpSum>(a.status + (int64_t)wv * a.n_tiles, tile, s_tot[wv], a.ds);
    if (lane == 0) s_base[wv] = ex;
  }
  __syncthreads();
  if (tile == a.n_tiles - 1 && tid == 0) {
    const int64_t nK = (int64_t)(s_base[0] + s_tot[0]);
    const int64_t nC = (int64_t)(s_base[1] + s_tot[1]);
    const int64_t nJ = (int64_t)(s_base[2] + s_tot[2]);
    a.ds->nK = (int32_t)nK;
    a.ds->nCL = (int32_t)nC;
    a.ds->nJ = (int32_t)nJ;
    a.ds->nO = a.waits ? (int32_t)(s_base[3] + s_tot[3]) : 0;
    const int64_t nLaunch = nJ - nK;
    a.cnt->n_admitted[HERSCHEL_KERNEL] = nK;
    a.cnt->n_admitted[HERSCHEL_LAUNCH] = nLaunch;
    a.cnt->n_admitted[HERSCHEL_CPU_OP] = nC - nLaunch;
    a.cnt->n_outside_window = a.n - nK - nC;
  }
#pragma unroll
  for (int j = 0; j < PREP_ITEMS; ++j) {
    const uint32_t r = (uint32_t)(base + (int64_t)j * PREP_THREADS + tid);
    if (fl & (1u << (4 * j))) {
      const uint64_t pos = s_base[0] + s_off[j][wv][0] + popc(s_bal[j][wv][0] & lt);
      if (in_range(a.ds, (int64_t)pos, a.n)) {
        a.kK[pos] = kA[j];
        a.vK[pos] = r;
        a.kRows[pos] = r;
        if (a.waits) {  // the device lane: the timeline key without its stream
          a.kD[pos] = ((kA[j] >> (a.sb + a.wb)) << a.wb) | (kA[j] & ((1ull << a.wb) - 1));
          a.vD[pos] = r;
        }
      }
    }
    if (fl & (2u << (4 * j))) {
      const uint64_t pos = s_base[1] + s_off[j][wv][1] + popc(s_bal[j][wv][1] & lt);
      if (in_range(a.ds, (int64_t)pos, a.n)) {
        a.kC[pos] = kA[j];
        a.vC[pos] = r;
      }
    }
    if (fl & (4u << (4 * j))) {
      const uint64_t pos = s_base[2] + s_off[j][wv][2] + popc(s_bal[j][wv][2] & lt);
      if (in_range(a.ds, (int64_t)pos, a.n)) {
        a.kJ[pos] = kB[j];
        a.vJ[pos] = r;
      }
    }
    if (fl & (8u << (4 * j))) {
      const uint64_t pos = s_base[3] + s_off[j][wv][3] + popc(s_bal[j][wv][3] & lt);
      if (in_range(a.ds, (int64_t)pos, a.n)) {
        a.kO[pos] = kB[j];
        a.vO[pos] = r;
      }
    }
  }
}

void launch_prep(Ctx& c) {
  if (c.n == 0) return;
  PrepArgs a;
  a.ev = c.ev;
  a.n = c.n;
  a.off = c.p.clock_offset;
  a.W0 = c.W0;
  a.W1 = c.W1;
  a.P = c.P;
  a.S = c.S;
  a.T = c.T;
  a.NN = c.NN;
  a.NOP = c.NOP;
  a.sb = c.sb;
  a.tb = c.tb;
  a.wb = c.wb;
  a.n_tiles = c.prep_tiles;
  a.jt_range = c.P <= JT_PROCS;
  a.waits = c.waits;
  a.nob = c.nob;
  a.sol = c.sol;
  a.NG = c.NG;
  a.ds = c.ds;
  a.cnt = c.o.counters;
  a.link = c.o.link;
  a.aux = c.o.aux;
  a.status = c.prep_status;
  a.kK = c.sK.k[0];
  a.vK = c.sK.v[0];
  a.kRows = c.k_rows;
  a.kC = c.sC.k[0];
  a.vC = c.sC.v[0];
  a.kJ = c.jkey;
  a.vJ = c.jrow;
  a.kD = c.sD.k[0];
  a.vD = c.sD.v[0];
  a.kO = c.sO.k[0];
  a.vO = c.sO.v[0];
  hipLaunchKernelGGL(k_prep, dim3((unsigned)c.prep_tiles), dim3(PREP_THREADS), 0, c.st, a);
}

int64_t prep_tile_rows() { return PREP_TILE; }

}  // namespace hx
