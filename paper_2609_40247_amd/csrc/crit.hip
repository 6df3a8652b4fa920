// Critical path (Section 6.1, "Execution progress and state", and the
// critical-path figure): submission, execution-order and synchronization
// dependencies decide what each piece of the window waited for.
//
// Every admitted record x has a start event S(x) at ts' and an end event
// E(x) at min(te', W1); event ids are 2 * row + (0 start, 1 end).  Each
// event is released by at most one other event:
//   E(kernel) <- its S;
//   E(launch) <- E(g) when the launch has no kernel of its own and g, the
//                process's kernel ending last strictly inside the call
//                (largest end, then largest row), exists; else its S;
//   E(op)     <- E(last child) if that child ends no later; else its S;
//   S(kernel) <- the later release of E(previous kernel on its stream), if
//                it ended by the start, and its launch (E if it ended by
//                then, else S if it started by then); the launch on a tie;
//   S(op or launch) <- the later of E(previous sibling), if it ended by the
//                start, and S(parent); the sibling on a tie.
// Children and siblings follow the containment order of the thread.  The
// path of a process runs back from E of its last-ending record; each step's
// time difference is charged to a part (kernel, API, sync, op, and the
// unattributed launch, queue and host gaps) and, for the first four, to a
// record.
//
// Device form: one pass per list builds every event's release (the host
// records from the containment order and its answers, the kernels from the
// timeline order and the join, the synchronizing calls by a binary search
// in the kernels sorted by (pid, end)); then the path is marked in two
// levels.  Event ids are cut into tiles of CP_TE consecutive ids (a tile
// holds the rows of a few delivery blocks, so most releases stay inside
// it): a workgroup per tile follows the releases inside its tile in LDS and
// gives each event its exit, the first event of its release chain outside
// the tile; one thread per process walks the exits from its last event and
// marks each one (the entries of the path into tiles); a workgroup per tile
// that holds a marked entry marks its chain inside the tile.  A path with
// more than walk_max exits left after the walk is marked by pointer
// doubling over the exits from the marked ones (round r marks the exits
// 2^r steps behind while the pointers double, until a round adds nothing),
// and the tiles are marked again.  A last pass charges the marked steps.
#include "internal.hpp"

namespace hx {

enum : uint8_t {
  CP_KERNEL = 1,
  CP_API = 2,
  CP_SYNC = 3,
  CP_OP = 4,
  CP_LAUNCH_GAP = 5,
  CP_QUEUE_GAP = 6,
  CP_HOST_GAP = 7,
  CP_SELF = 1 << 3,  // the step is charged to the event's own record
  CP_PRED = 2 << 3   // ... to the record of the event it steps to
};
constexpr int CP_PARTS = 8;         // per process: length, then the seven parts
constexpr int CP_LDS_PROCS = 64;    // processes whose parts a workgroup sums in LDS

struct CritArgs {
  int64_t n;
  int P;
  const int64_t* ts;
  const int64_t* te;
  const int32_t* pid;
  const int64_t* off;
  int64_t W0, W1;
  int wb, wb1;
  int sb, tb;  // stream and thread bits of the timeline and containment keys
  DevState* ds;
  const uint64_t* kK[2];  // timeline order (pid, stream, ts')
  const uint32_t* vK[2];
  const uint64_t* kC[2];  // containment order (pid, thread, ts', launch)
  const uint32_t* vC[2];
  const uint64_t* kE[2];  // kernel ends (pid, min(te', W1) - W0)
  const uint32_t* vE[2];
  const int32_t* par;     // containment answers, by position
  const int32_t* link;
  const int32_t* aux;
  const uint32_t* k_rows;  // admitted kernels in row order
  uint64_t* eK;            // the kernel-end list before its sort
  uint32_t* eV;
  int32_t* pred;  // [2n] release of each event (-1 none)
  uint8_t* code;  // [2n] its part and whom it is charged to
  uint8_t* mark;  // [2n] on the path (zeroed with the state)
  int32_t* ptr0;  // [2n] doubling pointers, ping-pong
  int32_t* ptr1;
  uint32_t* lastc1;  // [n] by containment position: last child's position + 1 (zeroed)
  uint8_t* hasnext;  // [n] by containment position: a later sibling exists (zeroed)
  uint64_t* zmax;    // [P] largest end - W0 + 1 (zeroed)
  uint32_t* zrow1;   // [P] last-ending record's row + 1 (zeroed)
  int64_t* crit_time;
  uint8_t* crit_flags;
  int64_t* crit_proc;
  int round;
  int walk_max;  // exits a process's walk marks before the doubling takes over
  bool final;    // the path is completely marked when the charging pass runs
};

// Tiles of event ids for the two-level marking: CP_TE ids per workgroup of
// CP_LT threads, in LDS.
constexpr int CP_TE = 8192;
constexpr int CP_TE_LOG = 13;
constexpr int CP_LT = 512;
constexpr int CP_EPT = CP_TE / CP_LT;
static_assert((1 << CP_TE_LOG) == CP_TE && CP_EPT * CP_LT == CP_TE, "tile of event ids");
// the marking pass works on the few tiles the path enters: more threads, fewer events each
constexpr int CP_MLT = 1024;
constexpr int CP_MEPT = CP_TE / CP_MLT;
static_assert(CP_MEPT * CP_MLT == CP_TE, "marking tile");

__device__ __forceinline__ int64_t cp_off(const CritArgs& a, int32_t p) { return a.off ? a.off[p] : 0; }
__device__ __forceinline__ int64_t cp_start(const CritArgs& a, uint32_t r) { return a.ts[r] - cp_off(a, a.pid[r]); }
__device__ __forceinline__ int64_t cp_end(const CritArgs& a, uint32_t r) {
  const int64_t e = a.te[r] - cp_off(a, a.pid[r]);
  return e < a.W1 ? e : a.W1;
}
// The same for a record of process p whose clock offset o is known (records
// of one process share it): one gather instead of three dependent ones.
__device__ __forceinline__ int64_t cp_end_o(const CritArgs& a, uint32_t r, int64_t o) {
  const int64_t e = a.te[r] - o;
  return e < a.W1 ? e : a.W1;
}

// Each process's largest end: a workgroup folds its records' ends per
// process in LDS (a single process would otherwise put every record's
// atomic on one address) and adds one atomic per process it saw.
__device__ __forceinline__ void z_init(unsigned long long* s_z, int P) {
  if (P <= CP_LDS_PROCS)
    for (int i = threadIdx.x; i < CP_LDS_PROCS; i += blockDim.x) s_z[i] = 0;
  __syncthreads();
}
__device__ __forceinline__ void z_add1(const CritArgs& a, unsigned long long* s_z, int32_t p, unsigned long long v) {
  if (a.P <= CP_LDS_PROCS)
    atomicMax(&s_z[p], v);
  else
    atomicMax((unsigned long long*)&a.zmax[p], v);
}
// Called by every lane of the wave (valid or not): a wave whose valid lanes
// share one process adds its maximum once.
__device__ __forceinline__ void z_add(const CritArgs& a, unsigned long long* s_z, bool valid, int32_t p,
                                      int64_t end) {
  const uint64_t vb = ballot(valid);
  if (!vb) return;
  unsigned long long v = valid ? (unsigned long long)(end - a.W0 + 1) : 0ull;
  const int lead = __ffsll((long long)vb) - 1;
  const int32_t p0 = shfl(p, lead);
  if (ballot(valid && p != p0) == 0) {
    for (int d = 1; d < WAVE; d <<= 1) {
      const unsigned long long o = shfl_xor(v, d);
      v = o > v ? o : v;
    }
    if (lane_id() == lead) z_add1(a, s_z, p0, v);
  } else if (valid) {
    z_add1(a, s_z, p, v);
  }
}
__device__ __forceinline__ void z_flush(const CritArgs& a, unsigned long long* s_z) {
  if (a.P > CP_LDS_PROCS) return;
  __syncthreads();
  for (int i = threadIdx.x; i < a.P; i += blockDim.x)
    if (s_z[i]) atomicMax((unsigned long long*)&a.zmax[i], s_z[i]);
}

// The kernel-end list, from the admitted kernels in row order (the sort is
// stable, so kernels with equal ends stay in row order).
__global__ __launch_bounds__(256) void k_crit_elist(CritArgs a) {
  const int64_t cnt = a.ds->nK;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < cnt; i += (int64_t)gridDim.x * 256) {
    const uint32_t r = a.k_rows[i];
    a.eK[i] = ((uint64_t)a.pid[r] << a.wb1) | (uint64_t)(cp_end(a, r) - a.W0);
    a.eV[i] = r;
  }
}

// Host records, one per containment position: the start event's release,
// a launch's end event, each op's last child, each process's largest end.
__global__ __launch_bounds__(256) void k_crit_host(CritArgs a) {
  __shared__ unsigned long long s_z[CP_LDS_PROCS];
  z_init(s_z, a.P);
  const int64_t cnt = a.ds->nCL;
  const int pc = (int)a.ds->sort_parity[SORT_C], pe = (int)a.ds->sort_parity[SORT_E];
  const uint64_t* keys = a.kC[pc];
  const uint32_t* vals = a.vC[pc];
  const uint64_t* ekeys = a.kE[pe];
  const uint32_t* evals = a.vE[pe];
  const int64_t ne = a.ds->nK;
  const uint64_t emask = (1ull << a.wb1) - 1;
  for (int64_t q0 = (int64_t)blockIdx.x * 256; q0 < cnt; q0 += (int64_t)gridDim.x * 256) {  // uniform per workgroup
    const int64_t q = q0 + threadIdx.x;
    const bool valid = q < cnt;
    int32_t p = 0;
    int64_t te_ = 0, ts_ = 0;
    uint32_t r = 0;
    bool launch = false, sync = false;  // a launch; one without a kernel of its own
    uint64_t target = 0;
    if (valid) {
      r = vals[q];
      const uint64_t key = keys[q];
      const bool isop = (key & 1) == 0;
      const uint64_t seg = key >> (a.wb + 1);
      const int32_t pq = a.par[q];
      // previous sibling: up the answers from the position before, to a
      // record with the same parent (never past the parent itself)
      int64_t sibq = -1;
      int64_t j = q - 1;
      if (j >= 0 && (keys[j] >> (a.wb + 1)) == seg) {
        while (j >= 0 && in_range(a.ds, j, cnt) && j != pq && a.par[j] != pq) j = a.par[j];
        if (j >= 0 && j != pq) sibq = j;
      }
      // the key holds the process and the corrected start; the parent and
      // the sibling share the process, and so its clock offset
      p = (int32_t)(key >> (a.tb + a.wb + 1));
      const int64_t o = cp_off(a, p);
      ts_ = a.W0 + (int64_t)((key >> 1) & ((1ull << a.wb) - 1));
      te_ = cp_end_o(a, r, o);
      int32_t y = -1;
      uint8_t cd = 0;
      int64_t rel = I64MIN;
      if (pq >= 0) {
        const uint32_t pr = vals[pq];
        y = (int32_t)(2 * pr);
        cd = CP_OP | CP_PRED;
        rel = a.W0 + (int64_t)((keys[pq] >> 1) & ((1ull << a.wb) - 1));
      }
      if (sibq >= 0) {
        a.hasnext[sibq] = 1;  // not the last child of its parent
        const uint32_t sr = vals[sibq];
        const int64_t es = cp_end_o(a, sr, o);
        if (es <= ts_ && es >= rel) {
          y = (int32_t)(2 * sr + 1);
          cd = CP_HOST_GAP;
        }
      }
      a.pred[2 * r] = y;
      a.code[2 * r] = cd;
      launch = !isop;
      sync = launch && a.aux[r] == 0;  // no kernel of its own: a synchronizing call
      target = ((uint64_t)p << a.wb1) | (uint64_t)(te_ - a.W0);
    }
    // A synchronizing call's end waits for the process's kernel ending last
    // inside the call: the last kernel end below (process, the call's end)
    // in the sorted kernel ends.  The whole wave searches for one call at a
    // time, 64 ends per step (four dependent loads for a million kernels
    // instead of twenty).
    int64_t at = 0;  // first kernel end at or above the target
    uint64_t todo = ne > 0 ? ballot(sync) : 0ull;
    while (todo) {
      const int src = __ffsll((unsigned long long)todo) - 1;
      todo &= todo - 1;
      const uint64_t tg = shfl(target, src);
      int64_t lo = 0, hi = ne;  // every end below lo is below tg, every end from hi on is not
      while (hi - lo > WAVE) {
        const int64_t step = (hi - lo + WAVE - 1) / WAVE;
        const int64_t pos = lo + (int64_t)lane_id() * step;
        const bool in = pos < hi;
        const uint64_t kv = ekeys[in ? pos : lo];
        const int c = popc(ballot(in && kv < tg));
        const int nin = popc(ballot(in));
        const int64_t nlo = c > 0 ? lo + (int64_t)(c - 1) * step + 1 : lo;
        hi = c < nin ? lo + (int64_t)c * step : hi;
        lo = nlo;
      }
      const int64_t pos = lo + lane_id();
      const bool in = pos < hi;
      const uint64_t kv = ekeys[in ? pos : ne - 1];
      const int64_t found = lo + popc(ballot(in && kv < tg));
      if (lane_id() == src) at = found;
    }
    if (launch) {
      int32_t g = -1;
      if (sync && at > 0) {
        const uint64_t k = ekeys[at - 1];
        if ((k >> a.wb1) == (uint64_t)p && (int64_t)(k & emask) > ts_ - a.W0) g = (int32_t)evals[at - 1];
      }
      if (g >= 0) {
        a.pred[2 * r + 1] = 2 * g + 1;
        a.code[2 * r + 1] = CP_SYNC | CP_SELF;
      } else {
        a.pred[2 * r + 1] = (int32_t)(2 * r);
        a.code[2 * r + 1] = CP_API | CP_SELF;
      }
    }
    z_add(a, s_z, valid, p, te_);
  }
  z_flush(a, s_z);
}

// Kernels, one per timeline position (the timeline order and the join: no
// containment answer, so this pass runs beside the host records').
__global__ __launch_bounds__(256) void k_crit_kernels(CritArgs a) {
  __shared__ unsigned long long s_z[CP_LDS_PROCS];
  z_init(s_z, a.P);
  const int64_t cnt = a.ds->nK;
  const int pk = (int)a.ds->sort_parity[SORT_K];
  const uint64_t* keys = a.kK[pk];
  const uint32_t* vals = a.vK[pk];
  for (int64_t i0 = (int64_t)blockIdx.x * 256; i0 < cnt; i0 += (int64_t)gridDim.x * 256) {  // uniform per workgroup
    const int64_t i = i0 + threadIdx.x;
    const bool valid = i < cnt;
    int32_t p = 0;
    int64_t te_ = 0;
    if (valid) {
      const uint32_t r = vals[i];
      const int64_t kr = i > 0 && (keys[i - 1] >> a.wb) == (keys[i] >> a.wb) ? (int64_t)vals[i - 1] : -1;
      const int32_t L = a.link[r];
      // the key holds the process and the corrected start; the stream
      // predecessor and the launch share the process, and so its offset
      p = (int32_t)(keys[i] >> (a.sb + a.wb));
      const int64_t o = cp_off(a, p);
      const int64_t ts_ = a.W0 + (int64_t)(keys[i] & ((1ull << a.wb) - 1));
      te_ = cp_end_o(a, r, o);
      int32_t y = -1;
      uint8_t cd = 0;
      int64_t rel = I64MIN;
      if (kr >= 0) {
        const int64_t e = cp_end_o(a, (uint32_t)kr, o);
        if (e <= ts_) {
          y = (int32_t)(2 * kr + 1);
          cd = CP_QUEUE_GAP;
          rel = e;
        }
      }
      if (L >= 0) {
        const int64_t eL = cp_end_o(a, (uint32_t)L, o), sL = a.ts[L] - o;
        if (eL <= ts_) {
          if (eL >= rel) {
            y = 2 * L + 1;
            cd = CP_LAUNCH_GAP;
          }
        } else if (sL <= ts_ && sL >= rel) {
          y = 2 * L;
          cd = CP_API | CP_PRED;
        }
      }
      a.pred[2 * r] = y;
      a.code[2 * r] = cd;
      a.pred[2 * r + 1] = (int32_t)(2 * r);
      a.code[2 * r + 1] = CP_KERNEL | CP_SELF;
    }
    z_add(a, s_z, valid, p, te_);
  }
  z_flush(a, s_z);
}

// Each parent's last child (the child that is no other child's previous
// sibling, as the host pass has marked them), one per containment position.
__global__ __launch_bounds__(256) void k_crit_last(CritArgs a) {
  const int64_t ncl = a.ds->nCL;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < ncl; i += (int64_t)gridDim.x * 256)
    if (!a.hasnext[i]) {
      const int32_t pq = a.par[i];
      if (pq >= 0) a.lastc1[pq] = (uint32_t)(i + 1);
    }
}

// Ops' end events, once every last child is known.
__global__ __launch_bounds__(256) void k_crit_ops(CritArgs a) {
  const int64_t cnt = a.ds->nCL;
  const int pc = (int)a.ds->sort_parity[SORT_C];
  const uint64_t* keys = a.kC[pc];
  const uint32_t* vals = a.vC[pc];
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < cnt; q += (int64_t)gridDim.x * 256) {
    if (keys[q] & 1) continue;  // a launch
    const uint32_t r = vals[q];
    const int64_t lc = (int64_t)a.lastc1[q] - 1;
    int32_t y = (int32_t)(2 * r);
    if (lc >= 0 && in_range(a.ds, lc, cnt)) {
      const uint32_t lr = vals[lc];
      if (cp_end(a, lr) <= cp_end(a, r)) y = (int32_t)(2 * lr + 1);
    }
    a.pred[2 * r + 1] = y;
    a.code[2 * r + 1] = CP_OP | CP_SELF;
  }
}

// Rows: events of rows outside the window release nothing; the charged
// times start at zero; each process's last-ending record (largest end,
// then largest row).
__global__ __launch_bounds__(256) void k_crit_rows(CritArgs a) {
  for (int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x; r < a.n; r += (int64_t)gridDim.x * 256) {
    if (a.link[r] == -2) {
      a.pred[2 * r] = -1;
      a.pred[2 * r + 1] = -1;
      continue;
    }
    if (a.crit_time) a.crit_time[r] = 0;
    const int32_t p = a.pid[r];
    if ((uint64_t)(cp_end(a, (uint32_t)r) - a.W0 + 1) == a.zmax[p]) atomicMax(&a.zrow1[p], (uint32_t)(r + 1));
  }
}

// Each event's exit from its tile (into ptr1): the release of the last
// event of its release chain inside the tile (-1 where the chain ends in the
// tile).  In LDS every event points to its release inside the tile, or to
// itself when the release lies outside it or there is none; pointer jumping
// takes every event to the end of its chain inside the tile (at most CP_TE
// events: CP_TE_LOG rounds, fewer when a round changes nothing).
__global__ __launch_bounds__(CP_LT) void k_crit_local(CritArgs a) {
  __shared__ int32_t s_j[CP_TE];
  const int64_t ne = 2 * a.n;
  const int64_t tb = (int64_t)blockIdx.x * CP_TE;
  if (tb >= ne) return;
  const int tn = (int)min((int64_t)CP_TE, ne - tb);
  const int tid = threadIdx.x;
#pragma unroll
  for (int k = 0; k < CP_EPT; ++k) {
    const int i = tid + k * CP_LT;
    const int64_t y = i < tn ? (int64_t)a.pred[tb + i] : -1;
    s_j[i] = (y >= tb && y < tb + tn) ? (int)(y - tb) : i;
  }
  __syncthreads();
  for (int r = 0; r < CP_TE_LOG; ++r) {
    int32_t v[CP_EPT];
    bool ch = false;
#pragma unroll
    for (int k = 0; k < CP_EPT; ++k) {
      const int t = s_j[tid + k * CP_LT];
      v[k] = s_j[t];
      ch |= v[k] != t;
    }
    if (!__syncthreads_or(ch)) break;  // (also orders the reads before the writes)
#pragma unroll
    for (int k = 0; k < CP_EPT; ++k) s_j[tid + k * CP_LT] = v[k];
    __syncthreads();
  }
#pragma unroll
  for (int k = 0; k < CP_EPT; ++k) {
    const int i = tid + k * CP_LT;
    if (i < tn) a.ptr1[tb + i] = a.pred[tb + s_j[i]];
  }
}

// Each process's path from E of its last-ending record: the exits, walked
// one after another and marked (they are the path's entries into tiles).
// After walk_max exits the walk marks where it stands and leaves the rest to
// the doubling.
__global__ __launch_bounds__(256) void k_crit_walk(CritArgs a) {
  const int p = blockIdx.x * 256 + threadIdx.x;
  if (p >= a.P) return;
  const uint32_t z = a.zrow1[p];
  if (!z) return;
  const int64_t ne = 2 * a.n;
  int64_t e = 2 * (int64_t)(z - 1) + 1;
  for (int s = 0; e >= 0 && in_range(a.ds, e, ne); ++s) {
    a.mark[e] = 1;
    if (s >= a.walk_max) {
      atomicOr(&a.ds->crit_more, 1u);
      break;
    }
    e = a.ptr1[e];
  }
}

// The path inside each tile that holds a marked event: from every marked
// event, its release chain inside the tile, by pointer doubling in LDS
// (round r marks the events 2^r releases behind the marked ones).
__global__ __launch_bounds__(CP_MLT) void k_crit_mark_local(CritArgs a) {
  __shared__ int32_t s_j[CP_TE];
  __shared__ uint8_t s_m[CP_TE];
  const int64_t ne = 2 * a.n;
  const int64_t tb = (int64_t)blockIdx.x * CP_TE;
  if (tb >= ne) return;
  const int tn = (int)min((int64_t)CP_TE, ne - tb);
  const int tid = threadIdx.x;
  bool any = false;
#pragma unroll
  for (int k = 0; k < CP_MEPT; ++k) {
    const int i = tid + k * CP_MLT;
    const uint8_t m = i < tn ? a.mark[tb + i] : (uint8_t)0;
    s_m[i] = m;
    any |= m != 0;
  }
  if (!__syncthreads_or(any)) return;  // the path does not pass this tile
#pragma unroll
  for (int k = 0; k < CP_MEPT; ++k) {
    const int i = tid + k * CP_MLT;
    const int64_t y = i < tn ? (int64_t)a.pred[tb + i] : -1;
    s_j[i] = (y >= tb && y < tb + tn) ? (int)(y - tb) : i;
  }
  __syncthreads();
  for (int r = 0; r < CP_TE_LOG; ++r) {
    int32_t t[CP_MEPT], v[CP_MEPT];
    bool m[CP_MEPT];
    bool ch = false;
#pragma unroll
    for (int k = 0; k < CP_MEPT; ++k) {
      const int i = tid + k * CP_MLT;
      t[k] = s_j[i];
      v[k] = s_j[t[k]];
      m[k] = s_m[i] != 0;
      ch |= v[k] != t[k] || (m[k] && !s_m[t[k]]);
    }
    if (!__syncthreads_or(ch)) break;
#pragma unroll
    for (int k = 0; k < CP_MEPT; ++k) {
      if (m[k]) s_m[t[k]] = 1;
      s_j[tid + k * CP_MLT] = v[k];
    }
    __syncthreads();
  }
#pragma unroll
  for (int k = 0; k < CP_MEPT; ++k) {
    const int i = tid + k * CP_MLT;
    if (i < tn && s_m[i]) a.mark[tb + i] = 1;
  }
}

// One doubling round over the exits (only when a walk stopped short): every
// marked event marks the event its pointer names (2^round exits back), and
// every pointer is replaced by its target's.  A round after one that marked
// nothing does nothing: the path's entries are marked.
__global__ __launch_bounds__(256) void k_crit_round(CritArgs a) {
  const int rd = a.round;
  if (!a.ds->crit_more) return;
  if (rd > 0 && a.ds->crit_new[rd - 1] == 0) return;
  const int32_t* in = rd == 0 ? a.ptr1 : (rd & 1) ? a.ptr0 : a.ptr1;
  int32_t* out = (rd & 1) ? a.ptr1 : a.ptr0;
  const int64_t ne = 2 * a.n;
  for (int64_t i0 = (int64_t)blockIdx.x * 256; i0 < ne; i0 += (int64_t)gridDim.x * 256) {  // uniform per workgroup
    const int64_t i = i0 + threadIdx.x;
    bool added = false;
    if (i < ne) {
      const int32_t t = in[i];
      if (t >= 0 && in_range(a.ds, t, ne)) {
        if (a.mark[i] && !a.mark[t]) {
          a.mark[t] = 1;
          added = true;
        }
        out[i] = in[t];
      } else {
        out[i] = -1;
      }
    }
    const uint64_t b = ballot(added);
    if (b && lane_id() == 0) atomicAdd(&a.ds->crit_new[rd], (uint32_t)popc(b));
  }
}

// Charges: per row, each of its marked events' step; the root of each path
// gives its length.  Parts of up to CP_LDS_PROCS processes are summed in LDS.
// Each of the three outputs may be NULL.
__global__ __launch_bounds__(256) void k_crit_attr(CritArgs a) {
  __shared__ unsigned long long s_part[CP_LDS_PROCS * CP_PARTS];
  if (!a.final && a.ds->crit_more) return;  // the doubling comes first
  int64_t* const proc = a.crit_proc;
  const bool lds = proc && a.P <= CP_LDS_PROCS;
  if (lds)
    for (int i = threadIdx.x; i < CP_LDS_PROCS * CP_PARTS; i += 256) s_part[i] = 0;
  __syncthreads();
  for (int64_t r = (int64_t)blockIdx.x * 256 + threadIdx.x; r < a.n; r += (int64_t)gridDim.x * 256) {
    if (a.link[r] == -2) continue;
    const int32_t p = a.pid[r];
    uint8_t fl = 0;
#pragma unroll
    for (int side = 0; side < 2; ++side) {
      const int64_t e = 2 * r + side;
      if (!a.mark[e]) continue;
      fl |= (uint8_t)(1 << side);
      const int64_t t = side ? cp_end(a, (uint32_t)r) : cp_start(a, (uint32_t)r);
      const int32_t y = a.pred[e];
      if (y < 0) {  // the path's first event
        if (proc) proc[(int64_t)p * CP_PARTS] = (int64_t)(a.zmax[p] - 1) + a.W0 - t;
        continue;
      }
      const uint32_t yr = (uint32_t)(y >> 1);
      const int64_t d = t - ((y & 1) ? cp_end(a, yr) : cp_start(a, yr));
      const uint8_t cd = a.code[e];
      const int part = cd & 7, who = cd >> 3;
      if (a.crit_time && who) atomicAdd((unsigned long long*)&a.crit_time[who == 1 ? (uint32_t)r : yr],
                                        (unsigned long long)d);
      if (lds)
        atomicAdd(&s_part[p * CP_PARTS + part], (unsigned long long)d);
      else if (proc)
        atomicAdd((unsigned long long*)&proc[(int64_t)p * CP_PARTS + part], (unsigned long long)d);
    }
    if (a.crit_flags) a.crit_flags[r] = fl;
  }
  if (!lds) return;
  __syncthreads();
  for (int i = threadIdx.x; i < a.P * CP_PARTS; i += 256)
    if (s_part[i] && (i % CP_PARTS) != 0) atomicAdd((unsigned long long*)&proc[i], s_part[i]);
}

static CritArgs crit_args(Ctx& c) {
  CritArgs a;
  a.n = c.n;
  a.P = c.P;
  a.ts = c.ev.ts;
  a.te = c.ev.te;
  a.pid = c.ev.pid;
  a.off = c.p.clock_offset;
  a.W0 = c.W0;
  a.W1 = c.W1;
  a.wb = c.wb;
  a.wb1 = c.wb1;
  a.sb = c.sb;
  a.tb = c.tb;
  a.ds = c.ds;
  for (int b = 0; b < 2; ++b) {
    a.kK[b] = c.sK.k[b];
    a.vK[b] = c.sK.v[b];
    a.kC[b] = c.sC.k[b];
    a.vC[b] = c.sC.v[b];
    a.kE[b] = c.sE.k[b];
    a.vE[b] = c.sE.v[b];
  }
  a.par = c.par;
  a.link = c.o.link;
  a.aux = c.o.aux;
  a.k_rows = c.k_rows;
  a.eK = c.sE.k[0];
  a.eV = c.sE.v[0];
  a.pred = c.crit_pred;
  a.code = c.crit_code;
  a.mark = c.crit_mark;
  a.ptr0 = c.crit_ptr[0];
  a.ptr1 = c.crit_ptr[1];
  a.lastc1 = c.crit_lastc1;
  a.hasnext = c.crit_hasnext;
  a.zmax = c.crit_zmax;
  a.zrow1 = c.crit_zrow1;
  a.crit_time = c.o.crit_time;
  a.crit_flags = c.o.crit_flags;
  a.crit_proc = c.o.crit_proc;
  a.round = 0;
  a.walk_max = c.crit_walk_max;
  a.final = !c.crit_deferred;
  return a;
}

static unsigned crit_grid(int64_t work) {
  return (unsigned)std::max<int64_t>(std::min<int64_t>(cdiv(work, 256 * 4), 4096), 1);
}

void launch_crit_elist(Ctx& c) {
  if (c.n == 0) return;
  CritArgs a = crit_args(c);
  hipLaunchKernelGGL(k_crit_elist, dim3(crit_grid(c.n)), dim3(256), 0, c.st, a);
}

int crit_rounds(int64_t n) {
  int r = 1;
  while (r < CRIT_MAX_ROUNDS && ((int64_t)1 << (r - 1)) < 2 * n) ++r;
  return r;
}

// The doubling over the exits, the tiles marked again, the charges.
static void launch_crit_rest(Ctx& c, CritArgs a) {
  const int rounds = crit_rounds(c.n);
  for (int rd = 0; rd < rounds; ++rd) {
    a.round = rd;
    hipLaunchKernelGGL(k_crit_round, dim3(crit_grid(2 * c.n)), dim3(256), 0, c.st, a);
  }
  const unsigned tiles = (unsigned)cdiv(2 * c.n, CP_TE);
  hipLaunchKernelGGL(k_crit_mark_local, dim3(tiles), dim3(CP_MLT), 0, c.st, a);
  a.final = true;
  hipLaunchKernelGGL(k_crit_attr, dim3(crit_grid(c.n)), dim3(256), 0, c.st, a);
}

// With c.crit_deferred the doubling is left out: the charging pass then
// does nothing if a walk stopped short (DevState::crit_more), and the caller
// runs launch_crit_deferred once the call has ended.
void launch_crit_kernels(Ctx& c) {
  if (c.n == 0) return;
  hipLaunchKernelGGL(k_crit_kernels, dim3(crit_grid(c.n)), dim3(256), 0, c.st, crit_args(c));
}

void launch_crit_front(Ctx& c) {
  if (c.n == 0) return;
  CritArgs a = crit_args(c);
  hipLaunchKernelGGL(k_crit_host, dim3(crit_grid(c.n)), dim3(256), 0, c.st, a);
  hipLaunchKernelGGL(k_crit_last, dim3(crit_grid(c.n)), dim3(256), 0, c.st, a);
  hipLaunchKernelGGL(k_crit_ops, dim3(crit_grid(c.n)), dim3(256), 0, c.st, a);
}

void launch_crit(Ctx& c) {
  if (c.n == 0) return;
  CritArgs a = crit_args(c);
  hipLaunchKernelGGL(k_crit_rows, dim3(crit_grid(c.n)), dim3(256), 0, c.st, a);
  const unsigned tiles = (unsigned)cdiv(2 * c.n, CP_TE);
  hipLaunchKernelGGL(k_crit_local, dim3(tiles), dim3(CP_LT), 0, c.st, a);
  hipLaunchKernelGGL(k_crit_walk, dim3((unsigned)cdiv(c.P, 256)), dim3(256), 0, c.st, a);
  if (!c.crit_deferred) {
    launch_crit_rest(c, a);
    return;
  }
  hipLaunchKernelGGL(k_crit_mark_local, dim3(tiles), dim3(CP_MLT), 0, c.st, a);
  hipLaunchKernelGGL(k_crit_attr, dim3(crit_grid(c.n)), dim3(256), 0, c.st, a);
}

void launch_crit_deferred(Ctx& c) {
  if (c.n == 0) return;
  CritArgs a = crit_args(c);
  launch_crit_rest(c, a);
}

}  // namespace hx
