// Per-stream timelines: busy time, idle gaps and coverage runs.
//
// Input: the admitted kernels sorted by (pid, stream, ts').  A kernel covers
// [ts', min(te', W1)) (empty when te' == ts').  Walking a stream in start
// order with the running maximum M of the covered ends, a kernel starts a
// new coverage run iff its start lies beyond M, leaves the gap [M, ts')
// uncovered, and adds max(0, end - max(ts', M)) to the busy time -- the idle
// intervals of GPU activity that the case study of Section 9.1 starts from.
//
// The running maximum is a segmented max-scan (segments = streams) carried
// across tiles by a decoupled look-back; a second look-back pair compacts
// the gaps (in (pid, stream, begin) order, including the full-window gap of
// a stream without kernels) and the run endpoints used by the overlap sweep.
#include "internal.hpp"

namespace hx {

constexpr int UN_THREADS = 1024;
constexpr int UN_ITEMS = 4;
constexpr int UN_TILE = UN_THREADS * UN_ITEMS;
static_assert(UN_ITEMS % 4 == 0, "a thread's keys and rows are loaded 16 bytes at a time");

struct UnionArgs {
  const uint64_t* k[2];
  const uint32_t* v[2];
  const int64_t* te;
  const int32_t* pid_col;
  const int64_t* off;
  int64_t W0, W1, W, thr;
  int P, S, sb, wb, wb1, pb;
  bool overlap;
  DevState* ds;
  herschel_counters* cnt;
  int64_t* busy;
  int64_t gap_cap;
  int32_t* gap_pid;
  int32_t* gap_stream;
  int64_t* gap_begin;
  int64_t* gap_end;
  uint8_t* gap_flags;
  uint64_t* ev_keys;  // coverage run endpoints for the overlap stage
  int64_t ev_cap;
  uint64_t* status;   // [3][tiles_max]: segmax, gap count, event count
  int64_t tiles_max;
  // which list: its count, sort, tile ticket, and where its totals go
  const int32_t* count;
  int sort_id;
  int ticket;
  bool want_gaps;     // the op-name lanes need no gaps
  int64_t* gaps_out;  // the gap count
  int32_t* ev_out;    // the endpoint count
};

struct Elem {
  int32_t seg;    // pid * S + stream
  int64_t s, e;   // start and clipped end, relative to W0
};

__device__ __forceinline__ int32_t seg_of_key(const UnionArgs& a, uint64_t key) {
  const uint64_t segbits = key >> a.wb;
  return (int32_t)(segbits >> a.sb) * a.S + (int32_t)(segbits & ((1u << a.sb) - 1));
}

__device__ __forceinline__ void put_gap(const UnionArgs& a, int64_t pos, int32_t seg, int64_t b, int64_t e) {
  if (pos < a.gap_cap) {  // each gap array may be NULL
    if (a.gap_pid) a.gap_pid[pos] = seg / a.S;
    if (a.gap_stream) a.gap_stream[pos] = seg % a.S;
    if (a.gap_begin) a.gap_begin[pos] = a.W0 + b;
    if (a.gap_end) a.gap_end[pos] = a.W0 + e;
    if (a.gap_flags) a.gap_flags[pos] = (uint8_t)((b == 0 ? 1 : 0) | (e == a.W ? 2 : 0));
  }
}

// Events are staged in LDS at their position within the tile (the tile
// then writes them out whole, coalesced).
__device__ __forceinline__ void put_event(const UnionArgs& a, uint64_t* s_ev, int64_t pos, int32_t seg, int64_t t) {
  if (in_range(a.ds, pos, 2 * UN_TILE)) {
    const uint64_t pid = (uint64_t)(seg / a.S), stream = (uint64_t)(seg % a.S);
    s_ev[pos] = (pid << (a.wb1 + a.sb)) | ((uint64_t)t << a.sb) | stream;
  }
}

// Walks this thread's elements with the incoming carry.  MODE 0 counts gaps
// and events and accumulates busy time; MODE 1 writes gaps and events.
template <int MODE>
__device__ __forceinline__ void walk(const UnionArgs& a, const Elem* x, int nv, int32_t prev_seg, int32_t next_seg, uint64_t m_in,
                     int64_t i0, int64_t nK, uint32_t* ngap, uint32_t* nev, int64_t gbase, int64_t ebase,
                     int64_t* s_busy, int32_t seg0, uint64_t* s_ev) {
  const int nseg = a.P * a.S;
  const bool full_gap = a.want_gaps && a.W > a.thr;
  uint64_t m = m_in;  // 0 none, else (max covered end) + 1
  int32_t prev = prev_seg;
  uint32_t g = 0, v = 0;
  int64_t busy_acc = 0;
  int32_t busy_seg = -1;
#pragma unroll
  for (int j = 0; j < UN_ITEMS; ++j) {
    if (j >= nv) continue;
    const Elem& q = x[j];
    if (q.seg != prev) {
      if (full_gap) {  // empty streams strictly between
        for (int32_t s = prev + 1; s < q.seg; ++s) {
          if (MODE == 1) put_gap(a, gbase + g, s, 0, a.W);
          ++g;
        }
      }
      m = 0;
    }
    const int64_t C = m ? (int64_t)m - 1 : 0;
    if (q.e > q.s) {
      if (a.want_gaps && q.s > C && q.s - C > a.thr) {
        if (MODE == 1) put_gap(a, gbase + g, q.seg, C, q.s);
        ++g;
      }
      if (a.overlap && (m == 0 || q.s > C)) {
        if (m != 0) {
          if (MODE == 1) put_event(a, s_ev, ebase + v, q.seg, C);
          ++v;
        }
        if (MODE == 1) put_event(a, s_ev, ebase + v, q.seg, q.s);
        ++v;
      }
      if (MODE == 0) {
        const int64_t lo = q.s > C ? q.s : C;
        if (q.e > lo) {
          if (busy_seg != q.seg) {
            if (busy_seg >= 0 && busy_acc) {
              if (busy_seg - seg0 < 64) atomicAdd((unsigned long long*)&s_busy[busy_seg - seg0], (unsigned long long)busy_acc);
              else atomicAdd((unsigned long long*)&a.busy[busy_seg], (unsigned long long)busy_acc);
            }
            busy_seg = q.seg;
            busy_acc = 0;
          }
          busy_acc += q.e - lo;
        }
      }
      const uint64_t me = (uint64_t)q.e + 1;
      m = me > m ? me : m;
    }
    const int32_t nxt = (j + 1 < nv) ? x[j + 1].seg : next_seg;
    if (nxt != q.seg) {
      const int64_t Cl = m ? (int64_t)m - 1 : 0;
      if (a.want_gaps && Cl < a.W && a.W - Cl > a.thr) {
        if (MODE == 1) put_gap(a, gbase + g, q.seg, Cl, a.W);
        ++g;
      }
      if (a.overlap && m != 0) {
        if (MODE == 1) put_event(a, s_ev, ebase + v, q.seg, Cl);
        ++v;
      }
      if (full_gap && i0 + j == nK - 1) {
        for (int32_t s = q.seg + 1; s < nseg; ++s) {
          if (MODE == 1) put_gap(a, gbase + g, s, 0, a.W);
          ++g;
        }
      }
    }
    prev = q.seg;
  }
  if (MODE == 0 && busy_seg >= 0 && busy_acc) {
    if (busy_seg - seg0 < 64) atomicAdd((unsigned long long*)&s_busy[busy_seg - seg0], (unsigned long long)busy_acc);
    else atomicAdd((unsigned long long*)&a.busy[busy_seg], (unsigned long long)busy_acc);
  }
  *ngap = g;
  *nev = v;
}

__global__ __launch_bounds__(UN_THREADS) void k_union(UnionArgs a) {
  __shared__ int s_tile;
  __shared__ uint64_t s_wv[UN_THREADS / WAVE];
  __shared__ int s_wh[UN_THREADS / WAVE];
  __shared__ uint64_t s_tile_excl;
  __shared__ int64_t s_busy[64];
  __shared__ int32_t s_seg0;
  __shared__ uint32_t s_scan[UN_THREADS / WAVE + 1];
  __shared__ uint32_t s_tot[2];
  __shared__ uint64_t s_base[2];
  __shared__ uint64_t s_ev[2 * UN_TILE];  // the tile's coverage-run endpoints, in order

  const int tid = threadIdx.x, lane = lane_id(), wv = tid / WAVE;
  const int64_t nK = *a.count;
  const int par = (int)a.ds->sort_parity[a.sort_id];
  const uint64_t* keys = a.k[par];
  const uint32_t* vals = a.v[par];
  const int64_t ntiles = nK > 0 ? cdiv(nK, UN_TILE) : 1;
  if ((int64_t)blockIdx.x >= ntiles) return;  // no tile: stay off the ticket counter
  const int tile = take_ticket(a.ds, a.ticket, &s_tile);
  const int64_t base = (int64_t)tile * UN_TILE;
  const int nseg = a.P * a.S;

  if (nK == 0) {  // no kernels: one full-window gap per stream
    const bool full_gap = a.want_gaps && a.W > a.thr;
    for (int s = tid; s < nseg; s += UN_THREADS)
      if (full_gap) put_gap(a, s, s, 0, a.W);
    if (tid == 0) {
      *a.gaps_out = full_gap ? nseg : 0;
      if (a.cnt) a.cnt->n_gaps_total = full_gap ? nseg : 0;
      *a.ev_out = 0;
    }
    return;
  }

  if (tid < 64) s_busy[tid] = 0;
  if (tid == 0) s_seg0 = seg_of_key(a, keys[base]);

  // The thread's UN_ITEMS consecutive keys and rows (16-byte loads when the
  // thread's group lies inside the list, clamped single loads at its end),
  // then every end-time and clock-offset gather, so that each round of loads
  // is in flight together.
  const int64_t i0 = base + (int64_t)tid * UN_ITEMS;
  const int nv = nK - i0 >= UN_ITEMS ? UN_ITEMS : nK - i0 > 0 ? (int)(nK - i0) : 0;
  uint64_t kv[UN_ITEMS];
  uint32_t rv[UN_ITEMS];
  if (nv == UN_ITEMS) {
    const uint4* kp = reinterpret_cast<const uint4*>(keys + i0);
    const uint4* rp = reinterpret_cast<const uint4*>(vals + i0);
#pragma unroll
    for (int h = 0; h < UN_ITEMS / 2; ++h) {
      const uint4 w = kp[h];
      kv[2 * h] = (uint64_t)w.x | ((uint64_t)w.y << 32);
      kv[2 * h + 1] = (uint64_t)w.z | ((uint64_t)w.w << 32);
    }
#pragma unroll
    for (int h = 0; h < UN_ITEMS / 4; ++h) {
      const uint4 w = rp[h];
      rv[4 * h] = w.x;
      rv[4 * h + 1] = w.y;
      rv[4 * h + 2] = w.z;
      rv[4 * h + 3] = w.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < UN_ITEMS; ++j) {
      const int64_t idx = i0 + j < nK ? i0 + j : nK - 1;
      kv[j] = keys[idx];
      rv[j] = vals[idx];
    }
  }
  const bool has = nv > 0;
  const int64_t iprev = i0 < nK ? i0 - 1 : nK - 1, inext = i0 + nv < nK ? i0 + nv : nK - 1;
  const uint64_t kprev = keys[iprev > 0 ? iprev : 0];
  const uint64_t knext = keys[inext];
  int64_t tev[UN_ITEMS], offv[UN_ITEMS];
#pragma unroll
  for (int j = 0; j < UN_ITEMS; ++j) tev[j] = a.te[rv[j]];
#pragma unroll
  for (int j = 0; j < UN_ITEMS; ++j) offv[j] = a.off ? a.off[(int32_t)((kv[j] >> a.wb) >> a.sb)] : 0;
  Elem x[UN_ITEMS];
#pragma unroll
  for (int j = 0; j < UN_ITEMS; ++j) {
    if (j < nv) {
      x[j].seg = seg_of_key(a, kv[j]);
      x[j].s = (int64_t)(kv[j] & ((1ull << a.wb) - 1));
      const int64_t tec = tev[j] - offv[j];  // corrected end; may lie far beyond W1
      x[j].e = tec >= a.W1 ? a.W : tec - a.W0;
    } else {
      x[j].seg = -1;
      x[j].s = x[j].e = 0;
    }
  }
  const int32_t prev_seg = (has && i0 > 0) ? seg_of_key(a, kprev) : -1;
  const int32_t next_seg = (has && i0 + nv < nK) ? seg_of_key(a, knext) : -1;

  // Thread aggregate for the segmented max-scan.
  uint64_t agg = 0;
  if (has) {
    bool head = false;
    uint64_t m = 0;
    int32_t prev = prev_seg;
#pragma unroll
    for (int j = 0; j < UN_ITEMS; ++j) {
      if (j >= nv) continue;
      if (x[j].seg != prev) {
        head = true;
        m = 0;
      }
      if (x[j].e > x[j].s) {
        const uint64_t me = (uint64_t)x[j].e + 1;
        m = me > m ? me : m;
      }
      prev = x[j].seg;
    }
    int32_t last_seg = x[0].seg;
#pragma unroll
    for (int j = 1; j < UN_ITEMS; ++j)
      if (j < nv) last_seg = x[j].seg;
    agg = OpSegMax::make((uint32_t)last_seg, head, m);
  }
  // Ordered inclusive scan over the wave (valid threads form a prefix).
  uint64_t inc = agg;
  bool hv = has;
  for (int d = 1; d < WAVE; d <<= 1) {
    const uint64_t o = shfl_up(inc, d);
    const int oh = shfl_up((int)hv, d);
    if (lane >= d && oh) {
      inc = hv ? OpSegMax::combine(o, inc) : o;
      hv = true;
    }
  }
  // every lane takes part in the shuffles; lane 0 discards the result
  const uint64_t lane_excl = shfl_up(inc, 1);
  const int prev_hv = shfl_up((int)hv, 1);
  const bool lane_excl_has = lane > 0 && prev_hv;
  if (lane == WAVE - 1) {
    s_wv[wv] = inc;
    s_wh[wv] = hv;
  }
  __syncthreads();
  if (tid == 0) {
    uint64_t run = 0;
    bool rh = false;
    for (int w = 0; w < UN_THREADS / WAVE; ++w) {
      const uint64_t t = s_wv[w];
      const bool th = s_wh[w];
      s_wv[w] = run;
      s_wh[w] = rh;
      if (th) {
        run = rh ? OpSegMax::combine(run, t) : t;
        rh = true;
      }
    }
    s_tile_excl = run;  // tile aggregate (temporarily)
  }
  __syncthreads();
  if (wv == 0) {
    const uint64_t ex = wave_lookback<OpSegMax>(a.status, tile, s_tile_excl, a.ds);
    if (lane == 0) s_tile_excl = ex;
  }
  __syncthreads();
  // Exclusive prefix for this thread: tile prefix, then waves, then lanes.
  uint64_t pre = s_tile_excl;
  bool pre_has = tile > 0;
  if (s_wh[wv]) {
    pre = pre_has ? OpSegMax::combine(pre, s_wv[wv]) : s_wv[wv];
    pre_has = true;
  }
  if (lane_excl_has) {
    pre = pre_has ? OpSegMax::combine(pre, lane_excl) : lane_excl;
    pre_has = true;
  }
  const uint64_t m_in = (has && pre_has && (int32_t)OpSegMax::seg(pre) == x[0].seg) ? OpSegMax::m(pre) : 0;

  uint32_t ngap = 0, nev = 0;
  if (has) walk<0>(a, x, nv, prev_seg, next_seg, m_in, i0, nK, &ngap, &nev, 0, 0, s_busy, s_seg0, s_ev);
  uint32_t gtot, etot;
  const uint32_t gex = block_excl_sum<UN_THREADS>(ngap, s_scan, &gtot);
  const uint32_t eex = block_excl_sum<UN_THREADS>(nev, s_scan, &etot);
  if (tid == 0) {
    s_tot[0] = gtot;
    s_tot[1] = etot;
  }
  __syncthreads();
  if (wv < 2) {
    const uint64_t ex = wave_lookback<OpSum>(a.status + (int64_t)(1 + wv) * a.tiles_max, tile, s_tot[wv], a.ds);
    if (lane == 0) s_base[wv] = ex;
  }
  if (tid < 64 && s_busy[tid]) atomicAdd((unsigned long long*)&a.busy[s_seg0 + tid], (unsigned long long)s_busy[tid]);
  __syncthreads();
  if (tile == ntiles - 1 && tid == 0) {
    const int64_t g = (int64_t)(s_base[0] + s_tot[0]);
    *a.gaps_out = g;
    if (a.cnt) a.cnt->n_gaps_total = g;
    *a.ev_out = (int32_t)(s_base[1] + s_tot[1]);
  }
  if (has && (ngap || nev)) {
    uint32_t g2, e2;
    walk<1>(a, x, nv, prev_seg, next_seg, m_in, i0, nK, &g2, &e2, (int64_t)s_base[0] + gex, (int64_t)eex, s_busy, s_seg0,
            s_ev);
  }
  __syncthreads();
  const uint32_t ne = s_tot[1];
  const int64_t eb = (int64_t)s_base[1];
  for (uint32_t i = tid; i < ne; i += UN_THREADS)
    if (in_range(a.ds, eb + i, a.ev_cap)) a.ev_keys[eb + i] = s_ev[i];
}

static UnionArgs union_args(Ctx& c, const SortBufs& sb_, int S, int sbits) {
  UnionArgs a;
  a.k[0] = sb_.k[0];
  a.k[1] = sb_.k[1];
  a.v[0] = sb_.v[0];
  a.v[1] = sb_.v[1];
  a.te = c.ev.te;
  a.pid_col = c.ev.pid;
  a.off = c.p.clock_offset;
  a.W0 = c.W0;
  a.W1 = c.W1;
  a.W = c.W;
  a.thr = c.thr;
  a.P = c.P;
  a.S = S;
  a.sb = sbits;
  a.wb = c.wb;
  a.wb1 = c.wb1;
  a.pb = c.pb;
  a.ds = c.ds;
  a.tiles_max = c.union_tiles;
  a.sort_id = sb_.id;
  a.want_gaps = true;
  return a;
}

// Busy time, gaps and coverage-run endpoints of every (pid, stream).
void launch_timeline(Ctx& c) {
  UnionArgs a = union_args(c, c.sK, c.S, c.sb);
  a.overlap = c.overlap;
  a.cnt = c.o.counters;
  a.busy = c.o.busy ? c.o.busy : c.busy_ws;
  a.gap_cap = c.o.gap_capacity;
  a.gap_pid = c.o.gap_pid;
  a.gap_stream = c.o.gap_stream;
  a.gap_begin = c.o.gap_begin;
  a.gap_end = c.o.gap_end;
  a.gap_flags = c.o.gap_flags;
  a.ev_keys = c.ev_keys;
  a.ev_cap = c.ev_cap;
  a.status = c.union_status;
  a.count = &c.ds->nK;
  a.ticket = TK_UNION;
  a.gaps_out = &c.ds->n_gaps;
  a.ev_out = &c.ds->nEv;
  hipLaunchKernelGGL(k_union, dim3((unsigned)c.union_tiles), dim3(UN_THREADS), 0, c.st, a);
}

// The same scan over the device lane (every stream of a process at once):
// its gaps above the threshold are the GPU's idle intervals, in (pid, begin)
// order; and over the op-name lanes, whose busy time is each op name's span
// and whose coverage-run endpoints bound its union.
void launch_union_device(Ctx& c) {
  UnionArgs d = union_args(c, c.sD, 1, 0);
  d.overlap = false;
  d.cnt = nullptr;
  d.busy = c.dbusy_ws;
  d.gap_cap = c.dg_cap;
  d.gap_pid = c.dg_pid;
  d.gap_stream = nullptr;
  d.gap_begin = c.dg_begin;
  d.gap_end = c.dg_end;
  d.gap_flags = nullptr;
  d.ev_keys = nullptr;
  d.ev_cap = 0;
  d.status = c.union_status_d;
  d.count = &c.ds->nK;
  d.ticket = TK_UNION_D;
  d.gaps_out = &c.ds->nDgap;
  d.ev_out = &c.ds->nDev;
  hipLaunchKernelGGL(k_union, dim3((unsigned)c.union_tiles), dim3(UN_THREADS), 0, c.st, d);
}

void launch_union_opnames(Ctx& c) {
  UnionArgs o = union_args(c, c.sO, c.NOP, c.nob);
  o.overlap = true;
  o.want_gaps = false;
  o.cnt = nullptr;
  o.busy = c.o.op_span ? c.o.op_span : c.op_span_ws;
  o.gap_cap = 0;
  o.gap_pid = nullptr;
  o.gap_stream = nullptr;
  o.gap_begin = nullptr;
  o.gap_end = nullptr;
  o.gap_flags = nullptr;
  o.ev_keys = c.oev;
  o.ev_cap = c.oev_cap;
  o.status = c.union_status_o;
  o.count = &c.ds->nO;
  o.ticket = TK_UNION_O;
  o.gaps_out = &c.ds->nOgap;
  o.ev_out = &c.ds->nOev;
  hipLaunchKernelGGL(k_union, dim3((unsigned)c.union_tiles), dim3(UN_THREADS), 0, c.st, o);
}

int64_t union_tile_elems() { return UN_TILE; }

}  // namespace hx
