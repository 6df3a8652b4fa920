// Containment: op nesting, launch -> op, per-op inclusive aggregates.
//
// Kernel composition (Section 6.1) needs each launch's enclosing Python call
// and each call's parent; calls are recorded with their native thread and
// nest (Section 5.2).  With the admitted ops and launches of a thread sorted
// by (ts' up, te' down, row up; ops before launches at equal ts'), the parent
// of an op and the op of a launch are both "the nearest earlier op whose end
// lies after my start".  That is a previous-greater query: every op stores
// V = (thread segment, min(te', W1)) packed so that one unsigned comparison
// against (my segment, my ts') decides both "same thread" and "ends after my
// start"; launches store 0.  A 64-ary max pyramid over V (levels in LDS for
// the tile, in HBM above it) and an exclusive prefix max per position answer
// the query by walking back only as far as the answer.
//
// The answers form a forest whose preorder is the sorted order, so the
// subtree of an op is a contiguous range.  Inclusive aggregates (T_op: first
// kernel start, last kernel end, Section 6.1) are accumulated per tile in
// LDS; only the few ops still open at a tile edge go through global atomics.
#include "internal.hpp"

namespace hx {

constexpr int CT_THREADS = 256;
constexpr int CT_ITEMS = 16;
constexpr int CT_TILE = CT_THREADS * CT_ITEMS;  // 4096 positions = one M2 entry
static_assert(CT_TILE == 64 * 64, "a containment tile is one entry of pyramid level 2");

struct ContainArgs {
  uint64_t* k[2];
  uint32_t* v[2];
  const int64_t* ts;
  const int64_t* te;
  const int64_t* off;
  int64_t W0, W1, W;
  int tb, wb, vb;
  DevState* ds;
  herschel_counters* cnt;
  int32_t* link;
  int32_t* aux;
  int32_t* op_nkern;
  int64_t* op_first;
  int64_t* op_last;
  int64_t* op_ksum;
  uint64_t* V;
  uint64_t* M[6];
  int64_t Mn[6];
  int nlev;
  uint64_t* pmt;
  uint64_t* vb_status;
  int32_t* par;
  // per-launch kernel aggregates (by row), written by the join
  const int64_t* lk_first;
  const int64_t* lk_last;
  const int64_t* lk_sum;
  // per aggregate tile: the ops open at its start (innermost first) and their number
  int32_t* ag_chain;
  int32_t* ag_nchain;
  int64_t ag_tiles;
};

__device__ __forceinline__ int32_t key_pid(const ContainArgs& a, uint64_t key) {
  return (int32_t)(key >> (a.tb + a.wb + 1));
}
__device__ __forceinline__ uint64_t key_seg(const ContainArgs& a, uint64_t key) { return key >> (a.wb + 1); }
__device__ __forceinline__ int64_t key_rel(const ContainArgs& a, uint64_t key) {
  return (int64_t)((key >> 1) & ((1ull << a.wb) - 1));
}
__device__ __forceinline__ bool key_is_op(uint64_t key) { return (key & 1) == 0; }

// Per-op outputs (each may be NULL): a plain store of whole aggregates, or
// atomic combination into ones that start at the identities.
__device__ __forceinline__ void op_store(const ContainArgs& a, uint32_t rr, int32_t nk, int64_t f, int64_t l,
                                         int64_t sm) {
  if (a.op_nkern) a.op_nkern[rr] = nk;
  if (a.op_first) a.op_first[rr] = f;
  if (a.op_last) a.op_last[rr] = l;
  if (a.op_ksum) a.op_ksum[rr] = sm;
}
__device__ __forceinline__ void op_combine(const ContainArgs& a, uint32_t rr, uint32_t nk, int64_t f, int64_t l,
                                           uint64_t sm) {
  if (a.op_nkern) atomicAdd(&a.op_nkern[rr], (int32_t)nk);
  if (a.op_first) atomicMin((long long*)&a.op_first[rr], (long long)f);
  if (a.op_last) atomicMax((long long*)&a.op_last[rr], (long long)l);
  if (a.op_ksum) atomicAdd((unsigned long long*)&a.op_ksum[rr], (unsigned long long)sm);
}

// ------------------------------------------------------- encoding, pyramid
// V and the first pyramid levels of one 4096-position tile: 16 waves, each
// wave four 64-position groups (one M1 entry each), every round of loads
// (keys, rows, end times) issued for all four groups together.  The tile
// maximum is M2; the levels above it take atomic maxima (they start at
// zero); the exclusive prefix maximum over earlier tiles comes from a
// decoupled look-back.
constexpr int VB_THREADS = 1024;
constexpr int VB_ITEMS = CT_TILE / VB_THREADS;

__global__ __launch_bounds__(VB_THREADS) void k_vbuild(ContainArgs a) {
  __shared__ uint64_t s_w[VB_THREADS / WAVE];
  __shared__ uint64_t s_tmax;
  const int tid = threadIdx.x, lane = lane_id(), wv = tid / WAVE;
  const int64_t n = a.ds->nCL;
  const int par = (int)a.ds->sort_parity[1];
  const uint64_t* keys = a.k[par];
  const uint32_t* vals = a.v[par];
  if ((int64_t)blockIdx.x * CT_TILE >= n) return;
  const int tile = blockIdx.x;
  const int64_t base = (int64_t)tile * CT_TILE;
  // item j of lane covers position base + wv*256 + j*64 + lane
  uint64_t key[VB_ITEMS];
  uint32_t row[VB_ITEMS];
  int64_t te[VB_ITEMS];
  // each round of loads is issued for all items together: indices are
  // clamped (to the last position, or row 0), never branched on
#pragma unroll
  for (int j = 0; j < VB_ITEMS; ++j) {
    const int64_t p = base + (int64_t)wv * (VB_ITEMS * WAVE) + j * WAVE + lane;
    const int64_t pc = p < n ? p : n - 1;
    key[j] = keys[pc];
    row[j] = vals[pc];
  }
#pragma unroll
  for (int j = 0; j < VB_ITEMS; ++j) {
    const int64_t p = base + (int64_t)wv * (VB_ITEMS * WAVE) + j * WAVE + lane;
    if (!(p < n && key_is_op(key[j]))) row[j] = ~0u;
  }
  int64_t offv[VB_ITEMS];
#pragma unroll
  for (int j = 0; j < VB_ITEMS; ++j) {
    te[j] = a.te[row[j] != ~0u ? row[j] : 0u];
    offv[j] = a.off ? a.off[key_pid(a, key[j])] : 0;
  }
  uint64_t wmax = 0;
#pragma unroll
  for (int j = 0; j < VB_ITEMS; ++j) {
    const int64_t p = base + (int64_t)wv * (VB_ITEMS * WAVE) + j * WAVE + lane;
    uint64_t v = 0;
    if (row[j] != ~0u) {
      const int64_t tec = te[j] - offv[j];
      const int64_t e = tec >= a.W1 ? a.W : tec - a.W0;
      v = (key_seg(a, key[j]) << a.vb) | (uint64_t)(e + 1);
    }
    if (p < n) a.V[p] = v;
    const uint64_t g = wave_allmax_u64(v);
    if (lane == 0 && p - lane < n) a.M[1][(p - lane) >> 6] = g;
    wmax = g > wmax ? g : wmax;
  }
  if (lane == 0) s_w[wv] = wmax;
  __syncthreads();
  if (tid == 0) {
    uint64_t t = 0;
    for (int w = 0; w < VB_THREADS / WAVE; ++w) t = s_w[w] > t ? s_w[w] : t;
    s_tmax = t;
    a.M[2][tile] = t;
    for (int l = 3; l < a.nlev; ++l)
      if (t) atomicMax((unsigned long long*)&a.M[l][tile >> (6 * (l - 2))], (unsigned long long)t);
  }
  __syncthreads();
  if (wv == 0) {
    const uint64_t ex = wave_lookback<OpMax>(a.vb_status, tile, s_tmax, a.ds);
    if (lane == 0) a.pmt[tile] = ex;
  }
}

// Live entries of pyramid level l for n positions.
__device__ __forceinline__ int64_t live(int64_t n, int l) {
  int64_t c = n;
  for (int i = 0; i < l; ++i) c = cdiv(c, 64);
  return c;
}

// Answer of a query whose answer lies before its tile: one wave climbs the
// pyramid from level 2 and descends, loading 64 entries per step and taking
// the highest lane above q with a ballot.  Called by a whole wave.
__device__ int64_t wave_escape(const ContainArgs& a, int64_t tile, uint64_t q, int64_t n) {
  const int lane = lane_id();
  int l = 2;
  int64_t idx = tile;
  int64_t f = -1;
  while (l < a.nlev) {
    const int64_t lo = (idx >> 6) << 6;
    const int64_t e = lo + lane;
    const uint64_t v = e < idx ? a.M[l][e] : 0ull;
    const uint64_t b = ballot(v > q);
    if (b) {
      f = lo + 63 - __clzll((long long)b);
      break;
    }
    idx >>= 6;
    ++l;
  }
  if (f < 0) return -1;  // only when the prefix maximum said otherwise
  while (l > 0) {
    const uint64_t* lower = l - 1 == 0 ? a.V : a.M[l - 1];
    const int64_t lo = f * 64;
    const int64_t hi = min(lo + 64, live(n, l - 1));
    const int64_t e = lo + lane;
    const uint64_t v = e < hi ? lower[e] : 0ull;
    const uint64_t b = ballot(v > q);
    if (!b) return -1;
    f = lo + 63 - __clzll((long long)b);
    --l;
  }
  return f;
}

// Largest j <= pos whose value exceeds q, given the wave's window maxima
// w[k] = max(v[l - 2^k + 1 .. l]) held by every lane l (k = 0..5): skip
// windows with no value above q, widest first.  -1 when there is none.
__device__ __forceinline__ int wave_lift(const uint64_t (&w)[6], int pos, uint64_t q) {
#pragma unroll
  for (int k = 5; k >= 0; --k) {
    const int src = pos < 0 ? 0 : pos;
    const uint64_t wm = __shfl(w[k], src, WAVE);  // every lane takes part
    if (pos - (1 << k) + 1 >= 0 && wm <= q) pos -= 1 << k;
  }
  return pos;
}

// One workgroup per 4096-position tile, 16 waves: a wave answers four
// 64-position groups, one lane per position.  Keys, rows and values of the
// tile are loaded up front; inside the tile every step reads LDS.
constexpr int QY_THREADS = 1024;
constexpr int QY_GROUPS = CT_TILE / 64;                  // 64 groups per tile
constexpr int QY_ROUNDS = QY_GROUPS / (QY_THREADS / WAVE);  // groups per wave
static_assert(QY_GROUPS == WAVE && QY_GROUPS % (QY_THREADS / WAVE) == 0, "one lane per group of the tile");
static_assert(CT_TILE <= 65536, "escaping positions are kept as 16-bit tile offsets");

__global__ __launch_bounds__(QY_THREADS) void k_query(ContainArgs a) {
  __shared__ uint64_t s_v[CT_TILE];
  __shared__ uint32_t s_val[CT_TILE];
  __shared__ uint64_t s_sub[CT_TILE / 8];   // maxima of 8-position blocks
  __shared__ uint64_t s_g[6][QY_GROUPS];    // window maxima over the tile's groups
  __shared__ uint64_t s_gpre[QY_GROUPS];    // max over the tile's earlier groups and all earlier tiles
  __shared__ uint16_t s_esc[CT_TILE];
  __shared__ uint64_t s_prev[QY_GROUPS];    // group maxima of the previous tile (its M1 entries)
  __shared__ int s_nesc;
  const int tid = threadIdx.x, lane = lane_id(), wv = tid / WAVE;
  const int64_t n = a.ds->nCL;
  const int par = (int)a.ds->sort_parity[1];
  const uint64_t* keys = a.k[par];
  const uint32_t* vals = a.v[par];
  const int64_t tile = blockIdx.x;
  const int64_t base = tile * CT_TILE;
  if (base >= n) return;
  const int64_t tn = min((int64_t)CT_TILE, n - base);
  const int ng = (int)cdiv(tn, 64);
  uint64_t key[QY_ROUNDS];
  uint32_t row[QY_ROUNDS];
  uint64_t vv[QY_ROUNDS];
#pragma unroll
  for (int r = 0; r < QY_ROUNDS; ++r) {
    const int lp = (wv + r * (QY_THREADS / WAVE)) * 64 + lane;
    const int64_t pc = base + (lp < tn ? lp : tn - 1);  // clamped: the loads stay in flight together
    key[r] = keys[pc];
    row[r] = vals[pc];
    vv[r] = a.V[pc];
  }
#pragma unroll
  for (int r = 0; r < QY_ROUNDS; ++r) {
    const int lp = (wv + r * (QY_THREADS / WAVE)) * 64 + lane;
    const bool live = lp < tn;
    if (!live) {
      key[r] = 0ull;
      row[r] = 0u;
    }
    s_v[lp] = live ? vv[r] : 0ull;
    s_val[lp] = row[r];
  }
  if (tid == 0) s_nesc = 0;
  __syncthreads();
  if (tid < CT_TILE / 8) {
    uint64_t m = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) m = s_v[tid * 8 + i] > m ? s_v[tid * 8 + i] : m;
    s_sub[tid] = m;
  }
  if (wv == 1) {  // the previous tile's group maxima: most escaping answers lie there
    const uint64_t pm = a.M[1][tile > 0 ? (tile - 1) * QY_GROUPS + lane : lane];
    s_prev[lane] = tile > 0 ? pm : 0ull;
  }
  if (wv == 0) {  // group-level window maxima and exclusive prefix maxima
    const uint64_t m1r = a.M[1][tile * QY_GROUPS + (lane < ng ? lane : 0)];
    const uint64_t m1 = lane < ng ? m1r : 0ull;
    uint64_t w = m1;
    s_g[0][lane] = w;
#pragma unroll
    for (int k = 1; k < 6; ++k) {
      const uint64_t o = shfl_up(w, 1u << (k - 1));
      if (lane >= (1 << (k - 1))) w = o > w ? o : w;
      s_g[k][lane] = w;
    }
    const uint64_t ex = wave_shift_up1_u64(wave_prefix_max_u64(m1), 0ull);
    const uint64_t pt = a.pmt[tile];
    s_gpre[lane] = lane == 0 ? pt : (ex > pt ? ex : pt);
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < QY_ROUNDS; ++r) {
    const int g = wv + r * (QY_THREADS / WAVE);
    const int lp = g * 64 + lane;
    const bool live = lp < tn;
    const uint64_t q = (key_seg(a, key[r]) << a.vb) | (uint64_t)(key_rel(a, key[r]) + 1);
    const uint64_t v = s_v[lp];
    uint64_t w[6];
    w[0] = v;
#pragma unroll
    for (int k = 1; k < 6; ++k) {
      const uint64_t o = shfl_up(w[k - 1], 1u << (k - 1));
      w[k] = (lane >= (1 << (k - 1)) && o > w[k - 1]) ? o : w[k - 1];
    }
    // exclusive prefix max inside the group, then the prefix before it
    uint64_t pm = wave_shift_up1_u64(wave_prefix_max_u64(v), 0ull);
    const uint64_t gp = s_gpre[g];
    pm = pm > gp ? pm : gp;
    const bool want = live && pm > q;
    // level 0: this group
    const int f0 = wave_lift(w, lane - 1, q);
    int ans = -1;  // position in the tile
    bool escape = false;
    if (want) {
      if (f0 >= 0) {
        ans = g * 64 + f0;
      } else {
        // level 1: the tile's earlier groups, widest windows first
        int h = g - 1;
#pragma unroll
        for (int k = 5; k >= 0; --k)
          if (h - (1 << k) + 1 >= 0 && s_g[k][h] <= q) h -= 1 << k;
        if (h >= 0) {
          // the last 8-block of group h above q, then its last position
          // (group h holds a value above q; the bounds only guard that)
          int sb = h * 8 + 7;
          while (sb > h * 8 && s_sub[sb] <= q) --sb;
          int i = sb * 8 + 7;
          while (i > sb * 8 && s_v[i] <= q) --i;
          if (s_v[i] > q)
            ans = i;
          else
            set_status(a.ds, DS_LOGIC);
        } else {
          escape = true;
        }
      }
    }
    if (escape) {
      const int slot = atomicAdd(&s_nesc, 1);
      s_esc[slot] = (uint16_t)lp;
    } else if (live) {
      a.par[base + lp] = ans >= 0 ? (int32_t)(base + ans) : -1;
      a.link[row[r]] = ans >= 0 ? (int32_t)s_val[ans] : -1;
    }
  }
  __syncthreads();
  // answers in earlier tiles, one wave per query
  const int nesc = s_nesc;
  for (int e = wv; e < nesc; e += QY_THREADS / WAVE) {
    const int lp = s_esc[e];
    const int64_t p = base + lp;
    const uint64_t kk = keys[p];
    const uint64_t q = (key_seg(a, kk) << a.vb) | (uint64_t)(key_rel(a, kk) + 1);
    // the last group of the previous tile holding a value above q, then its
    // last position above q (one load); else the general climb
    int64_t ans = -1;
    const uint64_t gb = ballot(s_prev[lane] > q);
    if (gb) {
      const int g = 63 - __clzll((long long)gb);
      const int64_t e0 = (tile - 1) * CT_TILE + (int64_t)g * 64;
      const uint64_t v = a.V[e0 + lane];
      const uint64_t vb = ballot(v > q);
      if (vb) ans = e0 + 63 - __clzll((long long)vb);
    }
    if (!gb) ans = wave_escape(a, tile, q, n);
    if (lane == 0) {
      if (ans < 0) set_status(a.ds, DS_LOGIC);
      a.par[p] = (int32_t)ans;
      a.link[s_val[lp]] = ans >= 0 ? (int32_t)vals[ans] : -1;
    }
  }
}

// Depth by walking the parents; improper nesting; op aggregates reset.  Each
// thread walks DP_ITEMS positions' parent chains side by side, so the loads
// of one step of all chains are in flight together.
constexpr int DP_ITEMS = 2;

__global__ __launch_bounds__(256) void k_depth(ContainArgs a) {
  __shared__ unsigned long long s_imp;
  const int64_t n = a.ds->nCL;
  // Positions past the end take the last entry (clamped loads); with no
  // entry there is nothing to take, and nothing to do.
  if (n == 0) return;
  if (threadIdx.x == 0) s_imp = 0;
  __syncthreads();
  const int par = (int)a.ds->sort_parity[1];
  const uint64_t* keys = a.k[par];
  const uint32_t* vals = a.v[par];
  const int64_t p0 = (int64_t)blockIdx.x * 256 * DP_ITEMS + threadIdx.x;
  uint32_t row[DP_ITEMS];
  int64_t q[DP_ITEMS];
  // each round of loads is issued for all items together (clamped indices)
  uint64_t kk[DP_ITEMS];
#pragma unroll
  for (int u = 0; u < DP_ITEMS; ++u) {
    const int64_t p = p0 + u * 256;
    const int64_t pc = p < n ? p : n - 1;
    kk[u] = keys[pc];
    row[u] = vals[pc];
    q[u] = a.par[pc];
  }
#pragma unroll
  for (int u = 0; u < DP_ITEMS; ++u) {
    const bool op = p0 + u * 256 < n && key_is_op(kk[u]);
    if (!op) {
      row[u] = ~0u;
      q[u] = -1;
    }
  }
  // improper nesting: the op ends after its parent
  uint32_t imp = 0;
  uint32_t prow[DP_ITEMS];
#pragma unroll
  for (int u = 0; u < DP_ITEMS; ++u) prow[u] = vals[q[u] >= 0 ? q[u] : 0];
  int64_t te_own[DP_ITEMS], te_par[DP_ITEMS];
#pragma unroll
  for (int u = 0; u < DP_ITEMS; ++u) {
    te_own[u] = a.te[row[u] != ~0u ? row[u] : 0u];
    te_par[u] = a.te[q[u] >= 0 ? prow[u] : 0u];
  }
#pragma unroll
  for (int u = 0; u < DP_ITEMS; ++u)
    if (q[u] >= 0 && te_own[u] > te_par[u]) ++imp;  // one process: raw ends compare like corrected
  int32_t d[DP_ITEMS];
#pragma unroll
  for (int u = 0; u < DP_ITEMS; ++u) d[u] = 0;
  for (;;) {
    bool any = false;
    int64_t nq[DP_ITEMS];
#pragma unroll
    for (int u = 0; u < DP_ITEMS; ++u) nq[u] = a.par[q[u] >= 0 && q[u] < n ? q[u] : 0];
#pragma unroll
    for (int u = 0; u < DP_ITEMS; ++u) {
      if (q[u] >= 0 && in_range(a.ds, q[u], n)) {
        ++d[u];
        q[u] = nq[u];
        any = true;
      }
    }
    if (!any) break;
  }
#pragma unroll
  for (int u = 0; u < DP_ITEMS; ++u) {
    if (row[u] == ~0u) continue;
    a.aux[row[u]] = d[u];
  }
  // The ops open at the start of aggregate tile b: the chain of answers from
  // the position before it (that position first, if it is an op).  They, and
  // the ops open at the end of the last tile, are the only ops whose
  // aggregates are summed with atomics (the others are stored whole by the
  // aggregate pass): their aggregates start here at the identities.
  const int64_t b = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t ntl = cdiv(n, AG_TILE);
  auto init_op = [&](int64_t q) {
    const uint32_t rr = vals[q];
    op_store(a, rr, 0, I64MAX, I64MIN, 0);
  };
  if (b < ntl) {
    int nc = 0;
    if (b > 0) {
      const int64_t pe = b * AG_TILE - 1;
      for (int64_t q = key_is_op(keys[pe]) ? pe : a.par[pe]; q >= 0 && in_range(a.ds, q, n); q = a.par[q]) {
        if (nc < AG_CHAIN) a.ag_chain[b * AG_CHAIN + nc] = (int32_t)q;
        ++nc;
        init_op(q);
      }
    }
    a.ag_nchain[b] = nc;
  } else if (b == ntl) {
    const int64_t pe = n - 1;
    for (int64_t q = key_is_op(keys[pe]) ? pe : a.par[pe]; q >= 0 && in_range(a.ds, q, n); q = a.par[q]) init_op(q);
  }
  const uint64_t w = wave_sum_u64(imp);
  if (lane_id() == 0 && w) atomicAdd(&s_imp, (unsigned long long)w);
  __syncthreads();
  if (threadIdx.x == 0 && s_imp) atomicAdd((unsigned long long*)&a.cnt->n_improper_nesting, s_imp);
}

// ------------------------------------------------------ inclusive aggregates
constexpr int AG_THREADS = 256;
constexpr int AG_ITEMS = AG_TILE / AG_THREADS;
static_assert(AG_TILE % AG_THREADS == 0 && AG_CHAIN <= AG_THREADS, "aggregate tile layout");

// Adds (count, first, last, sum) to the op at sorted position q and every op
// above it, in HBM: the part of a chain deeper than the table of ops open at
// a tile start.
__device__ void agg_add_global(const ContainArgs& a, int64_t q, uint32_t nk, int64_t f, int64_t l, uint64_t sm) {
  const uint32_t* vals = a.v[(int)a.ds->sort_parity[1]];
  for (int64_t r = q; r >= 0; r = a.par[r]) {
    const uint32_t rr = vals[r];
    op_combine(a, rr, nk, f, l, sm);
  }
}

// One workgroup per AG_TILE positions, AG_ITEMS per thread (striped).  The
// answers form a forest whose preorder is the sorted order, and an op's
// depth is its parent's plus one.  Every launch adds its kernels to its own
// op; then, deepest level first, every op adds its totals to its parent, so
// each op passes its totals up once (an op at the tile edge holds the part
// of its subtree inside the tile).  Ops open at the tile start (found by the
// depth pass) collect what reaches them in a table and take a prefix over
// it, innermost first; ops still open at the tile end, and the open ops of
// the start, add into HBM with atomics; the others are stored.
__global__ __launch_bounds__(AG_THREADS) void k_opagg(ContainArgs a) {
  __shared__ int32_t s_par[AG_TILE];
  __shared__ uint32_t s_nk[AG_TILE];
  __shared__ int64_t s_first[AG_TILE];
  __shared__ int64_t s_last[AG_TILE];
  __shared__ uint64_t s_sum[AG_TILE];
  __shared__ uint8_t s_open[AG_TILE];
  __shared__ int32_t s_chain[AG_CHAIN];  // ops open at the tile start, innermost first
  __shared__ uint32_t c_nk[AG_CHAIN];
  __shared__ int64_t c_first[AG_CHAIN], c_last[AG_CHAIN];
  __shared__ uint64_t c_sum[AG_CHAIN];
  __shared__ int s_dmin, s_dmax, s_last_op;
  const int tid = threadIdx.x, lane = lane_id();
  const int64_t n = a.ds->nCL;
  const int par = (int)a.ds->sort_parity[1];
  const uint64_t* keys = a.k[par];
  const uint32_t* vals = a.v[par];
  const int64_t base = (int64_t)blockIdx.x * AG_TILE;
  if (base >= n) return;
  const int64_t tn = min((int64_t)AG_TILE, n - base);

  // round 1: keys, rows, answers; the open chain of the tile start
  uint64_t key[AG_ITEMS];
  uint32_t row[AG_ITEMS];
  int32_t pr[AG_ITEMS];
#pragma unroll
  for (int u = 0; u < AG_ITEMS; ++u) {
    const int i = tid + u * AG_THREADS;
    const int64_t pc = base + (i < tn ? i : tn - 1);
    key[u] = keys[pc];
    row[u] = vals[pc];
    pr[u] = a.par[pc];
  }
  const int32_t chv = tid < AG_CHAIN ? a.ag_chain[(int64_t)blockIdx.x * AG_CHAIN + tid] : -1;
  const int32_t ncv = a.ag_nchain[blockIdx.x];
  // round 2: an op's depth or a launch's kernel count (both in aux), and a
  // launch's kernel aggregates (one round of loads: an op reads the
  // aggregates of row 0 instead of branching around the loads, so that its
  // reads hit one cached line and the loads need no wait of their own)
  int32_t av[AG_ITEMS];
  int64_t lf[AG_ITEMS], ll[AG_ITEMS];
  uint64_t ls[AG_ITEMS];
#pragma unroll
  for (int u = 0; u < AG_ITEMS; ++u) {
    const uint32_t lr = key_is_op(key[u]) ? 0u : row[u];
    av[u] = a.aux[row[u]];
    lf[u] = a.lk_first[lr];
    ll[u] = a.lk_last[lr];
    ls[u] = (uint64_t)a.lk_sum[lr];
  }
  int dmin = INT32_MAX, dmax = -1;
#pragma unroll
  for (int u = 0; u < AG_ITEMS; ++u) {
    const int i = tid + u * AG_THREADS;
    if (i < tn) {
      const bool op = key_is_op(key[u]);
      s_par[i] = pr[u];
      if (i == tn - 1) s_last_op = op;
      s_nk[i] = 0;
      s_first[i] = I64MAX;
      s_last[i] = I64MIN;
      s_sum[i] = 0;
      s_open[i] = 0;
      if (op) {
        dmin = av[u] < dmin ? av[u] : dmin;
        dmax = av[u] > dmax ? av[u] : dmax;
      }
    }
  }
  if (tid < AG_CHAIN) {
    s_chain[tid] = chv;
    c_nk[tid] = 0;
    c_first[tid] = I64MAX;
    c_last[tid] = I64MIN;
    c_sum[tid] = 0;
  }
  if (tid == 0) {
    s_dmin = INT32_MAX;
    s_dmax = -1;
  }
  for (int d = 1; d < WAVE; d <<= 1) {
    const int o1 = __shfl_xor(dmin, d, WAVE), o2 = __shfl_xor(dmax, d, WAVE);
    dmin = o1 < dmin ? o1 : dmin;
    dmax = o2 > dmax ? o2 : dmax;
  }
  __syncthreads();
  if (lane == 0) {
    atomicMin(&s_dmin, dmin);
    atomicMax(&s_dmax, dmax);
  }
  if (tid == 0) {
    // ops of this tile still open at its end receive later contributions
    const int64_t last = tn - 1;
    int64_t q = s_last_op ? base + last : s_par[last];
    while (q >= base) {
      s_open[q - base] = 1;
      q = s_par[q - base];
    }
  }
  // Adds (count, first, last, sum) to the op at sorted position q: in LDS
  // when q lies in the tile, to the table of ops open at the tile start when
  // it lies before it, and to HBM beyond the table.  (The LDS arrays are
  // named here, not passed by pointer, so that these stay LDS atomics.)
  const int kn0 = ncv < AG_CHAIN ? ncv : AG_CHAIN;
  auto add = [&](int64_t q, uint32_t nk, int64_t f, int64_t l, uint64_t sm) {
    if (q >= base) {
      const int li = (int)(q - base);
      atomicAdd(&s_nk[li], nk);
      atomicMin((long long*)&s_first[li], (long long)f);
      atomicMax((long long*)&s_last[li], (long long)l);
      atomicAdd((unsigned long long*)&s_sum[li], (unsigned long long)sm);
      return;
    }
    if (q < 0) return;
    int k = 0;
    while (k < kn0 && s_chain[k] != q) ++k;
    if (k < kn0) {
      atomicAdd(&c_nk[k], nk);
      atomicMin((long long*)&c_first[k], (long long)f);
      atomicMax((long long*)&c_last[k], (long long)l);
      atomicAdd((unsigned long long*)&c_sum[k], (unsigned long long)sm);
      return;
    }
    agg_add_global(a, q, nk, f, l, sm);
  };
  // every launch to its own op
#pragma unroll
  for (int u = 0; u < AG_ITEMS; ++u) {
    const int i = tid + u * AG_THREADS;
    if (i < tn && !key_is_op(key[u]) && av[u] > 0) add(pr[u], (uint32_t)av[u], lf[u], ll[u], ls[u]);
  }
  __syncthreads();
  // every op to its parent, deepest level first
  const int d_lo = s_dmin, d_hi = s_dmax;
  for (int L = d_hi; L >= d_lo && L >= 0; --L) {
#pragma unroll
    for (int u = 0; u < AG_ITEMS; ++u) {
      const int i = tid + u * AG_THREADS;
      // the item's depth is in registers; only an op of this level reads LDS
      if (i < tn && key_is_op(key[u]) && av[u] == L && s_nk[i] > 0) add(pr[u], s_nk[i], s_first[i], s_last[i], s_sum[i]);
    }
    __syncthreads();
  }
  const int nc = ncv;
  const int kn = nc < AG_CHAIN ? nc : AG_CHAIN;
  if (tid == 0) {
    // the open ops of the tile start, innermost first: each holds what
    // reached it or any op inside it
    for (int k = 1; k < kn; ++k) {
      c_nk[k] += c_nk[k - 1];
      c_first[k] = c_first[k - 1] < c_first[k] ? c_first[k - 1] : c_first[k];
      c_last[k] = c_last[k - 1] > c_last[k] ? c_last[k - 1] : c_last[k];
      c_sum[k] += c_sum[k - 1];
    }
    // chains deeper than the table: the ops above it take the table's total
    if (nc > AG_CHAIN && c_nk[AG_CHAIN - 1]) {
      for (int64_t r = a.par[s_chain[AG_CHAIN - 1]]; r >= 0; r = a.par[r]) {
        const uint32_t rr = vals[r];
        op_combine(a, rr, c_nk[AG_CHAIN - 1], c_first[AG_CHAIN - 1], c_last[AG_CHAIN - 1], c_sum[AG_CHAIN - 1]);
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < AG_ITEMS; ++u) {
    const int i = tid + u * AG_THREADS;
    if (!(i < tn && key_is_op(key[u]))) continue;
    const uint32_t rr = row[u];
    if (s_open[i]) {
      if (s_nk[i]) {
        op_combine(a, rr, s_nk[i], s_first[i], s_last[i], s_sum[i]);
      }
    } else {
      op_store(a, rr, (int32_t)s_nk[i], s_first[i], s_last[i], (int64_t)s_sum[i]);
    }
  }
  if (tid < kn && c_nk[tid]) {
    const uint32_t rr = vals[s_chain[tid]];
    op_combine(a, rr, c_nk[tid], c_first[tid], c_last[tid], c_sum[tid]);
  }
}

static ContainArgs contain_args(Ctx& c) {
  ContainArgs a;
  a.k[0] = c.sC.k[0];
  a.k[1] = c.sC.k[1];
  a.v[0] = c.sC.v[0];
  a.v[1] = c.sC.v[1];
  a.ts = c.ev.ts;
  a.te = c.ev.te;
  a.off = c.p.clock_offset;
  a.W0 = c.W0;
  a.W1 = c.W1;
  a.W = c.W;
  a.tb = c.tb;
  a.wb = c.wb;
  a.vb = c.vb;
  a.ds = c.ds;
  a.cnt = c.o.counters;
  a.link = c.o.link;
  a.aux = c.o.aux;
  a.op_nkern = c.o.op_nkern;
  a.op_first = c.o.op_first;
  a.op_last = c.o.op_last;
  a.op_ksum = c.o.op_ksum;
  a.V = c.V;
  for (int l = 0; l < 6; ++l) {
    a.M[l] = c.M[l];
    a.Mn[l] = c.Mn[l];
  }
  a.nlev = c.nlev;
  a.pmt = c.pmt;
  a.vb_status = c.vb_status;
  a.par = c.par;
  a.lk_first = c.lk_first;
  a.lk_last = c.lk_last;
  a.lk_sum = c.lk_sum;
  a.ag_chain = c.ag_chain;
  a.ag_nchain = c.ag_nchain;
  a.ag_tiles = c.ag_tiles;
  return a;
}

void launch_contain(Ctx& c) {
  ContainArgs a = contain_args(c);
  const int64_t tiles = std::max<int64_t>(cdiv(c.sC.n_max, CT_TILE), 1);
  hipLaunchKernelGGL(k_vbuild, dim3((unsigned)tiles), dim3(VB_THREADS), 0, c.st, a);
  hipLaunchKernelGGL(k_query, dim3((unsigned)tiles), dim3(QY_THREADS), 0, c.st, a);
}

void launch_depth(Ctx& c) {
  ContainArgs a = contain_args(c);
  hipLaunchKernelGGL(k_depth, dim3((unsigned)std::max<int64_t>(cdiv(c.sC.n_max, 256 * DP_ITEMS), 1)), dim3(256), 0,
                     c.st, a);
}

void launch_opagg(Ctx& c) {
  ContainArgs a = contain_args(c);
  const int64_t tiles = std::max<int64_t>(cdiv(c.sC.n_max, AG_TILE), 1);
  hipLaunchKernelGGL(k_opagg, dim3((unsigned)tiles), dim3(AG_THREADS), 0, c.st, a);
}

}  // namespace hx
