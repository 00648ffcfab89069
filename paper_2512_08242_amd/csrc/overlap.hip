// chopper_overlap: compute/communication overlap (paper Section V-C) and
// launch bubbles (Section V-D eqs. 1-3; caption of Fig. end_to_end).
//
// An instant is compute-active iff some compute kernel covers it (c(t) > 0 in
// the +-1 event count), so the sweep reduces to the union of each GPU's
// compute intervals and the union of its communication intervals.  Walking
// the records in (gpu, kind, start') order, an interval opens a new union
// run iff its start lies beyond the running maximum of all earlier ends of
// the same (gpu, kind) -- a segmented max-scan.  Prefix sums of run lengths
// then give F(t) = active time before t for either kind by one binary
// search, and the time where both are active is accumulated per
// communication run, so every window (kernel, marker, GPU) costs a few
// binary searches and no per-window sweep.
#include "sort.h"
#include "wave.h"
#include "bindex.h"

namespace chopper {

bool validate_records(const chopper_records* r);
bool validate_markers(const chopper_markers* m);

constexpr int kOvIpt = 8;
constexpr int kOvTile = kBlock * kOvIpt;
constexpr int kSegs = 512;            // gpu * 2 + kind
static_assert(kOvTile == kWavesPerBlock * kWaveTile, "tile = block = 4 waves");

struct Runs {
  const int64_t* rs;      // run start
  const int64_t* re;      // run end
  const int64_t* pl;      // active time of the segment before the run
  // comm runs only, at dense index voff[g] + (j - first comm run of g):
  const int64_t* pov;     // exclusive prefix of overlapped time
  const int64_t* ovc;     // overlapped time inside the run
  const int64_t* fcrs;    // compute-active time before the run's start
  const uint32_t* voff;   // [G + 1] first dense index of every gpu
  BIndex X;               // bucket index of the run starts per segment
};

// Active time of a segment strictly before t, given the first run of the
// segment whose start is > t (so j = up - 1 is the run holding or preceding
// t).
__device__ inline int64_t F_at(const Runs& R, const BSeg& P, int64_t up,
                               int64_t t) {
  const int64_t j = up - 1;
  if (j < (int64_t)P.sb) return 0;
  const int64_t e = R.re[j] < t ? R.re[j] : t;
  return R.pl[j] + (e - R.rs[j]);
}

// the segment parameters of the first nseg segments, copied to LDS by the
// whole block (call before any thread leaves)
__device__ inline void segs_to_lds(BSeg* s_seg, const BSeg* segs, int nseg) {
  for (int i = threadIdx.x; i < nseg; i += blockDim.x) s_seg[i] = segs[i];
  __syncthreads();
}

// CO, MO, OV, ID of [a, b) on gpu g (Section V-C): compute-active time c,
// comm-active time m and the time where both are, o; both-active time
// before t is the overlap of the comm runs before t plus, inside the comm
// run holding t, the compute-active time up to t.
template <int K>
__device__ inline void window_k(const Runs& R, const BSeg (&Pc)[K],
                                const BSeg (&Pm)[K], const uint32_t (&vg)[K],
                                const int64_t (&a)[K], const int64_t (&b)[K],
                                int64_t (&out)[K][4]) {
  // compute and comm searches at both ends of every window, in lockstep
  int64_t lo[4 * K], hi[4 * K], t[4 * K];
#pragma unroll
  for (int q = 0; q < K; ++q) {
    t[4 * q + 0] = a[q];
    t[4 * q + 1] = b[q];
    t[4 * q + 2] = a[q];
    t[4 * q + 3] = b[q];
    bi_range(R.X, Pc[q], a[q], &lo[4 * q + 0], &hi[4 * q + 0]);
    bi_range(R.X, Pc[q], b[q], &lo[4 * q + 1], &hi[4 * q + 1]);
    bi_range(R.X, Pm[q], a[q], &lo[4 * q + 2], &hi[4 * q + 2]);
    bi_range(R.X, Pm[q], b[q], &lo[4 * q + 3], &hi[4 * q + 3]);
  }
  bsearch_k<4 * K>(R.rs, lo, hi, t);
#pragma unroll
  for (int q = 0; q < K; ++q) {
    const int64_t* l = lo + 4 * q;
    const int64_t ca = F_at(R, Pc[q], l[0], a[q]), cb = F_at(R, Pc[q], l[1], b[q]);
    const int64_t ma = F_at(R, Pm[q], l[2], a[q]), mb = F_at(R, Pm[q], l[3], b[q]);
    // both-active time before t: the overlap of the comm runs before the
    // one holding t, plus inside it either its whole overlap (t past its
    // end) or the compute-active time from its start to t -- F_c(t), known
    // above
    int64_t ob[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int64_t jm = l[2 + k] - 1;
      const int64_t tk = k ? b[q] : a[q];
      ob[k] = 0;
      if (jm < (int64_t)Pm[q].sb) continue;   // no comm run at or before t
      const int64_t v = (int64_t)vg[q] + (jm - (int64_t)Pm[q].sb);
      const int64_t before = R.pov[v] - R.pov[vg[q]];
      ob[k] = before +
              (tk < R.re[jm] ? (k ? cb : ca) - R.fcrs[v] : R.ovc[v]);
    }
    const int64_t c = cb - ca, m = mb - ma, o = ob[1] - ob[0];
    if (b[q] <= a[q]) {
      out[q][0] = out[q][1] = out[q][2] = out[q][3] = 0;
    } else {
      out[q][0] = c - o;
      out[q][1] = m - o;
      out[q][2] = o;
      out[q][3] = (b[q] - a[q]) - c - m + o;
    }
  }
}


// ---------------- union runs -----------------------------------------------
// Tiles of kOvTile korder positions, one block each; the block's four waves
// take kWaveTile consecutive positions apiece.  Loads are striped, and the
// ordered scans run on the blocked arrangement after an LDS transpose.

// Running sum restricted to the last segment; seg == kNone is the empty
// value (a two-sided identity).
struct SegSum {
  uint32_t seg;
  uint32_t pad;
  int64_t sum;
};
struct OpSegSum {
  __device__ SegSum operator()(SegSum a, SegSum b) const {
    if (b.seg == kNone) return a;
    if (a.seg == kNone || a.seg != b.seg) return b;
    return SegSum{b.seg, 0u, a.sum + b.sum};
  }
};
__device__ inline SegSum segsum_ident() { return SegSum{kNone, 0u, 0}; }
__device__ inline SegMax segmax_ident() { return SegMax{0u, kI64Min}; }

__device__ inline void korder_gather(const uint32_t* korder, const uint8_t* gpu,
                                     const uint8_t* cls, const int64_t* start,
                                     const int64_t* end, int64_t p,
                                     uint32_t& seg, int64_t& s, int64_t& e) {
  const uint32_t r = korder[p];
  seg = (uint32_t)gpu[r] * 2u + (uint32_t)kind_of(cls[r]);
  s = start[r];
  const int64_t x = end[r];
  e = x > s ? x : s;
}

// Exclusive scans of per-tile values over many blocks of 1024 threads:
// block b scans tiles [1024 b, 1024 b + 1024), one per thread, after
// folding every tile before them itself (thread t the b consecutive tiles
// from t b on, so the fold keeps the tile order); the block of the last
// tile also writes the total.
constexpr int kSpineSpan = 1024;
// most blocks of the fix-up pass (4 per compute unit)
constexpr unsigned kFixBlocks = 1024;

// Ordered fold of one value per thread over the block: the exclusive
// prefix of the thread and the block total.  `s_w` holds one value per
// wave and the total; wave 0 scans the wave totals.
constexpr int kSpineWaves = kSpineSpan / kWave;
template <typename T, typename Op>
__device__ inline T block_excl_ordered(T v, Op op, T ident, T* s_w, T* tot) {
  const int lane = lane_id(), w = (int)(threadIdx.x / kWave);
  const T incl = wave_incl(v, op, ident);
  if (lane == kWave - 1) s_w[w] = incl;
  __syncthreads();
  if (w == 0) {
    const T x = lane < kSpineWaves ? s_w[lane] : ident;
    const T xi = wave_incl(x, op, ident);
    const T xe = wave_shr1_any(ident, xi);
    if (lane < kSpineWaves) s_w[lane] = xe;
    if (lane == kWave - 1) s_w[kSpineWaves] = xi;
  }
  __syncthreads();
  *tot = s_w[kSpineWaves];
  const T pre = s_w[w];
  __syncthreads();
  return op(pre, wave_shr1_any(ident, incl));
}

template <typename T, typename Op>
__device__ inline T fold_before(const T* in, Op op, T ident, T* s_w) {
  const int64_t c = blockIdx.x, t = threadIdx.x;
  T p = ident;
  for (int64_t k = 0; k < c; ++k) p = op(p, in[t * c + k]);
  T tot;
  (void)block_excl_ordered(p, op, ident, s_w, &tot);
  return tot;
}

// The exclusive (segment, end) maximum before every tile (the carry; with
// the total), and the list of the tiles after the first whose carry has
// their first item's segment and reaches its start (fix[0] their number,
// cleared by the count pass; fix[1..] the tiles, in no particular order):
// the counts of only these change with the carry (k_runs_fix).
__global__ __launch_bounds__(kSpineSpan) void k_runs_carry(
    const SegMax* agg, SegMax* pre_out, int64_t ntiles, SegMax* total,
    const SegMax* first, uint32_t* fix) {
  __shared__ SegMax s_w[kSpineWaves + 1];
  OpSegMax op;
  const SegMax ident = segmax_ident();
  const SegMax before = fold_before(agg, op, ident, s_w);
  const int64_t i = (int64_t)blockIdx.x * kSpineSpan + threadIdx.x;
  const SegMax v = i < ntiles ? agg[i] : ident;
  SegMax tot;
  const SegMax pre = op(before, block_excl_ordered(v, op, ident, s_w, &tot));
  bool again = false;
  if (i < ntiles) {
    pre_out[i] = pre;
    const SegMax f = first[i];
    again = i > 0 && pre.seg == f.seg && pre.val >= f.val;
  }
  // one append per wave
  const uint64_t m = __ballot(again);
  if (m != 0) {
    uint32_t base = 0;
    if (lane_id() == 0) base = atomicAdd(fix, (uint32_t)__popcll(m));
    base = __shfl(base, 0, kWave);
    if (again) fix[1 + base + lanes_below(m)] = (uint32_t)i;
  }
  if (threadIdx.x == 0 && (int64_t)(blockIdx.x + 1) * kSpineSpan >= ntiles)
    *total = op(before, tot);
}

// The exclusive scan of the tiles' run counts (with the total) and the
// segmented scan of their union increments (with the total).  Block 0 also
// sets up the bucket index of the run starts of every (gpu, kind) segment
// before the runs are written: a segment's candidate item range is kept
// only if its first item is the first of the segment and its end the end
// (each is unique, so stale candidates fail); the buckets then span its
// items' starts, which include every run start, with about one per
// kKeysPerBucket items (a valid index for any count).  The run range of
// each segment (sb, se) is set after the write pass.
__global__ __launch_bounds__(kSpineSpan) void k_runs_spine2(
    const uint32_t* heads, uint32_t* run0, uint32_t* nruns,
    const SegSum* inc, SegSum* inc_pre, SegSum* inc_total, int64_t ntiles,
    int G, int64_t n, const uint32_t* korder, const uint8_t* gpu,
    const uint8_t* cls, const int64_t* start, const uint32_t* kcand,
    BSeg* segs, uint32_t* kr, int64_t btable_cap) {
  __shared__ uint32_t s_h[kSpineWaves + 1];
  __shared__ SegSum s_i[kSpineWaves + 1];
  OpSegSum op;
  const SegSum ident = segsum_ident();
  const uint32_t hb = fold_before(heads, OpAdd(), 0u, s_h);
  const SegSum ib = fold_before(inc, op, ident, s_i);
  const int64_t i = (int64_t)blockIdx.x * kSpineSpan + threadIdx.x;
  const uint32_t h = i < ntiles ? heads[i] : 0u;
  const SegSum v = i < ntiles ? inc[i] : ident;
  uint32_t ht;
  SegSum it;
  const uint32_t hp = hb + block_excl_ordered(h, OpAdd(), 0u, s_h, &ht);
  const SegSum ip = op(ib, block_excl_ordered(v, op, ident, s_i, &it));
  if (i < ntiles) {
    run0[i] = hp;
    inc_pre[i] = ip;
  }
  if (threadIdx.x == 0 && (int64_t)(blockIdx.x + 1) * kSpineSpan >= ntiles) {
    *nruns = hb + ht;
    *inc_total = op(ib, it);
  }
  if (blockIdx.x != 0) return;   // block-uniform
  const int t = (int)threadIdx.x;
  BSeg P;
  P.lo = 0;
  P.sb = P.se = 0;
  P.shift = 0;
  P.nb = 0;
  P.toff = 0;
  P.pad = 0;
  uint32_t ent = 0, kb = 0, ke = 0;
  if (t < 2 * G && n > 0) {
    const int64_t cb = kcand[t], ce = kcand[kSegs + t];
    // every load issued at a clamped position, the checks afterwards
    const int64_t q[4] = {cb < n ? cb : n - 1,
                          cb > 0 && cb - 1 < n ? cb - 1 : 0,
                          ce >= 1 && ce <= n ? ce - 1 : 0,
                          ce < n ? ce : n - 1};
    uint32_t r[4], sg[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = korder[q[i]];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      sg[i] = (uint32_t)gpu[r[i]] * 2u + (uint32_t)kind_of(cls[r[i]]);
    const int64_t lo = start[r[0]], last = start[r[2]];
    const uint32_t ts = (uint32_t)t;
    const bool ok = cb < n && ce <= n && ce > cb && sg[0] == ts &&
                    (cb == 0 || sg[1] != ts) && sg[2] == ts &&
                    (ce == n || sg[3] != ts);
    if (ok) {
      kb = (uint32_t)cb;
      ke = (uint32_t)ce;
      P.lo = lo;
      bi_geometry(lo, last, ce - cb, &P.shift, &P.nb);
      ent = P.nb + 1;
    }
  }
  uint32_t tot;
  const uint32_t pre = block_excl_ordered(ent, OpAdd(), 0u, s_h, &tot);
  if (t < 2 * G) {
    P.toff = (int64_t)pre < btable_cap ? pre : (uint32_t)btable_cap;
    if ((int64_t)pre + ent > btable_cap) P.nb = 0;
    segs[t] = P;
    kr[t] = kb;
    kr[kSegs + t] = ke;
  }
}

// Per-item view of a tile in the blocked arrangement: segment, start, end,
// exclusive running (seg, end) maximum, run-head flag and the length the
// item adds to the union of its segment.
struct RunItems {
  uint32_t seg[kTileIpt];
  int64_t s[kTileIpt];
  int64_t mx[kTileIpt];     // exclusive running max of the same segment
  int64_t inc[kTileIpt];
  uint32_t m_valid, m_head, m_newseg;
  uint32_t pseg0;           // segment of the item before the lane's first
  SegMax wagg;              // (segment, end) maximum of the wave's items
};

__device__ inline void run_items(int64_t tile, int64_t n,
                                 const uint32_t* korder, const uint8_t* gpu,
                                 const uint8_t* cls, const int64_t* start,
                                 const int64_t* end, const SegMax* tile_pre,
                                 int64_t* slice, RunItems& it) {
  const int lane = lane_id(), wv = (int)(threadIdx.x / kWave);
  const int64_t wbase = tile * kOvTile + (int64_t)wv * kWaveTile;
  uint32_t seg[kTileIpt];
  int64_t s[kTileIpt], e[kTileIpt];
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const int64_t p = wbase + (int64_t)j * kWave + lane;
    if (p < n) {
      korder_gather(korder, gpu, cls, start, end, p, seg[j], s[j], e[j]);
    } else {
      seg[j] = kNone;
      s[j] = e[j] = 0;
    }
  }
  wave_to_blocked(slice, s, lane);
  wave_to_blocked(slice, e, lane);
  wave_to_blocked((uint32_t*)slice, seg, lane);
  OpSegMax op;
  SegMax acc = segmax_ident();
  SegMax loc[kTileIpt];
  uint32_t m_valid = 0;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    loc[j] = acc;
    if (seg[j] != kNone) {
      m_valid |= 1u << j;
      acc = op(acc, SegMax{seg[j], e[j]});
    }
  }
  // lane tails scanned over the wave, then the waves of the block in order
  const SegMax incl = wave_incl(acc, op, segmax_ident());
  it.wagg = lane63(incl);
  __shared__ SegMax s_w[kWavesPerBlock];
  if (lane == kWave - 1) s_w[wv] = incl;
  __syncthreads();
  SegMax pre = tile_pre ? tile_pre[tile] : segmax_ident();
  for (int i = 0; i < kWavesPerBlock; ++i)
    if (i < wv) pre = op(pre, s_w[i]);
  pre = op(pre, wave_shr1_any(segmax_ident(), incl));
  const bool first_lane_of_all = tile == 0 && wv == 0 && lane == 0;
  it.pseg0 = first_lane_of_all ? kNone : pre.seg;
  uint32_t m_head = 0, m_newseg = 0;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const SegMax ex = op(pre, loc[j]);
    const bool first = first_lane_of_all && j == 0;
    const bool newseg = first || ex.seg != seg[j];
    const bool head = newseg || s[j] > ex.val;
    it.seg[j] = seg[j];
    it.s[j] = s[j];
    it.mx[j] = ex.val;
    if ((m_valid >> j) & 1u) {
      if (head) m_head |= 1u << j;
      if (newseg) m_newseg |= 1u << j;
      it.inc[j] = head ? e[j] - s[j] : (e[j] > ex.val ? e[j] - ex.val : 0);
    } else {
      it.inc[j] = 0;
    }
  }
  it.m_valid = m_valid;
  it.m_head = m_head;
  it.m_newseg = m_newseg;
}

// Number of runs (heads) and the segmented sum of union increments per tile,
// counted as if no earlier item reached into the tile (k_runs_fix corrects
// the tiles where one does), and also the tile's (segment, end) maximum and
// its first item (segment, start).
// Block 0 clears the segment run and korder ranges, the mixed-streams flag
// of the bubbles and the count of the fix-up list; the blocks together
// clear the bucket table of the run starts (filled by the write pass) and
// record, for every segment, the korder position of its first item and the
// end of its items (kcand [2][kSegs]); segments without items keep
// whatever the array held, so these are candidates that k_runs_spine2
// verifies against the items.
__global__ __launch_bounds__(kBlock) void k_runs_count(
    int64_t n, const uint32_t* korder, const uint8_t* gpu, const uint8_t* cls,
    const int64_t* start, const int64_t* end, SegMax* tile_agg,
    SegMax* tile_first, uint32_t* tile_heads, SegSum* tile_inc,
    uint32_t* ranges, uint32_t* mixed, uint32_t* kcand, uint32_t* btable,
    int64_t btable_cap, uint32_t* fix) {
  __shared__ int64_t s_slice[kWavesPerBlock][kSlice];
  if (blockIdx.x == 0) {
    for (int i = threadIdx.x; i < 4 * kSegs; i += kBlock) ranges[i] = 0;
    if (threadIdx.x == 0) {
      *mixed = 0;
      fix[0] = 0;
    }
  }
  bindex_clear(btable, btable_cap, blockIdx.x, gridDim.x);
  const int lane0 = lane_id();
  const int64_t wb0 = (int64_t)blockIdx.x * kOvTile +
                      (int64_t)(threadIdx.x / kWave) * kWaveTile;
  // segment of the item before the wave's first (for the boundaries)
  uint32_t sprev = kNone;
  if (lane0 == 0 && wb0 > 0 && wb0 <= n) {
    const uint32_t r = korder[wb0 - 1];
    sprev = (uint32_t)gpu[r] * 2u + (uint32_t)kind_of(cls[r]);
  }
  RunItems it;
  run_items(blockIdx.x, n, korder, gpu, cls, start, end, nullptr,
            s_slice[threadIdx.x / kWave], it);
  {
    // item p (blocked: wb0 + lane * 8 + j) starts a segment when its
    // predecessor's differs; the predecessor of a lane's first item is the
    // lane below's last (lane 0: the item before the wave)
    const uint32_t ps = wave_shr1_u32(sprev, it.seg[kTileIpt - 1]);
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j) {
      const int64_t p = wb0 + (int64_t)lane0 * kTileIpt + j;
      if (p >= n) break;
      const uint32_t pv = j ? it.seg[j - 1] : ps;
      const uint32_t sj = it.seg[j];
      if (p == 0 || pv != sj) {
        if (sj < (uint32_t)kSegs) kcand[sj] = (uint32_t)p;
        if (p > 0 && pv < (uint32_t)kSegs) kcand[kSegs + pv] = (uint32_t)p;
      }
      if (p == n - 1 && sj < (uint32_t)kSegs) kcand[kSegs + sj] = (uint32_t)n;
    }
  }
  OpSegSum op;
  SegSum acc = segsum_ident();
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j)
    if ((it.m_valid >> j) & 1u) acc = op(acc, SegSum{it.seg[j], 0u, it.inc[j]});
  acc = wave_incl(acc, op, segsum_ident());
  uint32_t c = (uint32_t)__popc(it.m_head);
  for (int d = kWave / 2; d > 0; d >>= 1) c += __shfl_xor(c, d, kWave);
  // the tile's (segment, end) maximum from the waves' ones
  OpSegMax om;
  const SegMax mx = it.wagg;
  __shared__ SegSum s_w[kWavesPerBlock];
  __shared__ uint32_t s_c[kWavesPerBlock];
  __shared__ SegMax s_m[kWavesPerBlock];
  const int lane = lane_id(), wv = (int)(threadIdx.x / kWave);
  if (lane == kWave - 1) {
    s_w[wv] = acc;
    s_c[wv] = c;
    s_m[wv] = mx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    SegSum t = s_w[0];
    uint32_t tc = s_c[0];
    SegMax tm = s_m[0];
    for (int i = 1; i < kWavesPerBlock; ++i) {
      t = op(t, s_w[i]);
      tc += s_c[i];
      tm = om(tm, s_m[i]);
    }
    tile_heads[blockIdx.x] = tc;
    tile_inc[blockIdx.x] = t;
    tile_agg[blockIdx.x] = tm;
    // the tile's first item (blocked arrangement: lane 0, item 0 of wave 0)
    tile_first[blockIdx.x] = SegMax{it.seg[0], it.s[0]};
  }
}

// Corrects the counts of the tiles listed by k_runs_carry, one wave per
// tile.  The carry c has the segment S of the tile's first item and reaches
// its start, so it changes the exclusive running maximum only of the tile's
// first items of S whose running end within the tile stays below c (a
// prefix of the tile): the first count took the first item as a run head of
// length end - start (its exclusive value came from no item), the others
// with their running end in the tile; with c they are heads only if they
// start after c, and add only what they reach beyond it.  The differences
// go into the tile's head count, and into its union sum when the whole tile
// is S (otherwise that sum is of a later segment).  The first tile is never
// listed: its carry is the empty one, as in its first count.
__global__ __launch_bounds__(kBlock) void k_runs_fix(
    int64_t n, const uint32_t* korder, const uint8_t* gpu, const uint8_t* cls,
    const int64_t* start, const int64_t* end, const SegMax* tile_pre,
    const uint32_t* fix, uint32_t* tile_heads, SegSum* tile_inc) {
  const int lane = lane_id();
  const uint32_t nfix = fix[0];
  const uint32_t w0 = blockIdx.x * kWavesPerBlock + threadIdx.x / kWave;
  for (uint32_t k = w0; k < nfix; k += gridDim.x * kWavesPerBlock) {
    const int64_t t = fix[1 + k];
    const SegMax c = tile_pre[t];
    const int64_t b = t * kOvTile;
    const int64_t te = b + kOvTile < n ? b + kOvTile : n;
    int64_t run = kI64Min;   // running end of the tile's items before
    uint32_t dh = 0;
    uint64_t di = 0;   // (differences modulo 2^64, as the sums wrap)
    for (int64_t p0 = b; p0 < te; p0 += kWave) {
      const int64_t p = p0 + lane;
      uint32_t seg = kNone;
      int64_t s = 0, e = 0;
      if (p < te) korder_gather(korder, gpu, cls, start, end, p, seg, s, e);
      const bool in = seg == c.seg;
      const int64_t incl = wave_incl(in ? e : kI64Min, OpMax(), kI64Min);
      const int64_t mo = (int64_t)wave_shr1((uint64_t)run, (uint64_t)incl);
      const int64_t m = mo > run ? mo : run;   // exclusive, within the tile
      const bool aff = in && (p == b || c.val > m);
      if (aff) {
        bool oh;
        int64_t oi;
        if (p == b) {
          // the first count's exclusive value: the empty one
          oh = c.seg != 0u || s > kI64Min;
          oi = oh ? e - s : (e > kI64Min ? e - kI64Min : 0);
        } else {
          oh = s > m;
          oi = oh ? e - s : (e > m ? e - m : 0);
        }
        const int64_t x = c.val > m ? c.val : m;
        const bool nh = s > x;
        const int64_t ni = nh ? e - s : (e > x ? e - x : 0);
        dh += (uint32_t)nh - (uint32_t)oh;
        di += (uint64_t)ni - (uint64_t)oi;
      }
      if (__ballot(!aff) != 0) break;   // the prefix ends in this chunk
      const int64_t cm = readlane64(incl, kWave - 1);
      run = cm > run ? cm : run;        // every earlier chunk's ends too
    }
    for (int d = kWave / 2; d > 0; d >>= 1) {
      dh += __shfl_xor(dh, d, kWave);
      di += __shfl_xor(di, d, kWave);
    }
    if (lane == 0) {
      tile_heads[t] += dh;
      if (tile_inc[t].seg == c.seg)
        tile_inc[t].sum = (int64_t)((uint64_t)tile_inc[t].sum + di);
    }
  }
}

// Writes the runs: start and union length before the run (the prefix of
// the segment's run lengths); every head closes the previous run at the
// running maximum, and segment starts record the run ranges.  Also fills
// the bucket index of the run starts (parameters from k_runs_spine2, table
// cleared by the first count pass) from the items: item p of segment S
// writes the entries of the buckets after its predecessor's start up to its
// own start with the number of the first run at or after p (the first run
// whose start reaches a bucket's lower bound), the segment's first item
// from bucket 0, its last item also the entries after its start with the
// segment's run end.  Over the items of S these are the entries that each
// run start and the segment's end write in a build from the run starts.
__global__ __launch_bounds__(kBlock) void k_runs_write(
    int64_t n, const uint32_t* korder, const uint8_t* gpu, const uint8_t* cls,
    const int64_t* start, const int64_t* end, const SegMax* tile_pre,
    const uint32_t* tile_run0, const SegSum* tile_inc0, const uint32_t* nruns,
    const SegMax* grand, int64_t* rs, int64_t* re, int64_t* pl,
    uint32_t* rhead, uint32_t* rbeg, uint32_t* rend, int G,
    const BSeg* bsegs, const uint32_t* kr, uint32_t* btable) {
  __shared__ int64_t s_slice[kWavesPerBlock][kSlice];
  // dynamic LDS: the 2G segments' bucket parameters, then their first item
  // positions and item ends
  extern __shared__ BSeg s_seg[];
  uint32_t* s_kr = reinterpret_cast<uint32_t*>(s_seg + 2 * G);
  for (int i = threadIdx.x; i < 2 * G; i += kBlock) {
    s_seg[i] = bsegs[i];
    s_kr[i] = kr[i];
    s_kr[2 * G + i] = kr[kSegs + i];
  }
  // (visible after the block barrier in run_items)
  // start of the item before the wave's first
  const int64_t wb0 = (int64_t)blockIdx.x * kOvTile +
                      (int64_t)(threadIdx.x / kWave) * kWaveTile;
  int64_t sbefore = 0;
  if (lane_id() == 0 && wb0 > 0 && wb0 <= n) sbefore = start[korder[wb0 - 1]];
  RunItems it;
  run_items(blockIdx.x, n, korder, gpu, cls, start, end, tile_pre,
            s_slice[threadIdx.x / kWave], it);
  const int lane = lane_id(), wv = (int)(threadIdx.x / kWave);
  OpSegSum op;
  SegSum acc = segsum_ident();
  SegSum loc[kTileIpt];
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    loc[j] = acc;
    if ((it.m_valid >> j) & 1u) acc = op(acc, SegSum{it.seg[j], 0u, it.inc[j]});
  }
  const SegSum incl = wave_incl(acc, op, segsum_ident());
  const uint32_t c = (uint32_t)__popc(it.m_head);
  const uint32_t cex = wave_prefix_small<4>(c);
  __shared__ SegSum s_w[kWavesPerBlock];
  __shared__ uint32_t s_c[kWavesPerBlock];
  if (lane == kWave - 1) {
    s_w[wv] = incl;
    s_c[wv] = cex + c;
  }
  __syncthreads();
  SegSum pre = tile_inc0[blockIdx.x];
  uint32_t r = tile_run0[blockIdx.x] + cex;
  for (int i = 0; i < kWavesPerBlock; ++i)
    if (i < wv) {
      pre = op(pre, s_w[i]);
      r += s_c[i];
    }
  pre = op(pre, wave_shr1_any(segsum_ident(), incl));
  const int64_t wbase = (int64_t)blockIdx.x * kOvTile + (int64_t)wv * kWaveTile;
  // the wave's runs are r0 .. r0 + H - 1; head k of the wave is run r0 + k
  const uint32_t r0 = r - cex;
  const uint32_t H = (uint32_t)__builtin_amdgcn_readlane((int)(cex + c), 63);
  uint32_t k[kTileIpt];
  int64_t vpl[kTileIpt];
  {
    uint32_t kk = cex;
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j) {
      k[j] = kk;
      kk += (it.m_head >> j) & 1u;
      const SegSum u = op(pre, loc[j]);
      vpl[j] = (u.seg == it.seg[j]) ? u.sum : 0;
    }
  }
  // segment ranges and the very last run (rare, scattered)
  uint32_t pseg = it.pseg0;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const int64_t p = wbase + (int64_t)lane * kTileIpt + j;
    if (((it.m_newseg >> j) & 1u)) {
      rbeg[it.seg[j]] = r0 + k[j];
      rbeg[2 * kSegs + it.seg[j]] = (uint32_t)p;     // korder positions
      if (p > 0) {
        rend[pseg] = r0 + k[j];
        rend[2 * kSegs + pseg] = (uint32_t)p;
      }
    }
    if (((it.m_valid >> j) & 1u) && p == n - 1) {
      const uint32_t R = *nruns;
      re[R - 1] = grand->val;
      rend[it.seg[j]] = R;
      rend[2 * kSegs + it.seg[j]] = (uint32_t)n;
    }
    if ((it.m_valid >> j) & 1u) pseg = it.seg[j];
  }
  // run columns, compacted through the wave's LDS slice so that the stores
  // of consecutive lanes go to consecutive runs
  int64_t* sl = s_slice[wv];
  auto emit = [&](const int64_t (&v)[kTileIpt], int64_t* dst) {
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j)
      if ((it.m_head >> j) & 1u) sl[k[j]] = v[j];
    wave_sync();
    for (uint32_t q = lane; q < H; q += kWave) dst[q] = sl[q];
    wave_sync();
  };
  emit(vpl, pl + r0);
  {
    // every head closes the previous run at the running maximum; the
    // first run of all has no predecessor
    int64_t* sl2 = sl;
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j)
      if ((it.m_head >> j) & 1u) sl2[k[j]] = it.mx[j];
    wave_sync();
    for (uint32_t q = lane; q < H; q += kWave)
      if (r0 + q > 0) re[r0 + q - 1] = sl2[q];
    wave_sync();
  }
  emit(it.s, rs + r0);
  // bucket entries of the run starts (blocked items: the predecessor of a
  // lane's first item is the lane below's last, lane 0's the item before
  // the wave)
  const int64_t sprev =
      (int64_t)wave_shr1((uint64_t)sbefore, (uint64_t)it.s[kTileIpt - 1]);
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    if (!((it.m_valid >> j) & 1u) || it.seg[j] >= (uint32_t)(2 * G)) continue;
    const uint32_t S = it.seg[j];
    const BSeg P = s_seg[S];
    if (P.nb == 0) continue;
    const int64_t p = wbase + (int64_t)lane * kTileIpt + j;
    const int64_t bi = bi_bucket(P, it.s[j]);
    const int64_t bp =
        p == (int64_t)s_kr[S] ? -1 : bi_bucket(P, j ? it.s[j - 1] : sprev);
    const uint32_t v = r0 + k[j];
    bi_fill_range(btable, P, bp, bi, v);
    if (p == (int64_t)s_kr[2 * G + S] - 1)
      bi_fill_range(btable, P, bi, P.nb, v + ((it.m_head >> j) & 1u));
  }
  {
    // segments, and the korder position of the head of every
    // communication run
    uint32_t* su = (uint32_t*)sl;
    uint32_t* sp = su + kWaveTile;
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j)
      if ((it.m_head >> j) & 1u) {
        su[k[j]] = it.seg[j];
        sp[k[j]] = (uint32_t)(wbase + (int64_t)lane * kTileIpt + j);
      }
    wave_sync();
    for (uint32_t q = lane; q < H; q += kWave)
      if (su[q] & 1u) rhead[r0 + q] = sp[q];
    wave_sync();
  }
}

// Overlapped time of the communication records (the compute-active time
// inside each), one thread per record over the dense indices of all GPUs;
// the korder tiles leave these records out, so that no tile mixes the
// window searches of compute records with these wide ones.
__device__ inline void overlap_gpu(int g, const Runs& R, int64_t* gwin);

// Block 0 also writes the GPU windows.
__global__ __launch_bounds__(kBlock) void k_comm_records(
    int G, const uint32_t* korder, const uint32_t* kbeg, const uint32_t* roff,
    const uint8_t* cdone, const int64_t* start, const int64_t* end, Runs R,
    int64_t* ovl, int64_t* gwin) {
  extern __shared__ BSeg s_seg[];   // 2G entries (dynamic LDS)
  __shared__ uint32_t s_roff[kSegs / 2 + 1];
  for (int i = threadIdx.x; i <= G; i += kBlock) s_roff[i] = roff[i];
  segs_to_lds(s_seg, R.X.seg, 2 * G);
  if (blockIdx.x == 0)
    for (int g = threadIdx.x; g < G; g += kBlock) overlap_gpu(g, R, gwin);
  const int64_t total = s_roff[G];
  for (int64_t v = (int64_t)blockIdx.x * kBlock + threadIdx.x; v < total;
       v += (int64_t)gridDim.x * kBlock) {
    if (cdone[v]) continue;        // alone in its run: written with the run
    int lo = 0, hi = G;            // the last g with roff[g] <= v
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if ((int64_t)s_roff[mid] <= v) lo = mid;
      else hi = mid;
    }
    const uint32_t r = korder[(int64_t)kbeg[2 * lo + 1] + (v - s_roff[lo])];
    const int64_t s = start[r], e0 = end[r];
    int64_t o = 0;
    if (e0 > s) {
      const BSeg P = s_seg[2 * lo];
      const int64_t t[2] = {s, e0};
      int64_t l2[2], h2[2];
      bi_range(R.X, P, s, &l2[0], &h2[0]);
      bi_range(R.X, P, e0, &l2[1], &h2[1]);
      bsearch_k<2>(R.rs, l2, h2, t);
      o = F_at(R, P, l2[1], e0) - F_at(R, P, l2[0], s);
    }
    ovl[r] = o;
  }
}

// overlapped time inside each comm run (compute-active time within it) and
// the compute-active time before it, at the run's dense index; a fixed grid
// strides over the dense indices of all GPUs
constexpr int kCommGrid = 2048;
// dense offsets (voff) of every gpu's communication runs and (roff) of its
// communication records (korder positions kbeg .. kend), from the segment
// table; every block computes them, block 0 also stores them
__device__ inline void comm_offsets(int G, const BSeg* seg,
                                    const uint32_t* kbeg, const uint32_t* kend,
                                    uint32_t* s_voff, uint32_t* s_roff,
                                    uint32_t* voff, uint32_t* roff) {
  if (threadIdx.x == 0) {
    uint32_t acc = 0, racc = 0;
    for (int g = 0; g < G; ++g) {
      s_voff[g] = acc;
      s_roff[g] = racc;
      const BSeg& P = seg[2 * g + 1];
      acc += P.se > P.sb ? P.se - P.sb : 0u;
      const uint32_t b = kbeg[2 * g + 1], e = kend[2 * g + 1];
      racc += e > b ? e - b : 0u;
    }
    s_voff[G] = acc;
    s_roff[G] = racc;
  }
  __syncthreads();
  if (blockIdx.x == 0)
    for (int i = threadIdx.x; i <= G; i += kBlock) {
      voff[i] = s_voff[i];
      roff[i] = s_roff[i];
    }
}

// Also completes the segment parameters of the run index with the run
// ranges of the write pass (every block in LDS, block 0 in memory for the
// later passes; the other fields are the same in both).
__global__ __launch_bounds__(kBlock) void k_runs_comm_overlap(
    Runs R, int G, const uint32_t* kbeg, const uint32_t* kend, uint32_t* voff,
    uint32_t* roff, int64_t* ovc, int64_t* fcrs, const uint32_t* korder,
    const uint32_t* rhead, int64_t* ovl, uint8_t* cdone, BSeg* segs_w,
    const uint32_t* rbeg, const uint32_t* rend) {
  extern __shared__ BSeg s_seg[];   // 2G entries (dynamic LDS)
  __shared__ uint32_t s_voff[kSegs / 2 + 1];
  __shared__ uint32_t s_roff[kSegs / 2 + 1];
  for (int i = threadIdx.x; i < 2 * G; i += kBlock) {
    BSeg P = R.X.seg[i];
    P.sb = rbeg[i];
    P.se = rend[i];
    s_seg[i] = P;
    if (blockIdx.x == 0) segs_w[i] = P;
  }
  __syncthreads();
  comm_offsets(G, s_seg, kbeg, kend, s_voff, s_roff, voff, roff);
  const int64_t total = s_voff[G];
  for (int64_t v = (int64_t)blockIdx.x * kBlock + threadIdx.x; v < total;
       v += (int64_t)gridDim.x * kBlock) {
    // gpu of dense index v: the last g with voff[g] <= v
    int lo = 0, hi = G;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if ((int64_t)s_voff[mid] <= v) lo = mid;
      else hi = mid;
    }
    const BSeg P = s_seg[2 * lo];
    const int64_t r = (int64_t)s_seg[2 * lo + 1].sb + (v - s_voff[lo]);
    const int64_t t[2] = {R.rs[r], R.re[r]};
    int64_t l2[2], h2[2];
    bi_range(R.X, P, t[0], &l2[0], &h2[0]);
    bi_range(R.X, P, t[1], &l2[1], &h2[1]);
    bsearch_k<2>(R.rs, l2, h2, t);
    const int64_t f = F_at(R, P, l2[0], t[0]);
    const int64_t oc = F_at(R, P, l2[1], t[1]) - f;
    ovc[v] = oc;
    fcrs[v] = f;
    // the run's records: korder positions from its head to the next run's
    // (or the segment's end); a record alone in its run spans exactly the
    // run (its end clamped to its start), so its overlapped time is the
    // run's.  Every communication record of the gpu gets its flag here.
    const BSeg Pm = s_seg[2 * lo + 1];
    const uint32_t hp = rhead[r];
    const uint32_t hq = r + 1 < (int64_t)Pm.se ? rhead[r + 1] : kend[2 * lo + 1];
    const int64_t d0 = (int64_t)s_roff[lo] - (int64_t)kbeg[2 * lo + 1];
    if (hq == hp + 1) {
      ovl[korder[hp]] = oc;
      cdone[d0 + hp] = 1;
    } else {
      for (uint32_t p = hp; p < hq; ++p) cdone[d0 + p] = 0;
    }
  }
}

// ---------------- queries ----------------------------------------------------
// Overlapped time of every record, in korder tiles of kWaveTile positions
// per wave.  Within a (gpu, kind) segment the starts are sorted, so the
// runs of the other kind that the tile's records can meet form one window:
// from the run holding the first start to the last run starting before the
// largest end.  One lane finds it through the bucket index, the wave stages
// it in LDS (coalesced), and every record searches LDS.  Records of another
// segment than the tile's first one, or tiles whose window is wider than
// kRunWin runs, search the bucket index directly.
constexpr int kRunWin = 256;

__global__ __launch_bounds__(kBlock) void k_overlap_records(
    int64_t n, int G, const uint32_t* korder, const uint8_t* gpu,
    const uint8_t* stream, const uint8_t* cls, const int64_t* start,
    const int64_t* end, Runs R, int64_t* ovl, int64_t* gap,
    uint32_t* mixed) {
  extern __shared__ BSeg s_seg[];   // 2G entries (dynamic LDS)
  __shared__ int64_t s_win[kWavesPerBlock][3][kRunWin];
  segs_to_lds(s_seg, R.X.seg, 2 * G);
  const int lane = lane_id(), wv = (int)(threadIdx.x / kWave);
  const int64_t base =
      ((int64_t)blockIdx.x * kWavesPerBlock + wv) * (int64_t)kWaveTile;
  if (base >= n) return;
  uint32_t r[kTileIpt], seg[kTileIpt], st[kTileIpt];
  int64_t s[kTileIpt], e[kTileIpt];
  uint32_t m_in = 0, m_valid = 0;   // position exists / and gpu < G
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const int64_t p = base + (int64_t)j * kWave + lane;
    const bool in = p < n;
    r[j] = korder[in ? p : base];
    seg[j] = (uint32_t)gpu[r[j]] * 2u + (uint32_t)kind_of(cls[r[j]]);
    st[j] = stream[r[j]];
    s[j] = start[r[j]];
    e[j] = end[r[j]];
    if (in) m_in |= 1u << j;
    if (in && (int)(seg[j] >> 1) < G) m_valid |= 1u << j;
  }
  // communication records are done by k_comm_records
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j)
    if (seg[j] & 1u) m_valid &= ~(1u << j);
  // the tile's main segment (its first compute item's) and the window of
  // the communication runs of that gpu
  uint32_t seg0 = kNone;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const uint64_t m = __ballot((m_valid >> j) & 1u);
    if (seg0 == kNone && m)
      seg0 = (uint32_t)__builtin_amdgcn_readlane((int)seg[j],
                                                 __ffsll((long long)m) - 1);
  }
  int64_t emax = kI64Min, smin = kI64Max;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j)
    if (((m_valid >> j) & 1u) && seg[j] == seg0) {
      emax = e[j] > emax ? e[j] : emax;
      smin = s[j] < smin ? s[j] : smin;
    }
  emax = lane63(wave_incl(emax, OpMax(), kI64Min));
  smin = lane63(wave_incl(smin, OpMin(), kI64Max));
  // seg0 = kNone: no compute record here
  const bool main_ok = seg0 != kNone && (int)(seg0 >> 1) < G;
  const BSeg Q = s_seg[main_ok ? (seg0 ^ 1u) : 0u];
  int64_t wlo = 0, whi = 0;
  if (main_ok && lane == 0) {
    int64_t lo[2], hi[2];
    const int64_t t[2] = {smin, emax};
    bi_range(R.X, Q, smin, &lo[0], &hi[0]);
    bi_range(R.X, Q, emax, &lo[1], &hi[1]);
    bsearch_k<2>(R.rs, lo, hi, t);
    wlo = lo[0] - 1 > (int64_t)Q.sb ? lo[0] - 1 : (int64_t)Q.sb;
    whi = lo[1];
  }
  // run positions fit 32 bits
  wlo = (int64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)wlo);
  whi = (int64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)whi);
  const int K = (int)(whi - wlo);
  const bool win = main_ok && K >= 0 && K <= kRunWin;
  int64_t* wrs = s_win[wv][0];
  int64_t* wre = s_win[wv][1];
  int64_t* wpl = s_win[wv][2];
  if (win) {
    for (int q = lane; q < K; q += kWave) {
      wrs[q] = R.rs[wlo + q];
      wre[q] = R.re[wlo + q];
      wpl[q] = R.pl[wlo + q];
    }
  }
  wave_sync();
  // window searches for the main segment, bucket searches for the rest;
  // the window's are searched with power-of-two steps, the same number of
  // probes in every lane, both ends at once
  const int hb = K > 0 ? 1 << (31 - __clz(K)) : 0;
  int64_t o[kTileIpt];
  uint32_t need = 0;    // records searched in the bucket index
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    o[j] = 0;
    const bool act = ((m_valid >> j) & 1u) && e[j] > s[j];
    const bool here = act && win && seg[j] == seg0;
    if (act && !here) need |= 1u << j;
    if (!here) continue;
    int ps = 0, pe = 0;   // runs starting at or before s, e
    for (int step = hb; step > 0; step >>= 1) {
      const int qs = ps + step <= K ? ps + step - 1 : K - 1;
      const int qe = pe + step <= K ? pe + step - 1 : K - 1;
      const int64_t vs = wrs[qs], ve = wrs[qe];
      ps += (ps + step <= K && vs <= s[j]) ? step : 0;
      pe += (pe + step <= K && ve <= e[j]) ? step : 0;
    }
    int64_t F[2];
#pragma unroll
    for (int z = 0; z < 2; ++z) {
      const int64_t t = z ? e[j] : s[j];
      const int q = (z ? pe : ps) - 1;
      const int qc = q >= 0 ? q : 0;
      const int64_t rs0 = wrs[qc], re0 = wre[qc], pl0 = wpl[qc];
      F[z] = q < 0 ? 0 : pl0 + ((re0 < t ? re0 : t) - rs0);
    }
    o[j] = F[1] - F[0];
  }
  // every position but the communication records of valid gpus (written
  // by k_comm_records) and the records searched below
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j)
    if (((m_in >> j) & 1u) && !((need >> j) & 1u) &&
        !((seg[j] & 1u) && (int)(seg[j] >> 1) < G))
      ovl[r[j]] = o[j];
  // Records of other segments, or tiles whose window did not fit: one
  // search code for all of them, the record picked by selects.  A compute
  // kernel's overlapped time is the comm-active time inside it and vice
  // versa.
  while (need) {
    const int jj = __builtin_ctz(need);
    need &= need - 1u;
    int64_t sj = s[0], ej = e[0];
    uint32_t gj = seg[0], rj = r[0];
#pragma unroll
    for (int j = 1; j < kTileIpt; ++j)
      if (j == jj) {
        sj = s[j];
        ej = e[j];
        gj = seg[j];
        rj = r[j];
      }
    const BSeg P = s_seg[gj ^ 1u];
    const int64_t t[2] = {sj, ej};
    int64_t lo[2], hi[2];
    bi_range(R.X, P, sj, &lo[0], &hi[0]);
    bi_range(R.X, P, ej, &lo[1], &hi[1]);
    bsearch_k<2>(R.rs, lo, hi, t);
    ovl[rj] = F_at(R, P, lo[1], ej) - F_at(R, P, lo[0], sj);
  }
  // Bubbles (Section V-D eqs. 1-3): when every GPU runs its compute
  // kernels on one stream, the previous compute record of a compute
  // record's (gpu, stream) is its predecessor in its (gpu, kind) segment of
  // korder.  Predecessors come from the lane below (lane 0: lane 63 of the
  // row above, or the position before the wave); a predecessor on another
  // stream sets *mixed, and the bubble pass then recomputes every bubble.
  {
    uint32_t lseg = kNone, lst = 0;
    int64_t lend = 0;
    if (base > 0) {
      const uint32_t rb = korder[base - 1];
      lseg = (uint32_t)gpu[rb] * 2u + (uint32_t)kind_of(cls[rb]);
      lst = stream[rb];
      lend = end[rb];
    }
    bool mix = false;
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j) {
      if (j > 0) {
        // lane 0 takes lane 63 of the row above
        lseg = wave_ror1_u32(seg[j - 1]);
        lst = wave_ror1_u32(st[j - 1]);
        const uint64_t ev = (uint64_t)e[j - 1];
        lend = (int64_t)((uint64_t)wave_ror1_u32((uint32_t)ev) |
                         (uint64_t)wave_ror1_u32((uint32_t)(ev >> 32)) << 32);
      }
      const uint32_t pseg = wave_shr1_u32(lseg, seg[j]);
      const uint32_t pst = wave_shr1_u32(lst, st[j]);
      const int64_t pe = (int64_t)wave_shr1((uint64_t)lend, (uint64_t)e[j]);
      if (!((m_in >> j) & 1u)) continue;
      int64_t gv = 0;
      if (!(seg[j] & 1u) && pseg == seg[j]) {
        mix = mix || pst != st[j];
        const int64_t b = s[j] - pe;
        gv = b > 0 ? b : 0;
      }
      gap[r[j]] = gv;
    }
    wave_flag_or(mixed, mix, 1u);
  }
}

// Window values of every marker, one per thread (more markers per thread
// in lockstep measured slower).
constexpr int kMarkPerThread = 1;

__global__ __launch_bounds__(kBlock) void k_overlap_markers(
    int64_t nm, int G, const uint8_t* mgpu, const int64_t* ms,
    const int64_t* me, Runs R, int64_t* mwin) {
  extern __shared__ BSeg s_seg[];   // 2G entries (dynamic LDS)
  segs_to_lds(s_seg, R.X.seg, 2 * G);
  const int64_t j0 =
      (int64_t)blockIdx.x * kBlock * kMarkPerThread + threadIdx.x;
  BSeg Pc[kMarkPerThread], Pm[kMarkPerThread];
  uint32_t vg[kMarkPerThread];
  int64_t a[kMarkPerThread], b[kMarkPerThread];
  bool use[kMarkPerThread];
#pragma unroll
  for (int q = 0; q < kMarkPerThread; ++q) {
    const int64_t j = j0 + (int64_t)q * kBlock;
    const uint32_t g = j < nm ? mgpu[j] : 0xFFFFFFFFu;
    use[q] = j < nm && g < (uint32_t)G;
    const uint32_t gg = use[q] ? g : 0u;
    Pc[q] = s_seg[gg * 2u];
    Pm[q] = s_seg[gg * 2u + 1u];
    vg[q] = R.voff[gg];
    a[q] = use[q] ? ms[j] : 0;
    b[q] = use[q] ? me[j] : 0;     // empty window when unused
  }
  int64_t w[kMarkPerThread][4];
  window_k<kMarkPerThread>(R, Pc, Pm, vg, a, b, w);
#pragma unroll
  for (int q = 0; q < kMarkPerThread; ++q) {
    const int64_t j = j0 + (int64_t)q * kBlock;
    if (j >= nm) continue;
    for (int z = 0; z < 4; ++z) mwin[4 * j + z] = use[q] ? w[q][z] : 0;
  }
}

// GPU window: the first run of a (gpu, kind) segment starts at its smallest
// start', the last run ends at its largest end'
__device__ inline void overlap_gpu(int g, const Runs& R, int64_t* gwin) {
  int64_t a = kI64Max, b = kI64Min;
  for (uint32_t seg = g * 2u; seg < g * 2u + 2u; ++seg) {
    const BSeg P = R.X.seg[seg];
    if (P.se > P.sb) {
      a = R.rs[P.sb] < a ? R.rs[P.sb] : a;
      b = R.re[P.se - 1] > b ? R.re[P.se - 1] : b;
    }
  }
  if (a == kI64Max) a = b = 0;
  const BSeg Pc[1] = {R.X.seg[g * 2]}, Pm[1] = {R.X.seg[g * 2 + 1]};
  const uint32_t vg[1] = {R.voff[g]};
  const int64_t aa[1] = {a}, bb[1] = {b};
  int64_t w[1][4];
  window_k<1>(R, Pc, Pm, vg, aa, bb, w);
  gwin[6 * g + 0] = a;
  gwin[6 * g + 1] = b;
  for (int z = 0; z < 4; ++z) gwin[6 * g + 2 + z] = w[0][z];
}

__global__ void k_overlap_gpus(int G, Runs R, int64_t* gwin) {
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g < G) overlap_gpu(g, R, gwin);
}

// ---------------- bubbles ----------------------------------------------------
// In (gpu, stream, start') order the bubble before a compute record is the
// time from the end of the previous compute record of the same (gpu,
// stream) to its start.  Per wave tile of `order` positions, the previous
// compute record comes from an exclusive "last compute record" scan in the
// blocked arrangement; the tile's first (gpu, stream) takes its carry by
// walking back before the tile over communication records, only when the
// tile holds a compute record of it (so each communication record is walked
// over at most once and the total work is linear).
struct LastComp {
  uint32_t key;     // (gpu, stream) of the last item; kNone: empty
  uint32_t has;     // a compute item of that key was seen
  int64_t end;      // its end
};
struct OpLastComp {
  __device__ LastComp operator()(LastComp a, LastComp b) const {
    if (b.key == kNone) return a;
    if (b.has || a.key != b.key) return b;
    return LastComp{b.key, a.has, a.end};
  }
};

__global__ __launch_bounds__(kBlock) void k_gap(
    int64_t n, const uint32_t* order, const uint8_t* gpu, const uint8_t* stream,
    const uint8_t* cls, const int64_t* start, const int64_t* end,
    const uint32_t* mixed, int64_t* gap) {
  __shared__ int64_t s_slice[kWavesPerBlock][kSlice];
  // (the compute-record pass wrote every bubble unless some GPU's compute
  // kernels run on several streams)
  if (__builtin_amdgcn_readfirstlane((int)flag_read(mixed)) == 0) return;
  const int lane = lane_id(), wv = (int)(threadIdx.x / kWave);
  const int64_t base =
      ((int64_t)blockIdx.x * kWavesPerBlock + wv) * (int64_t)kWaveTile;
  if (base >= n) return;
  int64_t* sl = s_slice[wv];
  uint32_t r[kTileIpt], key[kTileIpt], comp[kTileIpt];
  int64_t s[kTileIpt], e[kTileIpt];
  // the record before the tile, loaded with the tile's own (it usually
  // settles the carry below)
  const uint32_t rb = order[base > 0 ? base - 1 : 0];
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const int64_t p = base + (int64_t)j * kWave + lane;
    const bool in = p < n;
    r[j] = order[in ? p : base];
    key[j] = in ? (uint32_t)gpu[r[j]] * 256u + stream[r[j]] : kNone;
    comp[j] = in && !kind_of(cls[r[j]]) ? 1u : 0u;
    s[j] = start[r[j]];
    e[j] = end[r[j]];
  }
  const uint32_t kb_key = (uint32_t)gpu[rb] * 256u + stream[rb];
  const bool kb_compute = !kind_of(cls[rb]);
  const int64_t kb_end = end[rb];
  // carry into the tile for its first key
  const uint32_t key0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)key[0]);
  bool need = false;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) need = need || (comp[j] && key[j] == key0);
  LastComp carry{key0, 0u, 0};
  if (__ballot(need) != 0 && lane == 0 && base > 0) {
    // the record before the tile decides unless it is a communication
    // record of the same key; then walk further back
    int64_t q = base - 1;
    if (kb_key != key0) {
      q = -1;
    } else if (kb_compute) {
      carry.has = 1u;
      carry.end = kb_end;
      q = -1;
    } else {
      q = base - 2;
    }
    for (; q >= 0; --q) {
      const uint32_t rq = order[q];
      if ((uint32_t)gpu[rq] * 256u + stream[rq] != key0) break;
      if (!kind_of(cls[rq])) {
        carry.has = 1u;
        carry.end = end[rq];
        break;
      }
    }
  }
  carry.has = (uint32_t)__builtin_amdgcn_readfirstlane((int)carry.has);
  carry.end = (int64_t)(
      (uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)carry.end) |
      ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane(
           (int)(uint32_t)((uint64_t)carry.end >> 32)) << 32));
  // blocked arrangement
  int64_t eb[kTileIpt];
  uint32_t kb[kTileIpt], cb[kTileIpt];
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    eb[j] = e[j];
    kb[j] = key[j];
    cb[j] = comp[j];
  }
  wave_to_blocked(sl, eb, lane);
  wave_to_blocked((uint32_t*)sl, kb, lane);
  wave_to_blocked((uint32_t*)sl, cb, lane);
  OpLastComp op;
  const LastComp ident{kNone, 0u, 0};
  LastComp agg = ident;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j)
    agg = op(agg, LastComp{kb[j], cb[j], eb[j]});
  const LastComp incl = wave_incl(agg, op, ident);
  LastComp cur = op(carry, wave_shr1_any(ident, incl));
  // end of the previous compute record of the same key, per item (blocked)
  int64_t pe[kTileIpt];
  uint32_t ph[kTileIpt];
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    ph[j] = (cur.key == kb[j] && cur.has) ? 1u : 0u;
    pe[j] = cur.end;
    cur = op(cur, LastComp{kb[j], cb[j], eb[j]});
  }
  wave_to_striped(sl, pe, lane);
  wave_to_striped((uint32_t*)sl, ph, lane);
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const int64_t p = base + (int64_t)j * kWave + lane;
    if (p >= n) continue;
    int64_t gv = 0;
    if (comp[j] && ph[j]) {
      const int64_t b = s[j] - pe[j];
      gv = b > 0 ? b : 0;
    }
    gap[r[j]] = gv;
  }
}

// ---------------------------------------------------------------------------
struct OverlapLayout {
  int64_t ntiles;
  SegMax* tile_agg;
  SegMax* tile_pre;     // exclusive scan of tile_agg
  SegMax* tile_first;   // first item of every tile: (segment, start)
  uint32_t* fix;        // tiles that count again: their number, then them
  SegMax* grand;
  uint32_t* tile_heads;
  SegSum* tile_inc;
  SegSum* tile_incp;    // exclusive segmented scan of tile_inc
  SegSum* inc_total;
  uint32_t* tile_run0;
  uint32_t* nruns;
  uint32_t* scan_u32;
  int64_t* rs;
  int64_t* re;
  uint32_t* kcand;    // [2][kSegs] candidate item ranges of the segments
  uint32_t* kr;       // [2][kSegs] verified item ranges
  uint32_t* rhead;    // korder position of the head of each comm run
  uint8_t* cdone;     // comm record (dense index) done with its run
  uint32_t* mixed;    // some GPU's compute records on several streams
  uint32_t* rbeg;     // kSegs, then rend kSegs
  uint32_t* rend;
  int64_t* pl;
  int64_t* ovc;
  int64_t* pov;
  int64_t* fcrs;
  int64_t* scan_i64;
  int64_t* tot_i64;
  uint32_t* voff;
  uint32_t* roff;     // dense offsets of every gpu's communication records
  BSeg* bsegs;
  uint32_t* btable;
  int64_t btable_cap;
  uint32_t* btmp;
};

static OverlapLayout overlap_layout(Scratch& sc, int64_t n, int G) {
  OverlapLayout L;
  L.ntiles = ceil_div(n, kOvTile);
  L.tile_agg = sc.take<SegMax>(L.ntiles);
  L.tile_pre = sc.take<SegMax>(L.ntiles);
  L.tile_first = sc.take<SegMax>(L.ntiles);
  L.fix = sc.take<uint32_t>(L.ntiles + 1);
  L.grand = sc.take<SegMax>(1);
  L.tile_heads = sc.take<uint32_t>(L.ntiles);
  L.tile_inc = sc.take<SegSum>(L.ntiles);
  L.tile_incp = sc.take<SegSum>(L.ntiles);
  L.inc_total = sc.take<SegSum>(1);
  L.tile_run0 = sc.take<uint32_t>(L.ntiles);
  L.nruns = sc.take<uint32_t>(1);
  L.scan_u32 = sc.take<uint32_t>(scan_scratch_elems(L.ntiles));
  L.rs = sc.take<int64_t>(n);
  L.re = sc.take<int64_t>(n);
  L.kcand = sc.take<uint32_t>(2 * kSegs);
  L.kr = sc.take<uint32_t>(2 * kSegs);
  L.rhead = sc.take<uint32_t>(n);
  L.cdone = sc.take<uint8_t>(n);
  L.mixed = sc.take<uint32_t>(1);
  L.rbeg = sc.take<uint32_t>(4 * kSegs);   // run and korder ranges
  L.rend = L.rbeg ? L.rbeg + kSegs : nullptr;
  L.pl = sc.take<int64_t>(n);
  L.ovc = sc.take<int64_t>(n);
  L.pov = sc.take<int64_t>(n);
  L.fcrs = sc.take<int64_t>(n);
  L.scan_i64 = sc.take<int64_t>(scan_scratch_elems(n));
  L.tot_i64 = sc.take<int64_t>(2);
  L.voff = sc.take<uint32_t>(G + 1);
  L.roff = sc.take<uint32_t>(G + 1);
  L.bsegs = sc.take<BSeg>(kSegs);
  L.btable_cap = bindex_table_cap(n, kSegs);
  L.btable = sc.take<uint32_t>(L.btable_cap);
  L.btmp = sc.take<uint32_t>(kSegs + 1);
  return L;
}

}  // namespace chopper

using namespace chopper;

extern "C" int chopper_overlap(const chopper_records* rec,
                               const int64_t* start_al, const int64_t* end_al,
                               const uint32_t* order, const uint32_t* korder,
                               const chopper_markers* mk,
                               const int64_t* mstart_al, const int64_t* mend_al,
                               int64_t* ovl_out, int64_t* gap_out,
                               int64_t* mwin_out, int64_t* gwin_out,
                               void* scratch, size_t* scratch_bytes,
                               uint32_t* status, void* stream) {
  if (!validate_records(rec) || !validate_markers(mk) || !scratch_bytes)
    return CHOPPER_EINVAL;
  const int64_t n = rec->n;
  const int64_t nm = mk ? mk->n : 0;
  const int G = rec->n_gpus;
  if (n > 0 && (!start_al || !end_al || !order || !korder || !ovl_out ||
                !gap_out))
    return CHOPPER_EINVAL;
  if (nm > 0 && (!mstart_al || !mend_al || !mwin_out)) return CHOPPER_EINVAL;
  if (!gwin_out) return CHOPPER_EINVAL;
  Scratch probe(nullptr);
  overlap_layout(probe, n, G);
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  OverlapLayout L = overlap_layout(sc, n, G);
  const unsigned T = (unsigned)L.ntiles;

  if (n == 0)   // (otherwise the first count pass clears them)
    CHOPPER_HIP(launch("ov_fill", k_fill_u32, grid_for(4 * kSegs, kBlock),
                       dim3(kBlock), s, L.rbeg, (int64_t)(4 * kSegs), 0u));
  if (n > 0) {
    // union runs of every (gpu, kind)
    CHOPPER_HIP(launch("ov_runs_count", k_runs_count, dim3(T), dim3(kBlock), s,
                       n, korder, rec->gpu, rec->cls, start_al, end_al,
                       L.tile_agg, L.tile_first, L.tile_heads, L.tile_inc,
                       L.rbeg, L.mixed, L.kcand, L.btable, L.btable_cap,
                       L.fix));
    const dim3 sg((unsigned)ceil_div(L.ntiles, (int64_t)kSpineSpan));
    CHOPPER_HIP(launch("ov_runs_spine", k_runs_carry, sg, dim3(kSpineSpan), s,
                       (const SegMax*)L.tile_agg, L.tile_pre, L.ntiles,
                       L.grand, (const SegMax*)L.tile_first, L.fix));
    // (the waves loop over the listed tiles, however many there are)
    const unsigned fb = (unsigned)ceil_div(L.ntiles, (int64_t)kWavesPerBlock);
    CHOPPER_HIP(launch("ov_runs_fixup", k_runs_fix,
                       dim3(fb < kFixBlocks ? fb : kFixBlocks), dim3(kBlock),
                       s, n, korder, rec->gpu, rec->cls, start_al, end_al,
                       (const SegMax*)L.tile_pre, (const uint32_t*)L.fix,
                       L.tile_heads, L.tile_inc));
    CHOPPER_HIP(launch("ov_runs_inc_spine", k_runs_spine2, sg,
                       dim3(kSpineSpan), s, (const uint32_t*)L.tile_heads,
                       L.tile_run0, L.nruns, (const SegSum*)L.tile_inc,
                       L.tile_incp, L.inc_total, L.ntiles, G, n, korder,
                       rec->gpu, rec->cls, start_al, (const uint32_t*)L.kcand,
                       L.bsegs, L.kr, L.btable_cap));
    // (the write pass also fills the bucket index of the run starts)
    CHOPPER_HIP(launch_shm("ov_runs_write", k_runs_write, dim3(T),
                           dim3(kBlock),
                           sizeof(BSeg) * (size_t)(2 * G) +
                               sizeof(uint32_t) * (size_t)(4 * G),
                           s, n, korder, rec->gpu, rec->cls, start_al, end_al,
                           (const SegMax*)L.tile_pre,
                           (const uint32_t*)L.tile_run0,
                           (const SegSum*)L.tile_incp,
                           (const uint32_t*)L.nruns, (const SegMax*)L.grand,
                           L.rs, L.re, L.pl, L.rhead, L.rbeg, L.rend, G,
                           (const BSeg*)L.bsegs, (const uint32_t*)L.kr,
                           L.btable));
  } else {
    // no runs: empty segments
    CHOPPER_HIP(bindex_build(L.rs, (const uint32_t*)nullptr, 0, nullptr,
                             L.rbeg, L.rend, 1, kSegs, L.bsegs, L.btable,
                             L.btable_cap, L.btmp, s, false));
  }
  Runs R{L.rs, L.re, L.pl, L.pov, L.ovc, L.fcrs, L.voff,
         BIndex{L.rs, L.bsegs, L.btable}};
  // the query kernels hold the 2G segment parameters in LDS
  const size_t segs_bytes = sizeof(BSeg) * (size_t)(2 * G);
  // communication offsets (always, the marker windows read them) and the
  // overlap inside every communication run
  int64_t cg = ceil_div(n, (int64_t)kBlock);
  cg = cg < 1 ? 1 : (cg < kCommGrid ? cg : kCommGrid);
  CHOPPER_HIP(launch_shm("ov_runs_comm_overlap", k_runs_comm_overlap,
                         dim3((unsigned)cg), dim3(kBlock), segs_bytes, s, R, G,
                         (const uint32_t*)(L.rbeg + 2 * kSegs),
                         (const uint32_t*)(L.rbeg + 3 * kSegs), L.voff, L.roff,
                         L.ovc, L.fcrs, korder, (const uint32_t*)L.rhead,
                         ovl_out, L.cdone, L.bsegs, (const uint32_t*)L.rbeg,
                         (const uint32_t*)L.rend));

  if (n > 0) {

    CHOPPER_HIP(exclusive_scan<int64_t>(L.ovc, L.pov, n,
                                        (const uint32_t*)(L.voff + G),
                                        L.scan_i64, L.tot_i64 + 1, s));
    CHOPPER_HIP(launch_shm("ov_records", k_overlap_records,
                       dim3((unsigned)ceil_div(n, (int64_t)kOvTile)),
                       dim3(kBlock), segs_bytes, s, n, G, korder, rec->gpu,
                       rec->stream, rec->cls, start_al, end_al, R, ovl_out,
                       gap_out, L.mixed));
    CHOPPER_HIP(launch_shm("ov_comm_records", k_comm_records,
                           dim3((unsigned)cg), dim3(kBlock), segs_bytes, s, G,
                           korder,
                           (const uint32_t*)(L.rbeg + 2 * kSegs),
                           (const uint32_t*)L.roff, (const uint8_t*)L.cdone,
                           start_al, end_al, R, ovl_out, gwin_out));
  }
  if (nm > 0)
    CHOPPER_HIP(launch_shm("ov_markers", k_overlap_markers,
                           grid_for(nm, kBlock * kMarkPerThread),
                           dim3(kBlock), segs_bytes, s, nm, G, mk->gpu,
                           mstart_al, mend_al, R, mwin_out));
  if (n == 0)   // (otherwise the communication-records pass writes them)
    CHOPPER_HIP(launch("ov_gpus", k_overlap_gpus, grid_for(G, kBlock),
                     dim3(kBlock), s, G, R, gwin_out));
  if (n > 0) {
    CHOPPER_HIP(launch("ov_gap", k_gap,
                       dim3((unsigned)ceil_div(n, (int64_t)kOvTile)),
                       dim3(kBlock), s,
                       n, order, rec->gpu, rec->stream, rec->cls, start_al,
                       end_al, (const uint32_t*)L.mixed, gap_out));
  }
  return CHOPPER_OK;
}
