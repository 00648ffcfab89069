// chopper_attribute: every kernel record is assigned, level by level, to the
// annotation marker containing its aligned start (paper Section I
// granularities; III-A annotations for kernels, operations, layers and
// iterations).
//
// Markers are sorted by (gpu, level, empty, start') into contiguous
// per-(gpu, level) segments of non-empty markers, and a bucket index over
// each segment's starts narrows every search to a few markers.  The answer
// at a level is the last marker of the record's (gpu, level) segment whose
// start is <= the record's start, if the record starts before its end; the
// levels are independent, so a record searches all of them in lockstep.
#include "sort.h"
#include "bindex.h"
#include "wave.h"

namespace chopper {

bool validate_records(const chopper_records* r);
bool validate_markers(const chopper_markers* m);

// sorted marker columns (when the class partition did not write them)
__global__ __launch_bounds__(kBlock) void k_marker_gather(
    int64_t nm, const uint32_t* mord, const int64_t* ms, const int64_t* me,
    int64_t* sms, int64_t* sme, uint32_t* sid) {
  int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (p >= nm) return;
  uint32_t j = mord[p];
  sms[p] = ms[j];
  sme[p] = me[j];
  sid[p] = j;
}

// Overlap check between neighbours of a (gpu, level) segment and, with a
// table, the fill of the bucket index of the segment's marker starts
// (parameters and cleared table from bindex_prepare): every marker writes
// the entries between its predecessor's bucket and its own.
__global__ __launch_bounds__(kBlock) void k_marker_links(
    int G, int D, const uint32_t* coff, const int64_t* sms, const int64_t* sme,
    uint32_t* status, const BSeg* bsegs, uint32_t* btable) {
  // one block column per (gpu, level) segment
  const int seg = blockIdx.y;          // g * D + l
  const uint32_t cls = (uint32_t)seg * 2u;
  const int64_t b = coff[cls], e = coff[cls + 1];
  (void)G;
  (void)D;
  BSeg P;
  P.nb = 0;
  if (btable) P = bsegs[seg];
  bool ov = false;
  for (int64_t p = b + (int64_t)blockIdx.x * kBlock + threadIdx.x; p < e;
       p += (int64_t)gridDim.x * kBlock) {
    if (p + 1 < e && sme[p] > sms[p + 1]) ov = true;
    if (P.nb != 0) {
      const int64_t bi = bi_bucket(P, sms[p]);
      const int64_t bp = p == (int64_t)P.sb ? -1 : bi_bucket(P, sms[p - 1]);
      bi_fill_range(btable, P, bp, bi, (uint32_t)p);
      if (p == (int64_t)P.se - 1) bi_fill_range(btable, P, bi, P.nb, P.se);
    }
  }
  if (__ballot(ov) != 0 && (threadIdx.x & (kWave - 1)) == 0)
    atomicOr(status, (uint32_t)CHOPPER_ST_MARKER_OVERLAP);
}

// LDS pool per wave of marker starts, ends and ids, shared by the levels'
// windows (a wave tile of the finest level of a training trace spans a few
// hundred operation markers)
constexpr int kMarkWin = 512;

// One thread per (wave tile, level): the window of level-l markers for the
// tile's records of its first gpu, found ahead of the records kernel so that
// its waves do not wait on the search.  The tile's time range is taken from
// its first record and the last record of the same gpu (both found by
// position, exact for records in (gpu, start') order); the records kernel
// uses the window only when its records' starts lie inside that range.
// win [tile][level][2]: first marker position and count (count kNone:
// none); wt [2][tiles]: the range.
__global__ __launch_bounds__(kBlock) void k_attr_windows(
    int64_t n, int64_t ntiles, int G, int D, const uint8_t* gpu,
    const int64_t* start, BIndex X, uint32_t* win, int64_t* wt) {
  const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (t >= ntiles * D) return;
  const int64_t w = t / D;
  const int l = (int)(t - w * D);
  const int64_t base = w * (int64_t)kWaveTile;
  int64_t last = base + kWaveTile - 1 < n - 1 ? base + kWaveTile - 1 : n - 1;
  const uint32_t g0 = gpu[base];
  uint32_t* o = win + 2 * t;
  if (g0 >= (uint32_t)G) {
    o[0] = 0;
    o[1] = kNone;
    if (l == 0) {
      wt[w] = kI64Max;
      wt[ntiles + w] = kI64Min;
    }
    return;
  }
  // last position of gpu g0 in the tile (gpu ids non-decreasing there;
  // otherwise the range check of the records kernel rejects the window)
  if (gpu[last] != g0) {
    int64_t lo = base, hi = last;          // gpu[lo] == g0, gpu[hi] != g0
    while (hi - lo > 1) {
      const int64_t mid = (lo + hi) >> 1;
      if (gpu[mid] == g0) lo = mid;
      else hi = mid;
    }
    last = lo;
  }
  const int64_t smin = start[base], smax = start[last];
  if (smax < smin) {
    o[0] = 0;
    o[1] = kNone;
    if (l == 0) {
      wt[w] = kI64Max;
      wt[ntiles + w] = kI64Min;
    }
    return;
  }
  const BSeg P = X.seg[g0 * D + l];
  int64_t lo[2], hi[2];
  const int64_t tt[2] = {smin, smax};
  bi_range(X, P, smin, &lo[0], &hi[0]);
  bi_range(X, P, smax, &lo[1], &hi[1]);
  bsearch_k<2>(X.key, lo, hi, tt);
  const int64_t wlo = lo[0] - 1 > (int64_t)P.sb ? lo[0] - 1 : (int64_t)P.sb;
  const int64_t wk = lo[1] - wlo;
  o[0] = (uint32_t)wlo;
  o[1] = wk <= (int64_t)kMarkWin ? (uint32_t)wk : kNone;
  if (l == 0) {
    wt[w] = smin;
    wt[ntiles + w] = smax;
  }
}

// Records in natural order, wave tiles of kWaveTile, each lane owning eight
// consecutive records (vector loads and stores).  For the tile's first gpu,
// lane l finds the window of level-l markers that the tile's starts can
// fall in (from the marker holding the smallest start to the last one
// starting at or before the largest); the windows that fit the wave's LDS
// pool are staged there with the markers' ends and ids.  A lane searches a
// window for its first record and advances from there for the next ones,
// whose starts usually follow; records of other gpus and levels whose
// window does not fit search the bucket index.  The input order only
// affects speed.
template <int MaxD>
__global__ __launch_bounds__(kBlock) void k_attribute_records(
    int64_t n, int G, int D, const uint8_t* gpu, const int64_t* start,
    BIndex X, const int64_t* sme, const uint32_t* sid, const uint32_t* pwin,
    const int64_t* pwt, int64_t ntiles, uint32_t* idx) {
  __shared__ int64_t s_ps[kWavesPerBlock][kMarkWin];
  __shared__ int64_t s_pe[kWavesPerBlock][kMarkWin];
  __shared__ uint32_t s_pi[kWavesPerBlock][kMarkWin];
  const int lane = lane_id(), wv = (int)(threadIdx.x / kWave);
  const int64_t base =
      ((int64_t)blockIdx.x * kWavesPerBlock + wv) * (int64_t)kWaveTile;
  if (base >= n) return;
  int64_t* ps = s_ps[wv];
  int64_t* pe = s_pe[wv];
  uint32_t* pi = s_pi[wv];
  const int64_t k0 = base + (int64_t)lane * kTileIpt;   // lane's first record
  const bool full = base + kWaveTile <= n;                // uniform
  // the precomputed window of every level and its time range (loaded with
  // the records)
  const int64_t tile = base / kWaveTile;
  uint32_t pw_lo = 0, pw_k = kNone;
  if (lane < D) {
    const uint2 v = *reinterpret_cast<const uint2*>(pwin + 2 * (tile * D + lane));
    pw_lo = v.x;
    pw_k = v.y;
  }
  const int64_t pt_lo = pwt[tile], pt_hi = pwt[ntiles + tile];
  // vector loads only from suitably aligned columns
  const bool vload = full && ((uintptr_t)gpu & 7) == 0 &&
                     ((uintptr_t)start & 15) == 0;
  uint32_t g[kTileIpt];
  int64_t s[kTileIpt];
  if (vload) {
    const uint2 gv = *reinterpret_cast<const uint2*>(gpu + k0);
    const uint8_t* gb = reinterpret_cast<const uint8_t*>(&gv);
    const int4* sp = reinterpret_cast<const int4*>(start + k0);
    int64_t sv[kTileIpt];
#pragma unroll
    for (int q = 0; q < kTileIpt / 2; ++q)
      *reinterpret_cast<int4*>(&sv[2 * q]) = sp[q];
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j) {
      g[j] = gb[j];
      s[j] = sv[j];
    }
  } else {
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j) {
      const int64_t k = k0 + j;
      g[j] = k < n ? gpu[k] : 0xFFFFFFFFu;
      s[j] = k < n ? start[k] : 0;
    }
  }
  // lane l < D: window of level l -- the precomputed one when the tile's
  // starts lie in its range, else searched here.  The levels that fit the
  // pool are a prefix of the levels (offsets grow with the level), packed
  // from pool entry 0; entry q belongs to the last fitting level whose
  // offset is <= q.  Every lane issues the loads of all its entries before
  // writing any of them (one round trip to memory instead of one per level
  // and per 64 markers).
  constexpr int kStageIt = kMarkWin / kWave;
  int64_t vk[kStageIt], ve[kStageIt];
  uint32_t vi[kStageIt];
  int64_t wlo = 0, wk = 0, woff = 0;
  bool fits = false;
  auto stage_loads = [&](bool ok) {
    woff = wave_incl(wk, OpAdd(), (int64_t)0) - wk;
    fits = ok && lane < D && woff + wk <= kMarkWin;
    int64_t wl[MaxD], wn[MaxD], wo[MaxD];
#pragma unroll
    for (int l = 0; l < MaxD; ++l) {
      wl[l] = readlane64(wlo, l);
      wo[l] = readlane64(woff, l);
      wn[l] = readlane64(fits ? wk : (int64_t)-1, l);
    }
    int64_t ptot = 0;
#pragma unroll
    for (int l = 0; l < MaxD; ++l)
      if (l < D && wn[l] >= 0) ptot = wo[l] + wn[l];
#pragma unroll
    for (int i = 0; i < kStageIt; ++i) {
      const int64_t q = lane + (int64_t)i * kWave;
      if (q < ptot) {
        int64_t src = wl[0] + q - wo[0];
#pragma unroll
        for (int l = 1; l < MaxD; ++l)
          if (l < D && wn[l] >= 0 && q >= wo[l]) src = wl[l] + q - wo[l];
        vk[i] = X.key[src];
        ve[i] = sme[src];
        vi[i] = sid[src];
      }
    }
    return ptot;
  };
  // the precomputed windows' entries are loaded while the records arrive
  // (a tile of no valid gpu has none that fit)
  if (lane < D) {
    wlo = pw_lo;
    wk = pw_k == kNone ? (int64_t)kMarkWin + 1 : (int64_t)pw_k;
  }
  int64_t ptot = stage_loads(true);
  // a record is searched when it exists and its gpu is in range; records
  // past n (partial last tile) carry g = 0xFFFFFFFF and are never searched
  uint32_t m_ok = 0;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j)
    if (k0 + j < n && g[j] < (uint32_t)G) m_ok |= 1u << j;
  const uint32_t g0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)g[0]);
  const bool g0ok = g0 < (uint32_t)G;
  int64_t smin = kI64Max, smax = kI64Min;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j)
    if (((m_ok >> j) & 1u) && g[j] == g0) {
      smin = s[j] < smin ? s[j] : smin;
      smax = s[j] > smax ? s[j] : smax;
    }
  smin = lane63(wave_incl(smin, OpMin(), kI64Max));
  smax = lane63(wave_incl(smax, OpMax(), kI64Min));
  const bool pre = smin >= pt_lo && smax <= pt_hi;      // (uniform)
  if (!pre) {
    // the tile's starts leave the precomputed range: search the windows
    wlo = wk = 0;
    if (g0ok && lane < D) {
      const BSeg P = X.seg[g0 * D + lane];
      int64_t lo[2], hi[2];
      const int64_t t[2] = {smin, smax};
      bi_range(X, P, smin, &lo[0], &hi[0]);
      bi_range(X, P, smax, &lo[1], &hi[1]);
      bsearch_k<2>(X.key, lo, hi, t);
      wlo = lo[0] - 1 > (int64_t)P.sb ? lo[0] - 1 : (int64_t)P.sb;
      wk = lo[1] - wlo;
    }
    ptot = stage_loads(g0ok);
  }
#pragma unroll
  for (int i = 0; i < kStageIt; ++i) {
    const int64_t q = lane + (int64_t)i * kWave;
    if (q < ptot) {
      ps[q] = vk[i];
      pe[q] = ve[i];
      pi[q] = vi[i];
    }
  }
  wave_sync();
  // per level (one copy of the code: the level's window comes from the
  // lane that holds it): the window position of each record, then its
  // marker
#pragma unroll 1
  for (int l = 0; l < D; ++l) {
    const int wol = (int)readlane64(woff, l);
    const int nw = (int)readlane64(fits ? wk : (int64_t)-1, l);
    const int64_t* w = ps + wol;
    uint32_t out[kTileIpt];
    uint32_t need = 0;      // records searched in the bucket index
    if (nw <= 0) {
      // (uniform) no window (every record of the tile's gpu is searched)
      // or an empty one (no marker holds them)
#pragma unroll
      for (int j = 0; j < kTileIpt; ++j) {
        out[j] = kNone;
        if (((m_ok >> j) & 1u) && (nw < 0 || g[j] != g0)) need |= 1u << j;
      }
    } else {
      // window index of the last key <= t, or -1: a search with power-of-two
      // steps, the same number of probes in every lane
      const int hb = 1 << (31 - __clz(nw));
      auto search = [&](int64_t t) {
        int pos = 0;
        for (int step = hb; step > 0; step >>= 1) {
          const bool in = pos + step <= nw;
          if (in && w[in ? pos + step - 1 : nw - 1] <= t) pos += step;
        }
        return pos - 1;
      };
      int a = -1;             // window index of the previous record's key
      int64_t prev = kI64Max;
#pragma unroll
      for (int j = 0; j < kTileIpt; ++j) {
        const bool valid = (m_ok >> j) & 1u;
        const bool in = valid && g[j] == g0;
        if (valid && !in) need |= 1u << j;
        const int64_t sj = s[j];
        // a record at or after the previous one is at most two keys past
        // its key (else, and for the lane's first, a search)
        const int c0 = a >= 0 ? a : 0;
        const bool a1 = c0 + 1 < nw && w[c0 + 1 < nw ? c0 + 1 : nw - 1] <= sj;
        const int c1 = c0 + (a1 ? 1 : 0);
        const bool a2 = a1 && c1 + 1 < nw &&
                        w[c1 + 1 < nw ? c1 + 1 : nw - 1] <= sj;
        int pos = c1;
        if (in && (j == 0 || a < 0 || sj < prev || a2)) pos = search(sj);
        if (in) {
          a = pos;
          prev = sj;
        }
        // a < 0: the record starts before the window's first marker (the
        // window then begins at the segment's first marker)
        const int pc = pos >= 0 ? pos : 0;
        const int64_t mend = pe[wol + pc];
        const uint32_t mid = pi[wol + pc];
        out[j] = in && pos >= 0 && sj < mend ? mid : kNone;
      }
    }
    // another gpu, or a window that did not fit (rare): one search code for
    // all of them, the record picked by selects
    while (need) {
      const int jj = __builtin_ctz(need);
      need &= need - 1u;
      int64_t sj = s[0];
      uint32_t gj = g[0];
#pragma unroll
      for (int j = 1; j < kTileIpt; ++j)
        if (j == jj) {
          sj = s[j];
          gj = g[j];
        }
      const uint32_t sg = gj * D + l;
      const int64_t q = bi_upper(X, sg, sj) - 1;
      const uint32_t r =
          (q >= (int64_t)X.seg[sg].sb && sj < sme[q]) ? sid[q] : kNone;
#pragma unroll
      for (int j = 0; j < kTileIpt; ++j)
        if (j == jj) out[j] = r;
    }
    uint32_t* dst = idx + (int64_t)l * n + k0;
    if (full && ((uintptr_t)dst & 15) == 0) {
      uint4* d4 = reinterpret_cast<uint4*>(dst);
      d4[0] = make_uint4(out[0], out[1], out[2], out[3]);
      d4[1] = make_uint4(out[4], out[5], out[6], out[7]);
    } else {
#pragma unroll
      for (int j = 0; j < kTileIpt; ++j)
        if (k0 + j < n) dst[j] = out[j];
    }
  }
}

struct AttrLayout {
  uint32_t* mord;
  uint32_t* coff;
  int64_t* sms;
  int64_t* sme;
  uint32_t* sid;
  BSeg* bsegs;
  uint32_t* btable;
  int64_t btable_cap;
  uint32_t* btmp;
  uint32_t* pwin;     // [tiles][D][2] precomputed marker windows
  int64_t* pwt;       // [2][tiles] their time ranges
  int64_t ntiles;
  ClassSortLayout sort;
};

static AttrLayout attr_layout(Scratch& sc, int64_t n, int64_t nm, int G,
                              int D) {
  AttrLayout L;
  L.ntiles = ceil_div(n, (int64_t)kWaveTile);
  L.pwin = sc.take<uint32_t>(L.ntiles * D * 2);
  L.pwt = sc.take<int64_t>(2 * L.ntiles);
  const int C = G * D * 2 + 1;
  L.mord = sc.take<uint32_t>(nm);
  L.coff = sc.take<uint32_t>(C + 1);
  L.sms = sc.take<int64_t>(nm);
  L.sme = sc.take<int64_t>(nm);
  L.sid = sc.take<uint32_t>(nm);
  L.bsegs = sc.take<BSeg>((int64_t)G * D);
  L.btable_cap = bindex_table_cap(nm, (int64_t)G * D);
  L.btable = sc.take<uint32_t>(L.btable_cap);
  L.btmp = sc.take<uint32_t>((int64_t)G * D + 1);
  L.sort = class_sort_layout(sc, nm, C);
  return L;
}

}  // namespace chopper

using namespace chopper;

extern "C" int chopper_attribute(const chopper_records* rec,
                                 const int64_t* start_al,
                                 const chopper_markers* mk,
                                 const int64_t* mstart_al,
                                 const int64_t* mend_al, uint32_t* idx_out,
                                 void* scratch, size_t* scratch_bytes,
                                 uint32_t* status, void* stream) {
  if (!validate_records(rec) || !mk || !validate_markers(mk) || !scratch_bytes)
    return CHOPPER_EINVAL;
  const int64_t n = rec->n, nm = mk->n;
  const int G = rec->n_gpus, D = mk->depth;
  if (n > 0 && (!start_al || !idx_out)) return CHOPPER_EINVAL;
  if (nm > 0 && (!mstart_al || !mend_al)) return CHOPPER_EINVAL;
  Scratch probe(nullptr);
  attr_layout(probe, n, nm, G, D);
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  AttrLayout L = attr_layout(sc, n, nm, G, D);
  KeyMarker km{mk->gpu, mk->level, mstart_al, mend_al, G, D};
  bool range_err = false;
  // markers in start order (the usual case): the class partition writes the
  // sorted columns itself
  const MarkerColumns cols{mstart_al, mend_al, L.sms, L.sme, L.sid};
  bool gathered = false;
  rc = class_sort(km, L.sort, L.mord, L.coff, &range_err, s, -1, cols,
                  &gathered);
  if (rc != CHOPPER_OK) return rc;
  if (range_err)
    CHOPPER_HIP(launch("status_set", k_status_set, dim3(1), dim3(1), s,
                       (uint32_t)CHOPPER_ST_RANGE, status));
  // the bucket index of the non-empty marker starts of every (gpu, level)
  // is needed when there are records to attribute; the links pass fills it
  const bool index = n > 0 && D > 0;
  if (nm > 0 && !gathered)
    CHOPPER_HIP(launch("attr_marker_gather", k_marker_gather,
                       grid_for(nm, kBlock), dim3(kBlock), s, nm,
                       (const uint32_t*)L.mord, mstart_al, mend_al, L.sms,
                       L.sme, L.sid));
  if (index)
    CHOPPER_HIP(bindex_prepare(L.sms, L.coff, L.coff + 1, 2, G * D, L.bsegs,
                               L.btable, L.btable_cap, L.btmp, s));
  if (nm > 0) {
    const int64_t per_seg = ceil_div(nm, (int64_t)G * D);
    unsigned gx = (unsigned)ceil_div(per_seg, kBlock);
    if (gx < 1) gx = 1;
    if (gx > 1024) gx = 1024;
    CHOPPER_HIP(launch("attr_marker_links", k_marker_links,
                       dim3(gx, (unsigned)(G * D)), dim3(kBlock), s, G, D,
                       (const uint32_t*)L.coff, (const int64_t*)L.sms,
                       (const int64_t*)L.sme, status,
                       (const BSeg*)L.bsegs,
                       index ? L.btable : (uint32_t*)nullptr));
  }
  if (!index) return CHOPPER_OK;
  const BIndex X{L.sms, L.bsegs, L.btable};
  const unsigned grid = (unsigned)ceil_div(n, (int64_t)kWaveTile * kWavesPerBlock);
  CHOPPER_HIP(launch("attr_windows", k_attr_windows,
                     grid_for(L.ntiles * D, kBlock), dim3(kBlock), s, n,
                     L.ntiles, G, D, rec->gpu, start_al, X, L.pwin, L.pwt));
  auto run = [&](auto kern) -> int {
    CHOPPER_HIP(launch("attr_records", kern, dim3(grid), dim3(kBlock), s, n,
                       G, D, rec->gpu, start_al, X, (const int64_t*)L.sme,
                       (const uint32_t*)L.sid, (const uint32_t*)L.pwin,
                       (const int64_t*)L.pwt, L.ntiles, idx_out));
    return CHOPPER_OK;
  };
  if (D <= 4) return run(k_attribute_records<4>);
  return run(k_attribute_records<8>);
}
