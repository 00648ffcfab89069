// chopper_aggregate: metric aggregation at every granularity (paper Section
// III-C; granularities of Section I; duration and launch overhead as sums of
// kernel durations and bubbles, caption of Fig. end_to_end).
//
// Records are visited in (gpu, kind, start') order.  At marker level l the
// group of a record is identified by its deepest non-NONE marker among
// levels 0..l (or its GPU when all are NONE) and its kind; for nested
// markers that marker determines the whole path.  Rows are numbered in order
// of each group's first record:
//   1. election: atomicMin of the record position into a per-level owner
//      table keyed by group (only at positions where the key changes);
//   2. owners are counted per tile and one exclusive scan over the
//      level-major table of tile counts yields final row numbers, level
//      offsets included;
//   3. owners write the row header (path, gpu, kind, first record);
//   4. segmented reductions: tiles of 2048 items, eight consecutive items
//      per thread, a thread-local pass plus one block-wide segmented scan per
//      field.  The piece holding a row's first item stores the row; other
//      pieces of the same row (rare: the group's records are not
//      consecutive) go through a small overflow list applied with atomics.
// The finest level reads the records (counters exactly once); each coarser
// level reads the rows of the level below.  GPU and workload rows, which
// are few, accumulate with atomics.
#include <type_traits>

#include "sort.h"
#include "wave.h"

namespace chopper {

bool validate_records(const chopper_records* r);
bool validate_markers(const chopper_markers* m);

constexpr int kAggIpt = 8;
constexpr int kAggTile = kBlock * kAggIpt;
constexpr int kMaxLevels = 10;            // depth <= 8, + GPU + workload
constexpr int kMaxFields = 6 + 16;        // n dur gap ovl tmin tmax ctr[16]

struct FilterDev {
  uint64_t gpu_mask[4];
  uint32_t class_mask;
  uint32_t use_iter;
  uint32_t iter_lo, iter_hi;
  uint32_t active;
};

struct RecSrc {
  int64_t n;
  int D;
  int64_t M;
  const uint32_t* korder;
  const uint8_t* gpu;
  const uint8_t* cls;
  const int64_t* start;
  const int64_t* end;
  const uint32_t* idx;
  const int64_t* gap;
  const int64_t* ovl;
  const uint64_t* ctr;
  int nc;
  const uint32_t* mlabel;
  FilterDev f;
  // exact group ids of the marker levels ([D][n] by korder position), or
  // null: groups by the deepest marker (exact for nested markers)
  const uint32_t* gk;
  // the general path's items gathered once in korder position order (or
  // null: gathered through korder where used): marker path [D][n] and
  // gpu * 2 + kind (0xFFFF: left out by the filter)
  const uint32_t* ipath;
  const uint16_t* igk;
};

struct RowsDev {
  int64_t cap;
  uint32_t* path;
  uint8_t* gpu;
  uint8_t* kind;
  uint64_t* n;
  int64_t* dur;
  int64_t* gap;
  int64_t* ovl;
  int64_t* tmin;
  int64_t* tmax;
  uint32_t* first;
  uint64_t* ctr;
  uint32_t* firstpos;   // scratch: korder position of each row's first record
  int D;
  int nc;
};

// key space of a level
__host__ __device__ inline int64_t key_space(int li, int D, int64_t M) {
  if (li < D) return 2 * (M + 256);
  if (li == D) return 512;
  return 2;
}

__device__ inline bool rec_pass(const RecSrc& S, uint32_t r) {
  if (!S.f.active) return true;
  const uint32_t g = S.gpu[r], c = S.cls[r];
  if (!((S.f.gpu_mask[g >> 6] >> (g & 63)) & 1ull)) return false;
  if (c >= 32 || !((S.f.class_mask >> c) & 1u)) return false;
  if (S.f.use_iter) {
    if (S.D < 1) return false;
    const uint32_t m0 = S.idx[r];
    if (m0 == kNone || (int64_t)m0 >= S.M) return false;
    const uint32_t lab = S.mlabel[m0];
    if (lab < S.f.iter_lo || lab > S.f.iter_hi) return false;
  }
  return true;
}

// group key of a record with path p at level li (kNone: not aggregated)
__device__ inline uint32_t group_key(const uint32_t* p, int D, int64_t M,
                                     int li, uint32_t g, uint32_t kind) {
  if (li < D) {
    uint32_t slot = kNone;
    for (int l = 0; l <= li; ++l)
      if (p[l] != kNone) slot = p[l];
    if (slot == kNone) return (uint32_t)((M + g) * 2 + kind);
    if ((int64_t)slot >= M) return kNone;
    return slot * 2u + kind;
  }
  if (li == D) return g * 2u + kind;
  return kind;
}

// key of an item at level li: its exact group id at the marker levels when
// those are given (fpos = korder position of the item, or of the first
// record of a row), else the deepest-marker key
__device__ inline uint32_t item_key(const uint32_t* gk, int64_t nrec,
                                    const uint32_t* p, int D, int64_t M,
                                    int li, uint32_t g, uint32_t kind,
                                    uint32_t fpos) {
  if (gk && li < D) return gk[(int64_t)li * nrec + fpos];
  return group_key(p, D, M, li, g, kind);
}

// One record position: its record, pass flag, gpu, kind and path.
struct RecItem {
  uint32_t r;
  bool ok;
  uint32_t g, kind;
  uint32_t p[8];
};

__device__ inline void load_item(const RecSrc& S, int64_t pos, RecItem& it) {
  it.r = S.korder[pos];
  if (S.igk) {
    const uint32_t v = S.igk[pos];
    it.ok = v != 0xFFFFu;
    it.g = (v >> 1) & 255u;
    it.kind = v & 1u;
    for (int l = 0; l < S.D; ++l) it.p[l] = S.ipath[(int64_t)l * S.n + pos];
    return;
  }
  it.g = S.gpu[it.r];
  it.kind = (uint32_t)kind_of(S.cls[it.r]);
  it.ok = rec_pass(S, it.r);
  for (int l = 0; l < S.D; ++l) it.p[l] = S.idx[(int64_t)l * S.n + it.r];
}

// The general path's items in korder position order, gathered once.
__global__ __launch_bounds__(kBlock) void k_agg_items(RecSrc S, uint32_t* ipath,
                                                      uint16_t* igk) {
  const int64_t pos = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (pos >= S.n) return;
  const uint32_t r = S.korder[pos];
  const uint32_t g = S.gpu[r];
  const uint32_t kind = (uint32_t)kind_of(S.cls[r]);
  igk[pos] = rec_pass(S, r) ? (uint16_t)(g * 2u + kind) : (uint16_t)0xFFFFu;
  for (int l = 0; l < S.D; ++l)
    ipath[(int64_t)l * S.n + pos] = S.idx[(int64_t)l * S.n + r];
}

// ------------------------------------------------------------------ election
__global__ __launch_bounds__(kBlock) void k_agg_elect(RecSrc S, uint32_t act,
                                                      uint32_t** own) {
  __shared__ uint32_t s_last[kBlock];
  const int64_t base = (int64_t)blockIdx.x * kAggTile;
  RecItem it[kAggIpt];
  bool valid[kAggIpt];
  for (int j = 0; j < kAggIpt; ++j) {
    const int64_t pos = base + (int64_t)threadIdx.x * kAggIpt + j;
    valid[j] = pos < S.n;
    if (valid[j]) load_item(S, pos, it[j]);
  }
  for (int li = 0; li < S.D + 2; ++li) {
    if (!((act >> li) & 1u)) continue;
    uint32_t key[kAggIpt];
    for (int j = 0; j < kAggIpt; ++j) {
      const int64_t pos = base + (int64_t)threadIdx.x * kAggIpt + j;
      key[j] = (valid[j] && it[j].ok)
                   ? item_key(S.gk, S.n, it[j].p, S.D, S.M, li, it[j].g,
                              it[j].kind, (uint32_t)pos)
                   : kNone;
    }
    s_last[threadIdx.x] = key[kAggIpt - 1];
    __syncthreads();
    uint32_t prev = threadIdx.x > 0 ? s_last[threadIdx.x - 1] : kNone;
    for (int j = 0; j < kAggIpt; ++j) {
      const bool head = (threadIdx.x == 0 && j == 0) || key[j] != prev;
      if (key[j] != kNone && head) {
        const int64_t pos = base + (int64_t)threadIdx.x * kAggIpt + j;
        atomicMin(&own[li][key[j]], (uint32_t)pos);
      }
      prev = key[j];
    }
    __syncthreads();
  }
}

// owners per tile and level: position pos owns its key at level li
__global__ __launch_bounds__(kBlock) void k_agg_count(RecSrc S, uint32_t act,
                                                      uint32_t** own,
                                                      int64_t ntiles,
                                                      uint32_t* tilecnt) {
  const int64_t base = (int64_t)blockIdx.x * kAggTile;
  RecItem it[kAggIpt];
  bool valid[kAggIpt];
  for (int j = 0; j < kAggIpt; ++j) {
    const int64_t pos = base + (int64_t)threadIdx.x * kAggIpt + j;
    valid[j] = pos < S.n;
    if (valid[j]) load_item(S, pos, it[j]);
  }
  for (int li = 0; li < S.D + 2; ++li) {
    uint32_t c = 0;
    if ((act >> li) & 1u) {
      for (int j = 0; j < kAggIpt; ++j) {
        if (!valid[j] || !it[j].ok) continue;
        const int64_t pos = base + (int64_t)threadIdx.x * kAggIpt + j;
        const uint32_t key = item_key(S.gk, S.n, it[j].p, S.D, S.M, li,
                                      it[j].g, it[j].kind, (uint32_t)pos);
        if (key != kNone && own[li][key] == (uint32_t)pos) ++c;
      }
    }
    uint32_t tot;
    block_exclusive(c, OpAdd(), 0u, &tot);
    if (threadIdx.x == 0) tilecnt[(int64_t)li * ntiles + blockIdx.x] = tot;
  }
}

__global__ void k_agg_offsets(int L, int64_t ntiles, const uint32_t* tilebase,
                              const uint32_t* total, int64_t cap,
                              int64_t* level_offset, uint32_t* status) {
  const int li = threadIdx.x;
  if (li < L) level_offset[li] = ntiles > 0 ? tilebase[(int64_t)li * ntiles] : 0;
  if (li == L) {
    level_offset[L] = *total;
    if ((int64_t)*total > cap) atomicOr(status, (uint32_t)CHOPPER_ST_ROWS_OVERFLOW);
  }
}

// owners take their row: rowof[key] = row, header fields, and (atomic levels)
// initial sums
__global__ __launch_bounds__(kBlock) void k_agg_assign(
    RecSrc S, uint32_t act, uint32_t atomic_levels, uint32_t** own,
    uint32_t** rowof, int64_t ntiles, const uint32_t* tilebase, RowsDev R) {
  const int64_t base = (int64_t)blockIdx.x * kAggTile;
  RecItem it[kAggIpt];
  bool valid[kAggIpt];
  for (int j = 0; j < kAggIpt; ++j) {
    const int64_t pos = base + (int64_t)threadIdx.x * kAggIpt + j;
    valid[j] = pos < S.n;
    if (valid[j]) load_item(S, pos, it[j]);
  }
  for (int li = 0; li < S.D + 2; ++li) {
    if (!((act >> li) & 1u)) continue;   // uniform across the block
    uint32_t key[kAggIpt];
    bool mine[kAggIpt];
    uint32_t c = 0;
    for (int j = 0; j < kAggIpt; ++j) {
      const int64_t pos = base + (int64_t)threadIdx.x * kAggIpt + j;
      key[j] = (valid[j] && it[j].ok)
                   ? item_key(S.gk, S.n, it[j].p, S.D, S.M, li, it[j].g,
                              it[j].kind, (uint32_t)pos)
                   : kNone;
      mine[j] = key[j] != kNone && own[li][key[j]] == (uint32_t)pos;
      c += mine[j] ? 1u : 0u;
    }
    uint32_t tot;
    uint32_t row = block_exclusive(c, OpAdd(), 0u, &tot) +
                   tilebase[(int64_t)li * ntiles + blockIdx.x];
    for (int j = 0; j < kAggIpt; ++j) {
      if (!mine[j]) continue;
      const int64_t pos = base + (int64_t)threadIdx.x * kAggIpt + j;
      if (li == S.D + 1) {
        // workload rows span GPUs: ordered by kind alone
        row = tilebase[(int64_t)li * ntiles] +
              ((it[j].kind == 1u && own[li][0] != kNone) ? 1u : 0u);
      }
      rowof[li][key[j]] = row;
      if ((int64_t)row < R.cap) {
        for (int l = 0; l < S.D; ++l)
          R.path[(int64_t)l * R.cap + row] =
              (li < S.D && l <= li) ? it[j].p[l] : kNone;
        R.gpu[row] = (li == S.D + 1) ? (uint8_t)0xFF : (uint8_t)it[j].g;
        R.kind[row] = (uint8_t)it[j].kind;
        // workload rows: fixed after the reduction (k_agg_workload_first)
        R.first[row] = (li == S.D + 1) ? kNone : it[j].r;
        R.firstpos[row] = (uint32_t)pos;
        if ((atomic_levels >> li) & 1u) {
          R.n[row] = 0;
          R.dur[row] = 0;
          R.gap[row] = 0;
          R.ovl[row] = 0;
          R.tmin[row] = kI64Max;
          R.tmax[row] = kI64Min;
          for (int q = 0; q < R.nc; ++q) R.ctr[(int64_t)q * R.cap + row] = 0;
        }
      }
      ++row;
    }
  }
}

// ------------------------------------------------------------------ reduction
template <typename T>
struct FV {
  uint32_t f;
  T v;
};
template <typename T>
__device__ inline FV<T> shfl_up(FV<T> x, int d) {
  FV<T> r;
  r.f = __shfl_up(x.f, d, kWave);
  r.v = __shfl_up(x.v, d, kWave);
  return r;
}

struct CombAdd {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return a + b; }
};
struct CombMin {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const {
    return (int64_t)a < (int64_t)b ? a : b;
  }
};
struct CombMax {
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const {
    return (int64_t)a > (int64_t)b ? a : b;
  }
};
struct CombLeft {
  __device__ uint64_t operator()(uint64_t a, uint64_t) const { return a; }
};

template <typename Comb>
struct OpSeg {
  Comb c;
  __device__ FV<uint64_t> operator()(FV<uint64_t> a, FV<uint64_t> b) const {
    return FV<uint64_t>{a.f | b.f, b.f ? b.v : c(a.v, b.v)};
  }
};

// Segmented inclusive scan over the tile; items are blocked (thread t owns
// items t*kAggIpt ..).  head[j] starts a new segment.
template <typename Comb>
__device__ inline void seg_scan(const bool (&head)[kAggIpt],
                                uint64_t (&x)[kAggIpt], uint64_t identity,
                                Comb comb) {
  FV<uint64_t> acc{0u, identity};
  for (int j = 0; j < kAggIpt; ++j) {
    if (head[j]) acc = FV<uint64_t>{1u, x[j]};
    else acc.v = comb(acc.v, x[j]);
    x[j] = acc.v;
  }
  FV<uint64_t> tot;
  FV<uint64_t> pre = block_exclusive(acc, OpSeg<Comb>{comb},
                                     FV<uint64_t>{0u, identity}, &tot);
  bool seen = false;
  for (int j = 0; j < kAggIpt; ++j) {
    seen = seen || head[j];
    if (!seen) x[j] = comb(pre.v, x[j]);
  }
}

struct FieldRef {
  const uint64_t* a;
  const uint64_t* b;
  int mode;
  __device__ uint64_t get(uint32_t r) const {
    if (mode == 0) return 1ull;
    if (mode == 1) return a[r] - b[r];
    return a[r];
  }
};

// column of row field f (same bits for the signed columns)
__device__ inline uint64_t* row_column(const RowsDev& R, int f) {
  switch (f) {
    case 0: return R.n;
    case 1: return (uint64_t*)R.dur;
    case 2: return (uint64_t*)R.gap;
    case 3: return (uint64_t*)R.ovl;
    case 4: return (uint64_t*)R.tmin;
    case 5: return (uint64_t*)R.tmax;
    default: return R.ctr + (int64_t)(f - 6) * R.cap;
  }
}

// Item sources for the reduction: records in korder, or rows of a finer
// level.  Fields: 0 n, 1 dur, 2 gap, 3 ovl, 4 tmin, 5 tmax, 6.. counters.
struct FromRecords {
  static constexpr bool kRecords = true;
  RecSrc S;
  // columns of the fast reduction: start and end give n (no load), dur,
  // tmin and tmax; the plain sums are gap, ovl and the counters
  __device__ const int64_t* start_col() const { return S.start; }
  __device__ const int64_t* end_col() const { return S.end; }
  __device__ int nsum() const { return 2 + S.nc; }
  __device__ const uint64_t* sum_col(int i) const {
    if (i == 0) return (const uint64_t*)S.gap;
    if (i == 1) return (const uint64_t*)S.ovl;
    return S.ctr + (int64_t)(i - 2) * S.n;
  }
  __device__ int sum_dst(int i) const { return i < 2 ? 2 + i : 6 + (i - 2); }
  __device__ int64_t count() const { return S.n; }
  __device__ void load(int64_t i, uint32_t& r, bool& ok, uint32_t* p,
                       uint32_t& g, uint32_t& kind, uint32_t& fpos) const {
    RecItem it;
    load_item(S, i, it);
    r = it.r;
    g = it.g;
    kind = it.kind;
    ok = it.ok;
    for (int l = 0; l < S.D; ++l) p[l] = it.p[l];
    fpos = (uint32_t)i;
  }
  __device__ uint32_t first_of(uint32_t r) const { return r; }
  __device__ uint32_t index(int64_t i) const { return S.korder[i]; }
  __device__ bool ok(uint32_t r) const { return rec_pass(S, r); }
  __device__ uint32_t pathv(uint32_t r, int l) const {
    return S.idx[(int64_t)l * S.n + r];
  }
  __device__ uint32_t gpuv(uint32_t r) const { return S.gpu[r]; }
  __device__ uint32_t kindv(uint32_t r) const {
    return (uint32_t)kind_of(S.cls[r]);
  }
  __device__ uint32_t keyof(uint32_t r, int li) const {
    if (!rec_pass(S, r)) return kNone;
    uint32_t p[8];
    for (int l = 0; l < S.D; ++l) p[l] = pathv(r, l);
    return group_key(p, S.D, S.M, li, gpuv(r), kindv(r));
  }
  __device__ uint32_t key_at(int li, const uint32_t* p, uint32_t g,
                             uint32_t kind, uint32_t fpos) const {
    return item_key(S.gk, S.n, p, S.D, S.M, li, g, kind, fpos);
  }
  // column of field f, resolved once per field: mode 0 constant 1,
  // 1 a[r] - b[r], 2 a[r]
  __device__ FieldRef fref(int f) const {
    switch (f) {
      case 0: return FieldRef{nullptr, nullptr, 0};
      case 1: return FieldRef{(const uint64_t*)S.end, (const uint64_t*)S.start, 1};
      case 2: return FieldRef{(const uint64_t*)S.gap, nullptr, 2};
      case 3: return FieldRef{(const uint64_t*)S.ovl, nullptr, 2};
      case 4: return FieldRef{(const uint64_t*)S.start, nullptr, 2};
      case 5: return FieldRef{(const uint64_t*)S.end, nullptr, 2};
      default: return FieldRef{S.ctr + (int64_t)(f - 6) * S.n, nullptr, 2};
    }
  }
  __device__ uint64_t field(int f, uint32_t r) const {
    switch (f) {
      case 0: return 1ull;
      case 1: return (uint64_t)(S.end[r] - S.start[r]);
      case 2: return (uint64_t)S.gap[r];
      case 3: return (uint64_t)S.ovl[r];
      case 4: return (uint64_t)S.start[r];
      case 5: return (uint64_t)S.end[r];
      default: return S.ctr[(int64_t)(f - 6) * S.n + r];
    }
  }
};

struct FromRows {
  static constexpr bool kRecords = false;
  RowsDev R;
  int64_t M;        // number of markers (key space)
  const int64_t* level_offset;
  int lo_slot;      // level_offset index of the finer level
  const uint32_t* gk = nullptr;   // exact group ids (RecSrc::gk) or null
  int64_t nrec = 0;               // records (row stride of gk)
  // columns of the fast reduction: tmin and tmax, then the plain sums
  // n, dur, gap, ovl and the counters
  __device__ const int64_t* start_col() const { return R.tmin; }
  __device__ const int64_t* end_col() const { return R.tmax; }
  __device__ int nsum() const { return 4 + R.nc; }
  __device__ const uint64_t* sum_col(int i) const {
    if (i < 4) return (const uint64_t*)row_column(R, i);
    return R.ctr + (int64_t)(i - 4) * R.cap;
  }
  __device__ int sum_dst(int i) const { return i < 4 ? i : 6 + (i - 4); }
  __device__ int64_t count() const {
    int64_t a = level_offset[lo_slot], b = level_offset[lo_slot + 1];
    if (b > R.cap) b = R.cap;
    return b > a ? b - a : 0;
  }
  __device__ void load(int64_t i, uint32_t& r, bool& ok, uint32_t* p,
                       uint32_t& g, uint32_t& kind, uint32_t& fpos) const {
    r = (uint32_t)(level_offset[lo_slot] + i);
    g = R.gpu[r];
    kind = R.kind[r];
    ok = true;
    for (int l = 0; l < R.D; ++l) p[l] = R.path[(int64_t)l * R.cap + r];
    fpos = R.firstpos[r];
  }
  __device__ uint32_t first_of(uint32_t r) const { return R.first[r]; }
  __device__ uint32_t index(int64_t i) const {
    return (uint32_t)(level_offset[lo_slot] + i);
  }
  __device__ bool ok(uint32_t) const { return true; }
  __device__ uint32_t pathv(uint32_t r, int l) const {
    return R.path[(int64_t)l * R.cap + r];
  }
  __device__ uint32_t gpuv(uint32_t r) const { return R.gpu[r]; }
  __device__ uint32_t kindv(uint32_t r) const { return R.kind[r]; }
  __device__ uint32_t keyof(uint32_t r, int li) const {
    uint32_t p[8];
    for (int l = 0; l < R.D; ++l) p[l] = pathv(r, l);
    return group_key(p, R.D, M, li, gpuv(r), kindv(r));
  }
  __device__ uint32_t key_at(int li, const uint32_t* p, uint32_t g,
                             uint32_t kind, uint32_t fpos) const {
    return item_key(gk, nrec, p, R.D, M, li, g, kind, fpos);
  }
  __device__ FieldRef fref(int f) const {
    return FieldRef{(const uint64_t*)row_column(R, f), nullptr, 2};
  }
  __device__ uint64_t field(int f, uint32_t r) const {
    switch (f) {
      case 0: return R.n[r];
      case 1: return (uint64_t)R.dur[r];
      case 2: return (uint64_t)R.gap[r];
      case 3: return (uint64_t)R.ovl[r];
      case 4: return (uint64_t)R.tmin[r];
      case 5: return (uint64_t)R.tmax[r];
      default: return R.ctr[(int64_t)(f - 6) * R.cap + r];
    }
  }
};

struct Overflow {
  uint32_t* count;   // entries requested
  uint32_t* lost;    // sticky: set when an entry did not fit
  uint32_t* row;
  uint64_t* val;     // [kMaxFields][cap]
  int64_t cap;
};

__device__ inline void store_field(RowsDev& R, int f, uint32_t row,
                                   uint64_t v) {
  switch (f) {
    case 0: R.n[row] = v; break;
    case 1: R.dur[row] = (int64_t)v; break;
    case 2: R.gap[row] = (int64_t)v; break;
    case 3: R.ovl[row] = (int64_t)v; break;
    case 4: R.tmin[row] = (int64_t)v; break;
    case 5: R.tmax[row] = (int64_t)v; break;
    default: R.ctr[(int64_t)(f - 6) * R.cap + row] = v; break;
  }
}

__device__ inline void atomic_field(RowsDev& R, int f, uint32_t row,
                                    uint64_t v) {
  switch (f) {
    case 0: atomicAdd((unsigned long long*)&R.n[row], (unsigned long long)v); break;
    case 1: atomicAdd((unsigned long long*)&R.dur[row], (unsigned long long)v); break;
    case 2: atomicAdd((unsigned long long*)&R.gap[row], (unsigned long long)v); break;
    case 3: atomicAdd((unsigned long long*)&R.ovl[row], (unsigned long long)v); break;
    case 4: atomicMin((long long*)&R.tmin[row], (long long)v); break;
    case 5: atomicMax((long long*)&R.tmax[row], (long long)v); break;
    default:
      atomicAdd((unsigned long long*)&R.ctr[(int64_t)(f - 6) * R.cap + row],
                (unsigned long long)v);
      break;
  }
}

template <typename Src>
__global__ __launch_bounds__(kBlock) void k_agg_reduce(
    Src src, int li, int D, int64_t M, bool atomic_mode, const uint32_t* own,
    const uint32_t* rowof, RowsDev R, Overflow ovf, int nfields,
    uint32_t* status, uint32_t* cflag) {
  __shared__ uint32_t s_last[kBlock];
  __shared__ uint32_t s_head0[kBlock];
  const int64_t cnt = src.count();
  const int64_t base = (int64_t)blockIdx.x * kAggTile;
  if (base >= cnt) return;   // uniform: whole block
  uint32_t rid[kAggIpt], tgt[kAggIpt];
  bool head[kAggIpt], last[kAggIpt], valid[kAggIpt];
  uint64_t ownbit[kAggIpt];
  bool conflict = false;
  for (int j = 0; j < kAggIpt; ++j) {
    const int64_t i = base + (int64_t)threadIdx.x * kAggIpt + j;
    valid[j] = i < cnt;
    tgt[j] = kNone;
    ownbit[j] = 0;
    rid[j] = 0;
    if (!valid[j]) continue;
    uint32_t p[8], g, kind, fpos;
    bool ok;
    src.load(i, rid[j], ok, p, g, kind, fpos);
    if (!ok) continue;
    const uint32_t key = src.key_at(li, p, g, kind, fpos);
    if (key == kNone) continue;
    const uint32_t row = rowof[key];
    tgt[j] = row;
    ownbit[j] = (!atomic_mode && own[key] == fpos) ? 1ull : 0ull;
    // the row holds its first item's path: another path here means a
    // marker shared by different paths (markers not nested); past the
    // capacity the first item is read instead
    if (li < D) {
      if ((int64_t)row < R.cap) {
        for (int l = 0; l <= li; ++l)
          if (R.path[(int64_t)l * R.cap + row] != p[l]) conflict = true;
      } else if constexpr (Src::kRecords) {
        // (rows of a coarser level always precede those of a finer one, so
        // only the records' level has items past the capacity)
        const uint32_t ro = src.S.korder[own[key]];
        for (int l = 0; l <= li; ++l)
          if (src.S.idx[(int64_t)l * src.S.n + ro] != p[l]) conflict = true;
      }
    }
  }
  wave_flag_or(status, conflict, (uint32_t)CHOPPER_ST_PATH_CONFLICT);
  wave_flag_or(cflag, conflict, 1u);
  // piece boundaries
  s_last[threadIdx.x] = tgt[kAggIpt - 1];
  __syncthreads();
  uint32_t prev = threadIdx.x > 0 ? s_last[threadIdx.x - 1] : kNone;
  for (int j = 0; j < kAggIpt; ++j) {
    head[j] = (threadIdx.x == 0 && j == 0) || !valid[j] || tgt[j] != prev;
    prev = tgt[j];
  }
  s_head0[threadIdx.x] = head[0] ? 1u : 0u;
  __syncthreads();
  for (int j = 0; j < kAggIpt; ++j) {
    bool next_head;
    if (j + 1 < kAggIpt) next_head = head[j + 1];
    else next_head = threadIdx.x + 1 < kBlock ? s_head0[threadIdx.x + 1] != 0 : true;
    last[j] = valid[j] && tgt[j] != kNone && next_head;
  }
  // is the piece the first piece of its row? (propagated from the head)
  seg_scan(head, ownbit, 0ull, CombLeft());
  // overflow slots for non-first pieces
  uint32_t slot[kAggIpt];
  for (int j = 0; j < kAggIpt; ++j) {
    slot[j] = kNone;
    if (last[j] && !atomic_mode && ownbit[j] == 0 && (int64_t)tgt[j] < R.cap) {
      uint32_t e = atomicAdd(ovf.count, 1u);
      if ((int64_t)e < ovf.cap) {
        slot[j] = e;
        ovf.row[e] = tgt[j];
      } else {
        atomicOr(ovf.lost, 1u);
      }
    }
  }
  for (int f = 0; f < nfields; ++f) {
    uint64_t x[kAggIpt];
    for (int j = 0; j < kAggIpt; ++j) {
      const bool use = valid[j] && tgt[j] != kNone;
      if (f == 4) x[j] = use ? src.field(f, rid[j]) : (uint64_t)kI64Max;
      else if (f == 5) x[j] = use ? src.field(f, rid[j]) : (uint64_t)kI64Min;
      else x[j] = use ? src.field(f, rid[j]) : 0ull;
    }
    if (f == 4) seg_scan(head, x, (uint64_t)kI64Max, CombMin());
    else if (f == 5) seg_scan(head, x, (uint64_t)kI64Min, CombMax());
    else seg_scan(head, x, 0ull, CombAdd());
    for (int j = 0; j < kAggIpt; ++j) {
      if (!last[j] || (int64_t)tgt[j] >= R.cap) continue;
      if (atomic_mode) atomic_field(R, f, tgt[j], x[j]);
      else if (ownbit[j]) store_field(R, f, tgt[j], x[j]);
      else if (slot[j] != kNone) ovf.val[(int64_t)f * ovf.cap + slot[j]] = x[j];
    }
  }
}

// ------------------------------------------------------------------ fast path
// When every group is one run of consecutive items -- the keys met at piece
// boundaries strictly increase inside each (gpu, kind) segment, which holds
// when markers are numbered in the order they open -- rows are simply the
// pieces in item order: no owner tables, rows numbered by counting piece
// heads.  Each wavefront works alone on a tile of kWaveTile consecutive
// items (eight per lane); nothing is shared between the waves of a block.
// The fast path runs only without a record filter.
static_assert(kAggIpt == kTileIpt, "wave tiles hold eight items per lane");

// group key from the deepest non-NONE slot
__device__ inline uint32_t slot_key(uint32_t slot, int64_t M, uint32_t gk) {
  if (slot == kNone) return (uint32_t)((M + (gk >> 1)) * 2 + (gk & 1u));
  if ((int64_t)slot >= M) return kNone;
  return slot * 2u + (gk & 1u);
}

// Marker counts below which the natural-tile heads pass compares slots.
constexpr uint32_t kSlotFastM = 1u << 30;

// The same as selects: m2 = (uint32_t)(2 M) and mlim = min(M, 2^32 - 1)
// (so that slot >= mlim iff slot >= M for every slot below kNone).
struct SlotKeys {
  uint32_t m2, mlim;
  __device__ explicit SlotKeys(int64_t M)
      : m2((uint32_t)(2 * M)),
        mlim(M >= (int64_t)kNone ? kNone : (uint32_t)M) {}
  __device__ uint32_t operator()(uint32_t slot, uint32_t gk) const {
    const uint32_t kval = slot >= mlim ? kNone : slot * 2u + (gk & 1u);
    return slot == kNone ? m2 + gk : kval;
  }
};

// key of an item at level li (marker levels, then the GPU level)
template <int MaxD>
__device__ inline uint32_t level_key(const uint32_t (&p)[MaxD], uint32_t gk,
                                     int li, int D, int64_t M) {
  if (li >= D) return gk;
  uint32_t slot = kNone;
#pragma unroll
  for (int l = 0; l < MaxD; ++l)
    if (l <= li && p[l] != kNone) slot = p[l];
  return slot_key(slot, M, gk);
}

// One item's source index, gpu * 2 + kind and path (levels >= D are NONE),
// loaded without branches so that all loads of a tile are in flight at once.
template <int MaxD, typename Src>
__device__ inline void gather_item(const Src& src, int64_t i, int D,
                                   uint32_t& r, uint32_t& gk,
                                   uint32_t (&p)[MaxD]) {
  r = src.index(i);
  gk = src.gpuv(r) * 2u + src.kindv(r);
  if (D > 0) {        // uniform; without levels there is no path column
#pragma unroll
    for (int l = 0; l < MaxD; ++l) {
      const uint32_t v = src.pathv(r, l < D ? l : D - 1);
      p[l] = l < D ? v : kNone;
    }
  } else {
#pragma unroll
    for (int l = 0; l < MaxD; ++l) p[l] = kNone;
  }
}

// Per wave tile: number of piece heads at every level in [lv0, lv1] whose
// bit is set in `act` (tilecnt[(li - lv0) * nwt + tile]); flags[0] |= 1 when
// a key does not increase inside its segment, flags[1] |= 1 << kind for the
// kinds present; PATH_CONFLICT when two neighbours share a key but not the
// path.  Items are striped (item j * 64 + lane of the tile in lane `lane`);
// the previous item comes from the lane below by a DPP rotate.
template <int MaxD, typename Src>
__global__ __launch_bounds__(kBlock) void k_agg_heads(
    Src src, uint32_t act, int lv0, int lv1, int D, int64_t M, int64_t nwt,
    uint32_t* tilecnt, uint32_t* flags, uint32_t* status) {
  const int lane = lane_id();
  const int64_t w =
      (int64_t)blockIdx.x * kWavesPerBlock + (int64_t)(threadIdx.x / kWave);
  if (w >= nwt) return;
  // groups already known not to be runs: the counts are not used
  if (__builtin_amdgcn_readfirstlane((int)flag_read(&flags[0])) & 1) return;
  const int64_t cnt = src.count();
  const int64_t base = w * kWaveTile;
  if (base >= cnt) {
    if (lane <= lv1 - lv0) tilecnt[(int64_t)lane * nwt + w] = 0;
    return;
  }
  const int tile_n =
      (int)((cnt - base) < kWaveTile ? (cnt - base) : (int64_t)kWaveTile);
  uint32_t r[kAggIpt], gk[kAggIpt], p[kAggIpt][MaxD];
  uint32_t cr, cgk, cp[MaxD];      // the item before the tile
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) {
    const int q = j * kWave + lane;
    gather_item<MaxD>(src, base + (q < tile_n ? q : 0), D, r[j], gk[j], p[j]);
  }
  gather_item<MaxD>(src, base > 0 ? base - 1 : 0, D, cr, cgk, cp);
  (void)cr;
  bool cvalid = base > 0;          // lane 0's previous item exists
  uint64_t cpk = 0;                // 4-bit head counts per level, packed
  bool notinc = false, conflict = false;
  uint32_t kinds = 0;
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) {
    // previous item: lane below; lane 0 the last lane of the previous row
    uint32_t pp[MaxD], pgk;
#pragma unroll
    for (int l = 0; l < MaxD; ++l) {
      const uint32_t x = wave_ror1_u32(p[j][l]);
      pp[l] = lane == 0 ? cp[l] : x;
      cp[l] = x;
    }
    {
      const uint32_t x = wave_ror1_u32(gk[j]);
      pgk = lane == 0 ? cgk : x;
      cgk = x;
    }
    const bool pvalid = lane != 0 || cvalid;
    cvalid = true;
    const bool valid = j * kWave + lane < tile_n;
    uint32_t slot = kNone, pslot = kNone;
    bool eq = true;
#pragma unroll
    for (int li = 0; li < MaxD; ++li) {
      slot = p[j][li] != kNone ? p[j][li] : slot;
      pslot = pp[li] != kNone ? pp[li] : pslot;
      eq = eq && p[j][li] == pp[li];
      if (li >= D || li < lv0 || li > lv1 || !((act >> li) & 1u)) continue;
      const uint32_t key = slot_key(slot, M, gk[j]);
      const uint32_t pkey = pvalid ? slot_key(pslot, M, pgk) : kNone;
      if (valid && key == kNone) notinc = true;   // unkeyed item: general path
      if (key != pkey && key != kNone) {
        cpk += (valid ? 1ull : 0ull) << (4 * li);
        // inside a segment the no-marker group may only come first, so it
        // orders before every marker key in this test
        const int64_t ok = key >= 2 * M ? -1 : (int64_t)key;
        const int64_t opk = pkey >= 2 * M ? -1 : (int64_t)pkey;
        if (valid && pvalid && pgk == gk[j] && ok <= opk) notinc = true;
      } else if (valid && pvalid && key == pkey && key != kNone && !eq) {
        conflict = true;
      }
    }
    if (valid && D >= lv0 && D <= lv1 && ((act >> D) & 1u) &&
        (!pvalid || gk[j] != pgk)) {
      cpk += 1ull << (4 * D);
      kinds |= 1u << (gk[j] & 1u);
    }
  }
  // wave totals from bit planes of the per-lane counts (each at most 8)
  for (int li = lv0; li <= lv1; ++li) {
    const uint32_t c = (uint32_t)(cpk >> (4 * li)) & 15u;
    uint32_t tot = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b)
      tot += (uint32_t)__popcll(__ballot((c >> b) & 1u)) << b;
    if (lane == 0) tilecnt[(int64_t)(li - lv0) * nwt + w] = tot;
  }
  wave_flag_or(&flags[0], notinc, 1u);
  // a conflict sends the call to the general path, which groups by the
  // whole path
  if (__ballot(conflict) != 0 && lane == 0) {
    atomicOr(&flags[0], 2u);
    atomicOr(status, (uint32_t)CHOPPER_ST_PATH_CONFLICT);
  }
  // kinds present: the shared word is zeroed before the launch and only
  // gains bits, so a bit read as set here was set by this launch
  const uint32_t kk = (__ballot(kinds & 1u) != 0 ? 1u : 0u) |
                      (__ballot(kinds & 2u) != 0 ? 2u : 0u);
  if (lane == 0 && kk &&
      (__atomic_load_n(&flags[1], __ATOMIC_RELAXED) & kk) != kk)
    atomicOr(&flags[1], kk);
}

// Fast-path level offsets: the level-major scan gives every level but the
// workload level, whose rows are the kinds present.
// `stage` receives the three flags and the L + 1 offsets, so that the host
// reads them with one copy.
__global__ void k_agg_offsets_fast(int L, int64_t ntiles,
                                   const uint32_t* tilebase,
                                   const uint32_t* total, const uint32_t* flags,
                                   bool workload, int64_t cap,
                                   int64_t* level_offset, int64_t* stage,
                                   uint32_t* status) {
  if (threadIdx.x != 0) return;
  for (int li = 0; li < L; ++li) {
    const int64_t v = ntiles > 0 ? tilebase[(int64_t)li * ntiles] : 0;
    level_offset[li] = v;
    stage[3 + li] = v;
  }
  const int64_t tot =
      (int64_t)*total + (workload ? __popc(flags[1] & 3u) : 0);
  level_offset[L] = tot;
  stage[3 + L] = tot;
  for (int i = 0; i < 3; ++i) stage[i] = flags[i];
  // the counts are the row counts only when the fast path applies (and,
  // for the natural tiles, when the input order qualified)
  if (flags[0] == 0 && flags[2] == 0 && tot > cap)
    atomicOr(status, (uint32_t)CHOPPER_ST_ROWS_OVERFLOW);
}

// ------------------------------------------------------------ input order
// A profiler writes each GPU's records together and in start order.  For
// such input the (gpu, kind, start') order is the input order with every
// GPU's communication records moved after its compute records, so the fast
// path can read all columns in input order instead of through korder, where
// each sparse communication record would pull a whole cache line of every
// column.  A wave tile then covers consecutive input positions of one GPU
// and regroups its items by kind in LDS (compute first, order kept), which
// yields per (gpu, kind) exactly the item sequence of the korder tiles.
//
// Tiles: the natural tiles of kWaveTile positions, cut at GPU boundaries;
// GPU g owns tiles tb[g] .. tb[g + 1] - 1.  Head counts of a level are laid
// out as (gpu, kind, tile), so one exclusive scan numbers the rows in
// (gpu, kind, first record) order, as on the korder tiles.
struct NatGeom {
  const uint32_t* tb;   // [G + 1] first tile of every GPU; tb[G] = tiles
  const uint8_t* tg;    // [tiles] GPU of every tile
  const uint32_t* gs;   // [G] first input position of the GPU, kNone: none
  const uint32_t* ge;   // [G] one past its last position
  const int32_t* lp;    // [2][lps] last kind-k position before natural
                        // tile t, -1 if none
  const uint32_t* bad;  // nonzero: the input order does not qualify
  int64_t nnt;          // natural tiles
  int64_t lps;          // row stride of lp (nnt rounded up to kLpIpt)
  int G;
  // the fast-path flags, for a launch queued before the host has read them:
  // it does nothing unless flags[0] and flags[2] are both zero
  const uint32_t* fflags = nullptr;
};

struct NatTile {
  uint32_t g;
  int64_t base;
  int tile_n;
  int64_t prev[2];      // last kind-k position of the GPU before the tile
  uint32_t tbg, cg, tl; // GPU's first tile, its tile count, tile - tbg
};

// Geometry of tile tt; false past the last tile.
__device__ inline bool nat_tile(const NatGeom& N, int64_t tt, NatTile& T) {
  if (tt >= (int64_t)N.tb[N.G]) return false;
  const uint32_t g = N.tg[tt];
  const int64_t gs = N.gs[g], ge = N.ge[g];
  T.g = g;
  T.tbg = N.tb[g];
  T.cg = N.tb[g + 1] - T.tbg;
  T.tl = (uint32_t)(tt - T.tbg);
  const int64_t nt = gs / kWaveTile + T.tl;
  const int64_t a = nt * kWaveTile;
  T.base = a > gs ? a : gs;
  const int64_t e = a + kWaveTile < ge ? a + kWaveTile : ge;
  T.tile_n = (int)(e - T.base);
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    int64_t pv = -1;
    if (T.base > gs) {
      pv = N.lp[(int64_t)k * N.lps + nt];
      if (pv < gs) pv = -1;
    }
    T.prev[k] = pv;
  }
  return true;
}

// Kind regrouping of a tile: item q (striped) goes to LDS slot dst[j]
// (padded), compute items first; n0 = compute items.
__device__ inline void nat_regroup(const bool (&valid)[kAggIpt],
                                   const uint32_t (&kind)[kAggIpt], int lane,
                                   uint32_t (&dst)[kAggIpt], int* n0_out) {
  uint64_t m0[kAggIpt], m1[kAggIpt];
  uint32_t n0 = 0;
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) {
    m0[j] = __ballot(valid[j] && kind[j] == 0u);
    m1[j] = __ballot(valid[j] && kind[j] != 0u);
    n0 += (uint32_t)__popcll(m0[j]);
  }
  uint32_t c0 = 0, c1 = n0;
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) {
    uint32_t d = (uint32_t)(j * kWave + lane);
    if (valid[j]) d = kind[j] == 0u ? c0 + lanes_below(m0[j])
                                    : c1 + lanes_below(m1[j]);
    dst[j] = (uint32_t)pad8((int)d);
    c0 += (uint32_t)__popcll(m0[j]);
    c1 += (uint32_t)__popcll(m1[j]);
  }
  *n0_out = (int)n0;
}

template <typename T>
__device__ inline void wave_regroup_to_blocked(T* slice, T (&v)[kAggIpt],
                                               const uint32_t (&dst)[kAggIpt],
                                               int lane) {
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) slice[dst[j]] = v[j];
  wave_sync();
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) v[j] = slice[pad8(lane * kAggIpt + j)];
  wave_sync();
}

template <typename T>
__device__ inline void wave_blocked_to_regrouped(
    T* slice, T (&v)[kAggIpt], const uint32_t (&dst)[kAggIpt], int lane) {
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) slice[pad8(lane * kAggIpt + j)] = v[j];
  wave_sync();
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) v[j] = slice[dst[j]];
  wave_sync();
}

// Per natural tile: last position of each kind, the first position of every
// GPU, and whether the order qualifies (GPU ids never decrease, start'
// never decreases inside a GPU, every id below G).  Lane l reads positions
// 8l .. 8l + 7 of the tile, with vector loads when the columns allow.
__global__ __launch_bounds__(kBlock) void k_nat_pre(
    int64_t n, int G, const uint8_t* gpu, const uint8_t* cls,
    const int64_t* start, int64_t nnt, int64_t lps, int32_t* lpraw,
    uint32_t* gs, uint32_t* bad) {
  const int lane = lane_id();
  const int64_t nt =
      (int64_t)blockIdx.x * kWavesPerBlock + (int64_t)(threadIdx.x / kWave);
  if (nt >= nnt) return;
  // (the order is already known not to qualify: nothing here is used)
  if (__builtin_amdgcn_readfirstlane((int)flag_read(bad)) != 0) return;
  const int64_t base = nt * kWaveTile;
  const int64_t p0 = base + (int64_t)lane * kAggIpt;
  uint32_t g[kAggIpt], k[kAggIpt];
  int64_t s[kAggIpt];
  const bool vec = base + kWaveTile <= n && ((uintptr_t)gpu & 7) == 0 &&
                   ((uintptr_t)cls & 7) == 0 && ((uintptr_t)start & 15) == 0;
  if (vec) {
    const uint64_t gw = *(const uint64_t*)(gpu + p0);
    const uint64_t cw = *(const uint64_t*)(cls + p0);
#pragma unroll
    for (int j = 0; j < kAggIpt; j += 2) {
      const longlong2 v = *(const longlong2*)(start + p0 + j);
      s[j] = v.x;
      s[j + 1] = v.y;
    }
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) {
      g[j] = (uint32_t)(gw >> (8 * j)) & 0xFFu;
      k[j] = (uint32_t)kind_of((uint32_t)(cw >> (8 * j)) & 0xFFu);
    }
  } else {
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) {
      const int64_t p = p0 + j;
      g[j] = p < n ? (uint32_t)gpu[p] : 0u;
      k[j] = p < n ? (uint32_t)kind_of(cls[p]) : 0u;
      s[j] = p < n ? start[p] : 0;
    }
  }
  // the item before each lane's first: the lane below, or the tile's
  // predecessor for lane 0
  uint32_t pg = wave_shr1_u32(0u, g[kAggIpt - 1]);
  int64_t ps = dpp_any<kDppWaveShr1, 0xF>((int64_t)0, s[kAggIpt - 1]);
  if (lane == 0 && base > 0) {
    pg = gpu[base - 1];
    ps = start[base - 1];
  }
  bool wrong = false;
  int32_t last[2] = {-1, -1};
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) {
    const int64_t p = p0 + j;
    if (p < n) {
      if (g[j] >= (uint32_t)G) wrong = true;
      if (p > 0 && (g[j] < pg || (g[j] == pg && s[j] < ps))) wrong = true;
      if ((p == 0 || g[j] != pg) && g[j] < (uint32_t)G) gs[g[j]] = (uint32_t)p;
      last[k[j] ? 1 : 0] = (int32_t)p;
    }
    pg = g[j];
    ps = s[j];
  }
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const uint64_t m = __ballot(last[q] >= 0);
    const int32_t v =
        m ? __builtin_amdgcn_readlane(last[q], 63 - __clzll((long long)m))
          : -1;
    if (lane == 0) lpraw[(int64_t)q * lps + nt] = v;
  }
  wave_flag_or(bad, wrong, 1u);
}

// Block 0: GPU ranges, tile offsets and the GPU of every tile.  Blocks
// 1 ..: the exclusive running maximum of the last-position table over
// kLpSpan entries of each kind, each block taking the maximum of the entries
// before its span itself.
constexpr int kLpIpt = 4;                      // entries per thread and kind
constexpr int64_t kLpSpan = 1024 * kLpIpt;     // entries per block and kind
__global__ __launch_bounds__(1024) void k_nat_tiles(
    int64_t n, int G, int64_t nnt, int64_t lps, const int32_t* lpraw,
    int32_t* lp, const uint32_t* gs, uint32_t* ge, uint32_t* tb, uint8_t* tg,
    const uint32_t* bad) {
  if (*bad) return;
  __shared__ uint32_t s_c[256];
  __shared__ uint32_t s_tb[257];
  __shared__ int32_t s_w[2][1024 / kWave];
  __shared__ int32_t s_p[2][1024 / kWave];
  const int t = (int)threadIdx.x, lane = lane_id(), w = t / kWave;
  if (blockIdx.x == 0) {
    if (t < G) {
      const uint32_t a = gs[t];
      uint32_t e = (uint32_t)n;
      if (a != kNone) {
        for (int h = t + 1; h < G; ++h) {
          const uint32_t b = gs[h];
          if (b != kNone) {
            e = b;
            break;
          }
        }
      }
      ge[t] = a == kNone ? kNone : e;
      s_c[t] = a == kNone ? 0u
                          : (e - 1u) / (uint32_t)kWaveTile -
                                a / (uint32_t)kWaveTile + 1u;
    }
    __syncthreads();
    if (w == 0) {
      uint32_t carry = 0;
      for (int b0 = 0; b0 < G; b0 += kWave) {
        const uint32_t v = b0 + lane < G ? s_c[b0 + lane] : 0u;
        const uint32_t incl = wave_incl(v, OpAdd(), 0u);
        if (b0 + lane < G) {
          tb[b0 + lane] = carry + incl - v;
          s_tb[b0 + lane] = carry + incl - v;
        }
        carry += (uint32_t)__builtin_amdgcn_readlane((int)incl, kWave - 1);
      }
      if (lane == 0) {
        tb[G] = carry;
        s_tb[G] = carry;
      }
    }
    __syncthreads();
    for (int g = 0; g < G; ++g)
      for (uint32_t i = s_tb[g] + (uint32_t)t; i < s_tb[g + 1]; i += 1024)
        tg[i] = (uint8_t)g;
    return;
  }
  OpMax op;
  const int64_t b0 = (int64_t)(blockIdx.x - 1) * kLpSpan;
  const int64_t i0 = b0 + (int64_t)t * kLpIpt;
  int32_t pre[2] = {-1, -1}, v[2][kLpIpt], acc[2] = {-1, -1};
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const int32_t* row = lpraw + (int64_t)q * lps;
    for (int64_t i = (int64_t)t * kLpIpt; i < b0; i += kLpSpan) {
      const int4 x = *(const int4*)(row + i);
      pre[q] = op(pre[q], op(op(x.x, x.y), op(x.z, x.w)));
    }
    int4 x = make_int4(-1, -1, -1, -1);
    if (i0 < nnt) x = *(const int4*)(row + i0);
    v[q][0] = x.x;
    v[q][1] = i0 + 1 < nnt ? x.y : -1;
    v[q][2] = i0 + 2 < nnt ? x.z : -1;
    v[q][3] = i0 + 3 < nnt ? x.w : -1;
#pragma unroll
    for (int j = 0; j < kLpIpt; ++j) acc[q] = op(acc[q], v[q][j]);
  }
  int32_t incl[2];
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    incl[q] = wave_incl(acc[q], op, (int32_t)-1);
    const int32_t pw = lane63(wave_incl(pre[q], op, (int32_t)-1));
    if (lane == kWave - 1) {
      s_w[q][w] = incl[q];
      s_p[q][w] = pw;
    }
  }
  __syncthreads();
  if (i0 >= nnt) return;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    int32_t p = -1;
    for (int r = 0; r < 1024 / kWave; ++r) {
      p = op(p, s_p[q][r]);
      if (r < w) p = op(p, s_w[q][r]);
    }
    p = op(p, wave_shr1_any((int32_t)-1, incl[q]));
    int4 x;
    x.x = p;
    p = op(p, v[q][0]);
    x.y = p;
    p = op(p, v[q][1]);
    x.z = p;
    p = op(p, v[q][2]);
    x.w = p;
    *(int4*)(lp + (int64_t)q * lps + i0) = x;
  }
}

// Item of the natural tiles: gpu * 2 + kind and path of input position i.
template <int MaxD>
__device__ inline void nat_item(const RecSrc& S, int64_t i, uint32_t g, int D,
                                uint32_t& gk, uint32_t (&p)[MaxD]) {
  gk = g * 2u + (uint32_t)kind_of(S.cls[i]);
#pragma unroll
  for (int l = 0; l < MaxD; ++l) {
    const int ll = l < D ? l : (D > 0 ? D - 1 : 0);
    const uint32_t v = D > 0 ? S.idx[(int64_t)ll * S.n + i] : kNone;
    p[l] = l < D ? v : kNone;
  }
}

// Heads pass over the natural tiles: per level and kind the groups that
// start in the tile, at tilecnt[(li - lv0) * stride + 2 * tbg + k * cg + tl];
// entries past the last tile are zeroed.  Flags as in k_agg_heads.
template <int MaxD>
__global__ __launch_bounds__(kBlock) void k_agg_heads_nat(
    RecSrc S, NatGeom N, uint32_t act, int lv0, int lv1, int D, int64_t M,
    int64_t stride, uint32_t* tilecnt, uint32_t* flags, uint32_t* status) {
  __shared__ uint32_t s_k[kWavesPerBlock][kSlice];
  if (*N.bad) return;
  const int lane = lane_id();
  const int wv = (int)(threadIdx.x / kWave);
  const int64_t tt = (int64_t)blockIdx.x * kWavesPerBlock + wv;
  if (tt >= N.nnt + N.G) return;
  if (__builtin_amdgcn_readfirstlane((int)flag_read(&flags[0])) & 1) return;
  NatTile T;
  if (!nat_tile(N, tt, T)) {
    if (lane <= lv1 - lv0) {
      tilecnt[(int64_t)lane * stride + 2 * tt] = 0;
      tilecnt[(int64_t)lane * stride + 2 * tt + 1] = 0;
    }
    return;
  }
  uint32_t* sk = s_k[wv];
  uint32_t gk[kAggIpt], p[kAggIpt][MaxD], kind[kAggIpt], dst[kAggIpt];
  bool valid[kAggIpt];
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) {
    const int q = j * kWave + lane;
    valid[j] = q < T.tile_n;
    nat_item<MaxD>(S, T.base + (valid[j] ? q : 0), T.g, D, gk[j], p[j]);
    kind[j] = gk[j] & 1u;
  }
  int n0;
  nat_regroup(valid, kind, lane, dst, &n0);
  wave_regroup_to_blocked(sk, gk, dst, lane);
#pragma unroll
  for (int l = 0; l < MaxD; ++l) {
    uint32_t x[kAggIpt];
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) x[j] = p[j][l];
    wave_regroup_to_blocked(sk, x, dst, lane);
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) p[j][l] = x[j];
  }
  // the items before the tile, one per kind (same GPU)
  uint32_t qgk[2], qp[2][MaxD];
  bool qv[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    qv[k] = T.prev[k] >= 0;
    nat_item<MaxD>(S, qv[k] ? T.prev[k] : T.base, T.g, D, qgk[k], qp[k]);
  }
  // 4-bit head counts per level (the GPU level D included), per kind
  using Cnt = typename std::conditional<(MaxD + 1) * 4 <= 32, uint32_t,
                                        uint64_t>::type;
  // Every item of a run of the tile, and the item before the run, has the
  // tile's GPU and the run's kind, so the keys of two consecutive items
  // compare as their slots: equal iff the slots are, ordered as slot + 1
  // modulo 2^32 (which puts items with no marker first, as their keys are),
  // a slot at or above M giving no key.  That holds while keys of distinct
  // slots differ, M < 2^30; beyond, the call takes the general path.
  const uint32_t mlim = (uint32_t)(M < (int64_t)kSlotFastM ? M : 0);
  Cnt cpk[2] = {0, 0};
  bool notinc = M >= (int64_t)kSlotFastM, conflict = false;
  uint32_t kinds = 0;
  // previous item in the regrouped order: lane below for j == 0
  uint32_t cp[MaxD];
#pragma unroll
  for (int l = 0; l < MaxD; ++l) cp[l] = wave_shr1_u32(0u, p[kAggIpt - 1][l]);
  // (selects rather than branches: the conditions differ between lanes)
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) {
    const int v = lane * kAggIpt + j;
    const bool vv = v < T.tile_n;
    const bool comm = v >= n0;
    // the first item of a kind takes the item before the tile of its kind
    const bool first = v == n0 || v == 0;
    const bool fk = v == n0;
    const bool pvalid = first ? (fk ? qv[1] : qv[0]) : true;
    uint32_t pp[MaxD];
#pragma unroll
    for (int l = 0; l < MaxD; ++l)
      pp[l] = first ? (fk ? qp[1][l] : qp[0][l]) : cp[l];
#pragma unroll
    for (int l = 0; l < MaxD; ++l) cp[l] = p[j][l];
    Cnt inc = 0;
    uint32_t slot = kNone, pslot = kNone;
    bool eq = true;
#pragma unroll
    for (int li = 0; li < MaxD; ++li) {
      slot = p[j][li] != kNone ? p[j][li] : slot;
      pslot = pp[li] != kNone ? pp[li] : pslot;
      eq = eq & (p[j][li] == pp[li]);
      if (li >= D || li < lv0 || li > lv1 || !((act >> li) & 1u)) continue;
      const uint32_t s1 = slot + 1u, ps1 = pslot + 1u;
      const bool bad = s1 > mlim;        // no key
      const bool same = slot == pslot;
      const bool head = !bad & (!pvalid | !same);
      notinc = notinc | (vv & bad);
      inc += (vv & head) ? (Cnt)1 << (4 * li) : (Cnt)0;
      notinc = notinc | (vv & head & pvalid & (s1 <= ps1));
      // equal keys over different paths: the groups are not the runs
      conflict = conflict | (vv & pvalid & !bad & same & !eq);
    }
    if (D >= lv0 && D <= lv1 && ((act >> D) & 1u)) {
      const bool g = vv & !pvalid;
      inc += g ? (Cnt)1 << (4 * D) : (Cnt)0;
      kinds |= g ? (comm ? 2u : 1u) : 0u;
    }
    cpk[0] += comm ? (Cnt)0 : inc;
    cpk[1] += comm ? inc : (Cnt)0;
  }
  for (int li = lv0; li <= lv1; ++li) {
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const uint32_t c = (uint32_t)(cpk[k] >> (4 * li)) & 15u;
      uint32_t tot = 0;
#pragma unroll
      for (int b = 0; b < 4; ++b)
        tot += (uint32_t)__popcll(__ballot((c >> b) & 1u)) << b;
      if (lane == 0)
        tilecnt[(int64_t)(li - lv0) * stride + 2 * (int64_t)T.tbg +
                (int64_t)k * T.cg + T.tl] = tot;
    }
  }
  wave_flag_or(&flags[0], notinc, 1u);
  // a conflict sends the call to the general path, which groups by the
  // whole path
  if (__ballot(conflict) != 0 && lane == 0) {
    atomicOr(&flags[0], 2u);
    atomicOr(status, (uint32_t)CHOPPER_ST_PATH_CONFLICT);
  }
  const uint32_t kk = (__ballot(kinds & 1u) != 0 ? 1u : 0u) |
                      (__ballot(kinds & 2u) != 0 ? 2u : 0u);
  if (lane == 0 && kk &&
      (__atomic_load_n(&flags[1], __ATOMIC_RELAXED) & kk) != kk)
    atomicOr(&flags[1], kk);
}

// Piece structure of one level over a wave tile (blocked arrangement: lane
// holds items lane * 8 + j).  Pieces are maximal runs of equal keys.  Items
// [0, n0) and [n0, tile_n) are two separate runs of rows (the two kinds of
// a natural tile; n0 = tile_n on korder tiles): rows r0 + i for the pieces
// of the first, r1 + i for the second.  The first piece of each may continue
// a row of an earlier tile (c0, c1).
struct LevelTile {
  uint32_t m_head;    // item starts a piece (tile start and invalid items too)
  uint32_t m_hv;      // ... and is valid
  uint32_t m_last;    // valid item ends a piece
  uint32_t m_real;    // valid item starts a group (key differs from previous)
  uint32_t pfx;       // pieces started in the lanes below
  uint32_t NP;        // pieces in the tile
  uint32_t NP0;       // pieces of the first run
  uint32_t c0, c1;    // the run's first piece continues an earlier row
  int64_t r0, r1;     // row of the run's first new group
  uint32_t before;    // items of the lane before its first piece head
  WaveSegMasks masks; // lane segment flags for wave scans
};

// slot[j]: LDS slot of item j's value -- its piece index when it ends a
// piece, else a junk slot of its own lane.  prev0 / prev1: keys of the items
// before each run (kNone: none).
__device__ inline void level_tile(const uint32_t (&key)[kAggIpt],
                                  uint32_t prev0, uint32_t prev1, int n0,
                                  int tile_n, int lane, int64_t r0, int64_t r1,
                                  LevelTile& T, uint32_t (&slot)[kAggIpt]) {
  uint32_t m_valid = 0, m_real = 0, m_head = 0;
  uint32_t prev = wave_shr1_u32(prev0, key[kAggIpt - 1]);
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) {
    const int q = lane * kAggIpt + j;
    const bool valid = q < tile_n;
    const uint32_t k = key[j];
    if (q == n0) prev = prev1;
    if (valid) m_valid |= 1u << j;
    if (valid && k != prev) m_real |= 1u << j;
    if (!valid || q == 0 || q == n0 || k != prev) m_head |= 1u << j;
    prev = k;
  }
  const uint64_t h0 = __ballot(m_head & 1u);
  const uint32_t next0 =
      lane == kWave - 1 ? 1u : (uint32_t)((h0 >> (lane + 1)) & 1u);
  T.m_head = m_head;
  T.m_hv = m_head & m_valid;
  T.m_real = m_real;
  T.m_last = m_valid & ((m_head >> 1) | (next0 << (kAggIpt - 1)));
  const uint32_t hc = (uint32_t)__popc(T.m_hv);
  T.pfx = wave_prefix_small<4>(hc);
  T.NP = (uint32_t)__builtin_amdgcn_readlane((int)(T.pfx + hc), kWave - 1);
  if (n0 >= tile_n) {
    T.NP0 = T.NP;
    T.c1 = 0;
  } else {
    // pieces that start below position n0, and whether the item there is
    // a new group
    const int ln = n0 / kAggIpt, jn = n0 % kAggIpt;
    const uint32_t below =
        T.pfx + (uint32_t)__popc(T.m_hv & ((1u << jn) - 1u));
    T.NP0 = (uint32_t)__builtin_amdgcn_readlane((int)below, ln);
    const uint32_t real_n =
        (uint32_t)__builtin_amdgcn_readlane((int)((m_real >> jn) & 1u), ln);
    T.c1 = real_n ? 0u : 1u;
  }
  T.c0 = n0 > 0 && __ballot(lane == 0 && !(m_real & 1u)) != 0 ? 1u : 0u;
  T.r0 = r0;
  T.r1 = r1;
  T.before = m_head ? (uint32_t)(__ffs(m_head) - 1) : (uint32_t)kAggIpt;
  T.masks = wave_seg_masks(m_head != 0);
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) {
    const uint32_t idx =
        T.pfx + (uint32_t)__popc(T.m_hv & ((2u << j) - 1u)) - 1u;
    slot[j] = ((T.m_last >> j) & 1u) ? idx : (uint32_t)(kWaveTile + lane);
  }
}

// Row of piece q, or -1 when it continues a row of an earlier tile.
__device__ inline int64_t piece_row(const LevelTile& T, uint32_t q) {
  const bool second = q >= T.NP0;
  const uint32_t qi = second ? q - T.NP0 : q;
  const uint32_t cc = second ? T.c1 : T.c0;
  if (qi < cc) return -1;
  return (second ? T.r1 : T.r0) + (int64_t)(qi - cc);
}

// Reduction of one level -- with kTwo also the next coarser one -- when
// groups are runs.  Within a wave tile, rows are numbered from the tile's
// head count (level-major exclusive scan of the heads pass).  Every field
// goes striped -> blocked through the wave's LDS slice; sums take one plain
// prefix sum over the tile and a piece's total is the difference of the
// prefix at its last item and at the previous piece's last item (exact
// modulo 2^64), for both levels from the same prefix; tmin and tmax take a
// segmented scan per level.  Piece values are written to LDS at the piece's
// index, so that the stores of consecutive lanes go to consecutive rows.  A
// run's first piece may continue a row of an earlier tile: it goes to the
// tile's overflow slot of its level (korder tiles: slot w of level li,
// nwt + w of level li - 1; natural tiles: 2w + kind and 2nwt + 2w + kind).
// Every valid item has a key here (the heads pass sends traces with unkeyed
// items to the general path).  kNat: the natural tiles, items read in input
// order and regrouped by kind on the way to the blocked arrangement.
template <int MaxD, typename Src, bool kTwo, bool kNat>
__global__ __launch_bounds__(kBlock) void k_agg_fast_reduce(
    Src src, NatGeom N, int li, int D, int64_t M, const uint32_t* tilebase,
    const uint32_t* tilebase2, const int64_t* row0, RowsDev R, Overflow ovf,
    int64_t nwt) {
  __shared__ uint64_t s_v[kWavesPerBlock][kSlice];
  const int lane = lane_id();
  const int wv = (int)(threadIdx.x / kWave);
  const int64_t w = (int64_t)blockIdx.x * kWavesPerBlock + wv;
  if (w >= nwt) return;
  if constexpr (kNat) {
    if (N.fflags && __builtin_amdgcn_readfirstlane(
                        (int)(N.fflags[0] | N.fflags[2])) != 0)
      return;
  }
  int64_t base;
  int tile_n;
  NatTile NT;
  if constexpr (kNat) {
    if (!nat_tile(N, w, NT)) {
      if (lane < 2) {
        ovf.row[2 * w + lane] = kNone;
        if (kTwo) ovf.row[2 * nwt + 2 * w + lane] = kNone;
      }
      return;
    }
    base = NT.base;
    tile_n = NT.tile_n;
  } else {
    const int64_t cnt = src.count();
    base = w * kWaveTile;
    if (base >= cnt) {
      if (lane == 0) {
        ovf.row[w] = kNone;
        if (kTwo) ovf.row[nwt + w] = kNone;
      }
      return;
    }
    tile_n =
        (int)((cnt - base) < kWaveTile ? (cnt - base) : (int64_t)kWaveTile);
  }
  const int li2 = li - 1;
  uint64_t* sv = s_v[wv];
  uint32_t* sk = (uint32_t*)sv;
  // striped items: source index, gpu * 2 + kind, path, keys
  uint32_t rs[kAggIpt], gk[kAggIpt], p[kAggIpt][MaxD];
  uint32_t key[kAggIpt], key2[kAggIpt], dst[kAggIpt];
  uint32_t tprev[2] = {kNone, kNone}, tprev2[2] = {kNone, kNone};
  int n0 = tile_n;
  int64_t r0 = 0, r1 = 0, q0 = 0, q1 = 0;
  if constexpr (kNat) {
    bool valid[kAggIpt];
    uint32_t kind[kAggIpt];
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) {
      const int q = j * kWave + lane;
      valid[j] = q < tile_n;
      rs[j] = (uint32_t)(base + (valid[j] ? q : 0));
      nat_item<MaxD>(src.S, rs[j], NT.g, D, gk[j], p[j]);
      kind[j] = gk[j] & 1u;
    }
    nat_regroup(valid, kind, lane, dst, &n0);
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      if (NT.prev[k] < 0) continue;
      uint32_t cgk, cp[MaxD];
      nat_item<MaxD>(src.S, NT.prev[k], NT.g, D, cgk, cp);
      tprev[k] = level_key<MaxD>(cp, cgk, li, D, M);
      if (kTwo) tprev2[k] = level_key<MaxD>(cp, cgk, li2, D, M);
    }
    const int64_t e0 = 2 * (int64_t)NT.tbg + NT.tl;
    const int64_t e1 = e0 + NT.cg;
    r0 = tilebase[e0];
    r1 = tilebase[e1];
    if (kTwo) {
      q0 = tilebase2[e0];
      q1 = tilebase2[e1];
    }
  } else {
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) {
      const int q = j * kWave + lane;
      gather_item<MaxD>(src, base + (q < tile_n ? q : 0), D, rs[j], gk[j],
                        p[j]);
      dst[j] = 0;
    }
    uint32_t cr, cgk, cp[MaxD];
    gather_item<MaxD>(src, base > 0 ? base - 1 : 0, D, cr, cgk, cp);
    tprev[0] = base > 0 ? level_key<MaxD>(cp, cgk, li, D, M) : kNone;
    if (kTwo)
      tprev2[0] = base > 0 ? level_key<MaxD>(cp, cgk, li2, D, M) : kNone;
    // rows: the level offset (row0, when the scan covers this level only)
    // plus the scanned head count; row0[-1] is the second level's offset
    r0 = (row0 ? row0[0] - (int64_t)tilebase[0] : 0) + (int64_t)tilebase[w];
    if (kTwo)
      q0 = (row0 ? row0[-1] - (int64_t)tilebase2[0] : 0) +
           (int64_t)tilebase2[w];
  }
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) {
    const int q = j * kWave + lane;
    key[j] = q < tile_n ? level_key<MaxD>(p[j], gk[j], li, D, M) : kNone;
    key2[j] = kTwo && q < tile_n ? level_key<MaxD>(p[j], gk[j], li2, D, M)
                                 : kNone;
  }
  auto blk32 = [&](uint32_t (&x)[kAggIpt]) {
    if constexpr (kNat) wave_regroup_to_blocked(sk, x, dst, lane);
    else wave_to_blocked(sk, x, lane);
  };
  auto blk64 = [&](uint64_t (&x)[kAggIpt]) {
    if constexpr (kNat) wave_regroup_to_blocked(sv, x, dst, lane);
    else wave_to_blocked(sv, x, lane);
  };
  blk32(key);
  if (kTwo) blk32(key2);
  LevelTile T1, T2;
  uint32_t slot[kAggIpt], slot2[kAggIpt];
  level_tile(key, tprev[0], tprev[1], n0, tile_n, lane, r0, r1, T1, slot);
  if (kTwo)
    level_tile(key2, tprev2[0], tprev2[1], n0, tile_n, lane, q0, q1, T2,
               slot2);

  // headers of the rows that start here, written from the striped items:
  // the row of every group head goes back through LDS
  auto headers = [&](const LevelTile& T, int lv) {
    uint32_t rw[kAggIpt];
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) {
      const uint32_t idx =
          T.pfx + (uint32_t)__popc(T.m_hv & ((2u << j) - 1u)) - 1u;
      const int64_t row = piece_row(T, idx);
      rw[j] = ((T.m_real >> j) & 1u) && row >= 0 && row < R.cap
                  ? (uint32_t)row : kNone;
    }
    if constexpr (kNat) wave_blocked_to_regrouped(sk, rw, dst, lane);
    else wave_to_striped(sk, rw, lane);
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) {
      const uint32_t wr = rw[j];
      if (wr == kNone) continue;
#pragma unroll
      for (int l = 0; l < MaxD; ++l)
        if (l < D)
          R.path[(int64_t)l * R.cap + wr] =
              (lv < D && l <= lv) ? p[j][l] : kNone;
      R.gpu[wr] = (uint8_t)(gk[j] >> 1);
      R.kind[wr] = (uint8_t)(gk[j] & 1u);
      R.first[wr] = src.first_of(rs[j]);
    }
  };
  headers(T1, li);
  if (kTwo) headers(T2, li2);
  auto cont_row = [&](uint32_t c, int64_t r) -> uint32_t {
    return c && r >= 1 && r - 1 < R.cap ? (uint32_t)(r - 1) : kNone;
  };
  if (lane == 0) {
    if constexpr (kNat) {
      ovf.row[2 * w] = cont_row(T1.c0, T1.r0);
      ovf.row[2 * w + 1] = cont_row(T1.c1, T1.r1);
      if (kTwo) {
        ovf.row[2 * nwt + 2 * w] = cont_row(T2.c0, T2.r0);
        ovf.row[2 * nwt + 2 * w + 1] = cont_row(T2.c1, T2.r1);
      }
    } else {
      ovf.row[w] = cont_row(T1.c0, T1.r0);
      if (kTwo) ovf.row[nwt + w] = cont_row(T2.c0, T2.r0);
    }
  }
  // byte offsets of the striped items (sizes are below 2^29 here)
  uint32_t off[kAggIpt];
#pragma unroll
  for (int j = 0; j < kAggIpt; ++j) off[j] = rs[j] << 3;

  // piece values at the slots -> rows (and the overflow slots)
  auto store_pieces = [&](const LevelTile& T, int64_t obase, int f,
                          bool diff) {
    uint64_t* col = row_column(R, f);
    uint64_t* oslot = ovf.val + (int64_t)f * ovf.cap + obase +
                      (kNat ? 2 * w : w);
    wave_sync();
    for (uint32_t q = lane; q < T.NP; q += kWave) {
      uint64_t v = sv[q];
      if (diff && q > 0) v -= sv[q - 1];
      const int64_t row = piece_row(T, q);
      if (row < 0) {
        oslot[q >= T.NP0 ? 1 : 0] = v;
      } else if (row < R.cap) {
        col[row] = v;
      }
    }
    wave_sync();
  };
  auto put = [&](const uint32_t (&sl)[kAggIpt], const uint64_t (&x)[kAggIpt]) {
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) sv[sl[j]] = x[j];
  };
  const int64_t ob2 = kNat ? 2 * nwt : nwt;
  auto do_sum = [&](const uint64_t (&v)[kAggIpt], int f) {
    uint64_t x[kAggIpt];
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) x[j] = v[j];
    blk64(x);
#pragma unroll
    for (int j = 1; j < kAggIpt; ++j) x[j] += x[j - 1];
    const uint64_t incl = wave_incl(x[kAggIpt - 1], OpAdd(), (uint64_t)0);
    const uint64_t carry = wave_shr1(0ull, incl);
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) x[j] += carry;
    put(slot, x);
    store_pieces(T1, 0, f, true);
    if (kTwo) {
      put(slot2, x);
      store_pieces(T2, ob2, f, true);
    }
  };
  auto seg_pass = [&](const LevelTile& T, const uint32_t (&sl)[kAggIpt],
                      const uint64_t (&xin)[kAggIpt], int64_t obase, int f,
                      auto cmb) {
    using C = decltype(cmb);
    uint64_t x[kAggIpt];
    uint64_t acc = xin[0];
    x[0] = acc;
#pragma unroll
    for (int j = 1; j < kAggIpt; ++j) {
      acc = ((T.m_head >> j) & 1u) ? xin[j] : cmb(acc, xin[j]);
      x[j] = acc;
    }
    const uint64_t incl = wave_seg_incl<C>(T.masks, acc);
    const uint64_t carry = wave_shr1(C::ident, incl);
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j)
      sv[sl[j]] = (uint32_t)j < T.before ? cmb(carry, x[j]) : x[j];
    store_pieces(T, obase, f, false);
  };
  auto do_seg = [&](const uint64_t (&v)[kAggIpt], int f, auto cmb) {
    uint64_t x[kAggIpt];
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j) x[j] = v[j];
    blk64(x);
    seg_pass(T1, slot, x, 0, f, cmb);
    if (kTwo) seg_pass(T2, slot2, x, ob2, f, cmb);
  };
  auto load = [&](const uint64_t* col, uint64_t (&v)[kAggIpt]) {
#pragma unroll
    for (int j = 0; j < kAggIpt; ++j)
      v[j] = *(const uint64_t*)((const char*)col + off[j]);
  };

  const int ns = src.nsum();
  // three plain-sum columns in flight: each is loaded three fields ahead of
  // its use (the first ones staggered between the special fields)
  uint64_t va[kAggIpt], vb[kAggIpt], vc[kAggIpt];
  {
    uint64_t ts[kAggIpt], te[kAggIpt];
    load((const uint64_t*)src.start_col(), ts);
    load((const uint64_t*)src.end_col(), te);
    if (ns > 0) load(src.sum_col(0), va);
    if constexpr (Src::kRecords) {
      // n: the prefix of ones at a piece's last item is its position + 1
      uint64_t pos[kAggIpt];
#pragma unroll
      for (int j = 0; j < kAggIpt; ++j)
        pos[j] = (uint64_t)(lane * kAggIpt + j + 1);
      put(slot, pos);
      store_pieces(T1, 0, 0, true);
      if (kTwo) {
        put(slot2, pos);
        store_pieces(T2, ob2, 0, true);
      }
      uint64_t du[kAggIpt];
#pragma unroll
      for (int j = 0; j < kAggIpt; ++j) du[j] = te[j] - ts[j];
      if (ns > 1) load(src.sum_col(1), vb);
      do_sum(du, 1);
    } else {
      if (ns > 1) load(src.sum_col(1), vb);
    }
    do_seg(ts, 4, CMin());
    if (ns > 2) load(src.sum_col(2), vc);
    do_seg(te, 5, CMax());
  }
  for (int i = 0; i < ns; i += 3) {
    do_sum(va, src.sum_dst(i));
    if (i + 3 < ns) load(src.sum_col(i + 3), va);
    if (i + 1 < ns) {
      do_sum(vb, src.sum_dst(i + 1));
      if (i + 4 < ns) load(src.sum_col(i + 4), vb);
    }
    if (i + 2 < ns) {
      do_sum(vc, src.sum_dst(i + 2));
      if (i + 5 < ns) load(src.sum_col(i + 5), vc);
    }
  }
}

// GPU rows from the level-0 rows (with no marker level, the GPU rows
// themselves): the level-0 rows of one (gpu, kind) are consecutive and
// ordered by (tmin, first), and every record is in exactly one of them.
// Block b sums the rows of the pair gpu * 2 + kind = b into slot b of
// `pair` (fields, then tmin, first and a presence flag); a single block
// then numbers the pairs present, writes the GPU rows and adds them up into
// the workload rows (one per kind present, kind 0 first).
constexpr int kPairW = kMaxFields + 3;

// First row in [a0, a1) whose pair is >= k, for every thread of the block:
// a search with kBlock probes per round.
__device__ inline int64_t block_pair_lower(const RowsDev& R, int64_t a0,
                                           int64_t a1, uint32_t k,
                                           uint32_t* s_cnt) {
  int64_t lo = a0, hi = a1;           // answer in [lo, hi]
  while (hi > lo) {
    const int64_t step = (hi - lo + kBlock - 1) / kBlock;
    const int64_t p = lo + (int64_t)threadIdx.x * step;
    const bool below =
        p < hi && (uint32_t)R.gpu[p] * 2u + R.kind[p] < k;
    const uint64_t m = __ballot(below);
    __syncthreads();
    if (lane_id() == 0) s_cnt[threadIdx.x / kWave] = (uint32_t)__popcll(m);
    __syncthreads();
    uint32_t c = 0;
    for (int i = 0; i < kWavesPerBlock; ++i) c += s_cnt[i];
    // probes 0 .. c - 1 are below k (rows are sorted by pair)
    if (c == 0) return lo;
    const int64_t nlo = lo + (int64_t)(c - 1) * step + 1;
    const int64_t nhi = lo + (int64_t)c * step;
    lo = nlo;
    hi = nhi < hi ? nhi : hi;
  }
  return lo;
}

__global__ __launch_bounds__(kBlock) void k_agg_gpu_sums(
    const int64_t* level_offset, RowsDev R, int nfields, uint64_t* pair) {
  __shared__ uint32_t s_cnt[kWavesPerBlock];
  __shared__ uint64_t s_f[kWavesPerBlock][kMaxFields];
  const uint32_t b = blockIdx.x;
  uint64_t* slot = pair + (int64_t)b * kPairW;
  int64_t a0 = level_offset[0], a1 = level_offset[1];
  if (a1 > R.cap) a1 = R.cap;
  if (a0 > a1) a0 = a1;
  const int64_t lo = block_pair_lower(R, a0, a1, b, s_cnt);
  const int64_t hi = block_pair_lower(R, lo, a1, b + 1, s_cnt);
  if (lo >= hi) {
    if (threadIdx.x == 0) slot[kMaxFields + 2] = 0;
    return;
  }
  uint64_t acc[kMaxFields];
#pragma unroll
  for (int f = 0; f < kMaxFields; ++f)
    acc[f] = f == 5 ? (uint64_t)kI64Min : 0ull;
  for (int64_t r = lo + threadIdx.x; r < hi; r += kBlock) {
#pragma unroll
    for (int f = 0; f < kMaxFields; ++f) {
      if (f == 4 || f >= nfields) continue;
      const uint64_t x = row_column(R, f)[r];
      acc[f] = f == 5 ? ((int64_t)x > (int64_t)acc[f] ? x : acc[f])
                      : acc[f] + x;
    }
  }
#pragma unroll
  for (int f = 0; f < kMaxFields; ++f) {
    uint64_t v = acc[f];
    for (int d = kWave / 2; d > 0; d >>= 1) {
      const uint64_t o = __shfl_xor(v, d, kWave);
      v = f == 5 ? ((int64_t)o > (int64_t)v ? o : v) : v + o;
    }
    if (lane_id() == 0) s_f[threadIdx.x / kWave][f] = v;
  }
  __syncthreads();
  const int f = (int)threadIdx.x;
  if (f < nfields && f != 4) {
    uint64_t t = s_f[0][f];
    for (int i = 1; i < kWavesPerBlock; ++i)
      t = f == 5 ? ((int64_t)s_f[i][f] > (int64_t)t ? s_f[i][f] : t)
                 : t + s_f[i][f];
    slot[f] = t;
  }
  if (f == 0) {
    // the pair's first row has the smallest (tmin, first)
    slot[4] = (uint64_t)R.tmin[lo];
    slot[kMaxFields] = (uint64_t)R.tmin[lo];
    slot[kMaxFields + 1] = R.first[lo];
    slot[kMaxFields + 2] = 1;
  }
}

__global__ __launch_bounds__(1024) void k_agg_gpu_finish(
    const int64_t* level_offset, int D, RowsDev R, int nfields, int npairs,
    const uint64_t* pair) {
  __shared__ uint32_t s_rank[513];
  const int t = (int)threadIdx.x;
  if (t == 0) {
    uint32_t c = 0;
    for (int q = 0; q < npairs; ++q) {
      s_rank[q] = c;
      c += (uint32_t)pair[(int64_t)q * kPairW + kMaxFields + 2];
    }
    s_rank[npairs] = c;
  }
  __syncthreads();
  const int64_t g0 = level_offset[D];
  // GPU rows: one thread per (pair, field) of the pairs present
  for (int i = t; i < npairs * kPairW; i += 1024) {
    const int q = i / kPairW, f = i % kPairW;
    const uint64_t* slot = pair + (int64_t)q * kPairW;
    if (!slot[kMaxFields + 2]) continue;
    const int64_t row = g0 + s_rank[q];
    if (row >= R.cap) continue;
    if (f < nfields) {
      row_column(R, f)[row] = slot[f];
    } else if (f == kMaxFields) {
      R.first[row] = (uint32_t)slot[kMaxFields + 1];
      R.gpu[row] = (uint8_t)(q >> 1);
      R.kind[row] = (uint8_t)(q & 1);
      for (int l = 0; l < D; ++l) R.path[(int64_t)l * R.cap + row] = kNone;
    }
  }
  // workload rows: kind 0 first when present
  const int64_t w0 = level_offset[D + 1], w1 = level_offset[D + 2];
  for (int i = t; i < 2 * kPairW; i += 1024) {
    const uint32_t kd = (uint32_t)(i / kPairW);
    const int f = i % kPairW;
    bool any = false;
    uint64_t acc = f == 5 ? (uint64_t)kI64Min : 0ull;
    int64_t bt = kI64Max;
    uint32_t bf = kNone;
    for (int q = (int)kd; q < npairs; q += 2) {
      const uint64_t* slot = pair + (int64_t)q * kPairW;
      if (!slot[kMaxFields + 2]) continue;
      any = true;
      const uint64_t x = slot[f < kMaxFields ? f : 0];
      acc = f == 5 ? ((int64_t)x > (int64_t)acc ? x : acc) : acc + x;
      const int64_t tq = (int64_t)slot[kMaxFields];
      const uint32_t fq = (uint32_t)slot[kMaxFields + 1];
      if (tq < bt || (tq == bt && fq < bf)) {
        bt = tq;
        bf = fq;
      }
    }
    if (!any) continue;
    const int64_t w = w0 + (w1 - w0 == 2 ? (int64_t)kd : 0);
    if (w >= w1 || w >= R.cap) continue;
    if (f < nfields && f != 4) {
      row_column(R, f)[w] = acc;
    } else if (f == 4) {
      R.tmin[w] = bt;
    } else if (f == kMaxFields) {
      R.first[w] = bf;
      R.gpu[w] = 0xFF;
      R.kind[w] = (uint8_t)kd;
      for (int l = 0; l < D; ++l) R.path[(int64_t)l * R.cap + w] = kNone;
    }
  }
}

// first record of a workload row: the smallest input index among the records
// (or GPU rows) whose start equals the row's tmin
template <typename Src>
__global__ __launch_bounds__(kBlock) void k_agg_workload_first(
    Src src, int D, int64_t M, const uint32_t* rowof, RowsDev R) {
  const int64_t cnt = src.count();
  const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i >= cnt) return;
  uint32_t r, p[8], g, kind, fpos;
  bool ok;
  src.load(i, r, ok, p, g, kind, fpos);
  if (!ok) return;
  const uint32_t row = rowof[kind];
  if ((int64_t)row >= R.cap) return;
  if ((int64_t)src.field(4, r) == R.tmin[row])
    atomicMin(&R.first[row], src.first_of(r));
}

// Entries [0, nslots), or [0, *count) when nslots < 0; a slot holding
// kNone is empty.
// `clear` (optional): three flag words zeroed for the next heads pass
__global__ __launch_bounds__(kBlock) void k_agg_apply_overflow(
    Overflow ovf, RowsDev R, int nfields, int64_t nslots, uint32_t* clear) {
  const int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (clear && e < 3) clear[e] = 0;
  int64_t cnt = nslots >= 0 ? nslots : (int64_t)*ovf.count;
  if (cnt > ovf.cap) cnt = ovf.cap;
  if (e >= cnt) return;
  const uint32_t row = ovf.row[e];
  if (row == kNone || (int64_t)row >= R.cap) return;
  for (int f = 0; f < nfields; ++f)
    atomic_field(R, f, row, ovf.val[(int64_t)f * ovf.cap + e]);
}

// zero the sums of rows [level_offset[a], level_offset[b]) (atomic re-run)
__global__ __launch_bounds__(kBlock) void k_agg_zero_rows(
    const int64_t* level_offset, int a, int b, RowsDev R) {
  int64_t lo = level_offset[a], hi = level_offset[b];
  if (hi > R.cap) hi = R.cap;
  for (int64_t row = lo + (int64_t)blockIdx.x * kBlock + threadIdx.x; row < hi;
       row += (int64_t)gridDim.x * kBlock) {
    R.n[row] = 0;
    R.dur[row] = 0;
    R.gap[row] = 0;
    R.ovl[row] = 0;
    R.tmin[row] = kI64Max;
    R.tmax[row] = kI64Min;
    for (int q = 0; q < R.nc; ++q) R.ctr[(int64_t)q * R.cap + row] = 0;
  }
}

// ------------------------------------------------------- exact group ids
// Exact group ids, level by level from the outermost: the key of korder
// position p at marker level l is (its group id at level l - 1, or
// gpu * 2 + kind at l = 0) * (M + 2) + (its level-l marker, M + 1 for
// NONE), so that equal keys are equal paths; records left out by the filter
// get kfilt, above every key.  After a stable sort by key the group id of a
// position is the position of its group's first record.
__global__ __launch_bounds__(kBlock) void k_xk_keys(RecSrc S, int l,
                                                    const uint32_t* gprev,
                                                    uint64_t kfilt,
                                                    uint64_t* key,
                                                    uint32_t* val) {
  const int64_t pos = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (pos >= S.n) return;
  const uint32_t r = S.korder[pos];
  uint64_t k = kfilt;
  if (rec_pass(S, r)) {
    const uint64_t parent =
        l == 0 ? (uint64_t)S.gpu[r] * 2u + (uint64_t)kind_of(S.cls[r])
               : (uint64_t)gprev[pos];
    const uint32_t m = S.idx[(int64_t)l * S.n + r];
    const uint64_t mi = m == kNone ? (uint64_t)S.M + 1
                                   : ((int64_t)m >= S.M ? (uint64_t)S.M : m);
    k = parent * ((uint64_t)S.M + 2) + mi;
  }
  key[pos] = k;
  val[pos] = (uint32_t)pos;
}

__global__ __launch_bounds__(kBlock) void k_xk_heads(int64_t n,
                                                     const uint64_t* skey,
                                                     uint32_t* head) {
  const int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (q < n) head[q] = (q == 0 || skey[q] != skey[q - 1]) ? 1u : 0u;
}

// first[run] = position of the run's first item (the smallest: the sort is
// stable over ascending positions)
__global__ __launch_bounds__(kBlock) void k_xk_first(int64_t n,
                                                     const uint32_t* head,
                                                     const uint32_t* runx,
                                                     const uint32_t* sval,
                                                     uint32_t* first) {
  const int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (q < n && head[q]) first[runx[q]] = sval[q];
}

__global__ __launch_bounds__(kBlock) void k_xk_assign(
    int64_t n, const uint64_t* skey, uint64_t kfilt, const uint32_t* head,
    const uint32_t* runx, const uint32_t* sval, const uint32_t* first,
    uint32_t* gid) {
  const int64_t q = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (q >= n) return;
  gid[sval[q]] = skey[q] == kfilt ? kNone : first[runx[q] + head[q] - 1u];
}

__global__ void k_fill_u32_many(uint32_t** p, const int64_t* counts, int L,
                                uint32_t act) {
  const int li = blockIdx.y;
  if (li >= L || !((act >> li) & 1u)) return;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
       i < counts[li]; i += (int64_t)gridDim.x * blockDim.x)
    p[li][i] = 0xFFFFFFFFu;
}

__global__ void k_nat_init(uint32_t* flags, uint32_t* gs, int G) {
  const int i = (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (i < 3) flags[i] = 0;
  if (i < G) gs[i] = kNone;
}

__global__ void k_zero_u32(uint32_t* p, int n) {
  int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// ---------------------------------------------------------------------------
struct AggLayout {
  int L;
  int64_t ntiles;
  uint32_t* own[kMaxLevels];
  uint32_t* rowof[kMaxLevels];
  int64_t ks[kMaxLevels];
  uint32_t** own_tab;     // device copies of the pointer tables
  uint32_t** rowof_tab;
  int64_t* ks_dev;
  uint32_t* tilecnt;
  uint32_t* tilebase;
  uint32_t* scantmp;
  uint32_t* total;
  uint32_t* firstpos;
  uint32_t* ovf_count;    // [2]: count, lost
  uint32_t* ovf_row;
  uint64_t* ovf_val;
  int64_t ovf_cap;
  // fast path: head counts per wave tile of kWaveTile items
  int64_t ntiles_h;
  uint32_t* htc;          // [L][ntiles_h]
  uint32_t* htb;
  uint32_t* hscan;
  uint32_t* htotal;
  uint32_t* hflags;       // [0] keys not increasing, [1] kinds present,
                          // [2] input order unfit for the natural tiles
  uint32_t* htc2;         // one or two levels over rows
  uint32_t* htb2;
  uint32_t* hflags2;
  // natural tiles
  int G;
  int64_t nstride;        // 2 * (natural tiles + G): counts per level
  uint32_t* ntc;          // [L][nstride]
  uint32_t* ntb;
  uint32_t* nscan;
  int64_t lps;            // ntiles_h rounded up to kLpIpt
  int32_t* lpraw;         // [2][lps]
  int32_t* lp;
  uint8_t* tg;            // [ntiles_h + G]
  uint64_t* pair;         // [2G][kPairW] GPU row sums
  int64_t* stage;         // flags and level offsets for the host
  uint32_t* gs;           // [G]
  uint32_t* ge;
  uint32_t* gtb;          // [G + 1]
  // exact group ids (markers not nested)
  uint32_t* gk;           // [D][n]
  uint32_t* xflag;
  uint64_t* xskey;        // sorted keys
  uint32_t* xsval;        // positions in key order
  uint32_t* xhead;
  uint32_t* xrunx;
  uint32_t* xfirst;
  uint32_t* xtot;
  uint32_t* xscan;        // scan temporaries over n items
  ClassSortLayout xsort;
  uint32_t* ipath;        // [D][n] general-path items by korder position
  uint16_t* igk;          // [n]
};

static AggLayout agg_layout(Scratch& sc, int64_t n, int D, int64_t M,
                            int64_t cap, uint32_t act, int G) {
  AggLayout L;
  L.L = D + 2;
  L.ntiles = ceil_div(n, kAggTile);
  for (int li = 0; li < L.L; ++li) {
    // (exact group ids at the marker levels are korder positions < n)
    int64_t ks = key_space(li, D, M);
    if (li < D && n > ks) ks = n;
    L.ks[li] = ((act >> li) & 1u) ? ks : 1;
    L.own[li] = sc.take<uint32_t>(L.ks[li]);
    L.rowof[li] = sc.take<uint32_t>(L.ks[li]);
  }
  L.own_tab = sc.take<uint32_t*>(kMaxLevels);
  L.rowof_tab = sc.take<uint32_t*>(kMaxLevels);
  L.ks_dev = sc.take<int64_t>(kMaxLevels);
  L.tilecnt = sc.take<uint32_t>((int64_t)L.L * L.ntiles);
  L.tilebase = sc.take<uint32_t>((int64_t)L.L * L.ntiles);
  L.scantmp = sc.take<uint32_t>(scan_scratch_elems((int64_t)L.L * L.ntiles));
  L.total = sc.take<uint32_t>(1);
  L.firstpos = sc.take<uint32_t>(cap);
  L.ntiles_h = ceil_div(n, kWaveTile);
  L.nstride = 2 * (L.ntiles_h + G);
  L.ovf_cap = n / 64 > 65536 ? n / 64 : 65536;
  if (L.ovf_cap < 2 * L.nstride) L.ovf_cap = 2 * L.nstride;
  L.ovf_count = sc.take<uint32_t>(2);
  L.ovf_row = sc.take<uint32_t>(L.ovf_cap);
  L.ovf_val = sc.take<uint64_t>((int64_t)kMaxFields * L.ovf_cap);
  L.htc = sc.take<uint32_t>((int64_t)L.L * L.ntiles_h);
  L.htb = sc.take<uint32_t>((int64_t)L.L * L.ntiles_h);
  L.hscan = sc.take<uint32_t>(scan_scratch_elems((int64_t)L.L * L.ntiles_h));
  L.htotal = sc.take<uint32_t>(2);
  L.hflags = sc.take<uint32_t>(3);
  L.htc2 = sc.take<uint32_t>(2 * L.ntiles_h);
  L.htb2 = sc.take<uint32_t>(2 * L.ntiles_h);
  L.hflags2 = sc.take<uint32_t>(3);
  L.G = G;
  L.ntc = sc.take<uint32_t>((int64_t)L.L * L.nstride);
  L.ntb = sc.take<uint32_t>((int64_t)L.L * L.nstride);
  L.nscan = sc.take<uint32_t>(scan_scratch_elems((int64_t)L.L * L.nstride));
  L.lps = ceil_div(L.ntiles_h, (int64_t)kLpIpt) * kLpIpt;
  L.lpraw = sc.take<int32_t>(2 * L.lps);
  L.lp = sc.take<int32_t>(2 * L.lps);
  L.tg = sc.take<uint8_t>(L.ntiles_h + G);
  L.pair = sc.take<uint64_t>((int64_t)2 * G * kPairW);
  L.stage = sc.take<int64_t>(3 + kMaxLevels + 1);
  L.gs = sc.take<uint32_t>(G);
  L.ge = sc.take<uint32_t>(G);
  L.gtb = sc.take<uint32_t>(G + 1);
  L.gk = sc.take<uint32_t>((int64_t)(D > 0 ? D : 1) * n);
  L.xflag = sc.take<uint32_t>(1);
  L.xskey = sc.take<uint64_t>(n);
  L.xsval = sc.take<uint32_t>(n);
  L.xhead = sc.take<uint32_t>(n);
  L.xrunx = sc.take<uint32_t>(n);
  L.xfirst = sc.take<uint32_t>(n);
  L.xtot = sc.take<uint32_t>(1);
  L.xscan = sc.take<uint32_t>(scan_scratch_elems(n));
  L.xsort = class_sort_layout(sc, n, 256);
  L.ipath = sc.take<uint32_t>((int64_t)(D > 0 ? D : 1) * n);
  L.igk = sc.take<uint16_t>(n);
  return L;
}

static int bitlen_of(uint64_t x) {
  int b = 0;
  while (x) { ++b; x >>= 1; }
  return b;
}

// Exact group ids of the marker levels 0 .. lmax into L.gk (see k_xk_keys).
static int exact_group_ids(const AggLayout& L, const RecSrc& S, int lmax,
                           hipStream_t s) {
  const int64_t n = S.n;
  const dim3 g = grid_for(n, kBlock);
  for (int l = 0; l <= lmax; ++l) {
    // keys below kfilt = (parents) * (M + 2); parents: 512 (gpu, kind) ids
    // at level 0, positions below n after
    const unsigned __int128 kf =
        (unsigned __int128)(l == 0 ? 512u : (uint64_t)n) *
        (unsigned __int128)((uint64_t)S.M + 2);
    if (kf >> 63) return CHOPPER_EINVAL;
    const uint64_t kfilt = (uint64_t)kf;
    CHOPPER_HIP(launch("agg_exact_keys", k_xk_keys, g, dim3(kBlock), s, S, l,
                       (const uint32_t*)(l > 0 ? L.gk + (int64_t)(l - 1) * n
                                               : nullptr),
                       kfilt, L.xsort.key0, L.xsort.val0));
    int rc = radix_sort_pairs(L.xsort, bitlen_of(kfilt), L.xsval, L.xskey,
                              s);
    if (rc != CHOPPER_OK) return rc;
    CHOPPER_HIP(launch("agg_exact_keys", k_xk_heads, g, dim3(kBlock), s, n,
                       (const uint64_t*)L.xskey, L.xhead));
    CHOPPER_HIP(exclusive_scan<uint32_t>(L.xhead, L.xrunx, n, L.xscan,
                                         L.xtot, s));
    CHOPPER_HIP(launch("agg_exact_keys", k_xk_first, g, dim3(kBlock), s, n,
                       (const uint32_t*)L.xhead, (const uint32_t*)L.xrunx,
                       (const uint32_t*)L.xsval, L.xfirst));
    CHOPPER_HIP(launch("agg_exact_keys", k_xk_assign, g, dim3(kBlock), s, n,
                       (const uint64_t*)L.xskey, kfilt,
                       (const uint32_t*)L.xhead, (const uint32_t*)L.xrunx,
                       (const uint32_t*)L.xsval, (const uint32_t*)L.xfirst,
                       L.gk + (int64_t)l * n));
  }
  return CHOPPER_OK;
}

}  // namespace chopper

using namespace chopper;

// Fast path over all requested levels (MaxD >= depth); returns 1 when the
// groups are not runs and the general path must be used.  The natural tiles
// are tried first; when the input order does not qualify, the korder tiles
// count the heads again.
template <int kMD>
static int agg_fast(const AggLayout& L, const RecSrc& S, const RowsDev& R,
                    const Overflow& ovf, int64_t T, int Lv, uint32_t act,
                    int D, int64_t M, int nfields, chopper_rows* rows,
                    int level, bool want_workload, uint32_t* status,
                    hipEvent_t ready, hipStream_t s) {
  int rc = CHOPPER_OK;
  const int64_t Th = L.ntiles_h;
  const int G = L.G;
  const int64_t NW = Th + G;          // natural tile slots
  FromRecords fr{S};
  const NatGeom N{L.gtb, L.tg, L.gs, L.ge, L.lp, L.hflags + 2, Th, L.lps, G};
  const NatGeom none{};
  // the records reduction on the natural tiles: level li and, with `two`,
  // li - 1
  auto nat_records = [&](const NatGeom& NG, int li, bool two) -> int {
    const uint32_t* tb = L.ntb + (int64_t)li * L.nstride;
    const dim3 grid((unsigned)ceil_div(NW, (int64_t)kWavesPerBlock));
    if (two)
      CHOPPER_HIP(launch("agg_fast_reduce_records",
                         k_agg_fast_reduce<kMD, FromRecords, true, true>,
                         grid, dim3(kBlock), s, fr, NG, li, D, M, tb,
                         (const uint32_t*)(tb - L.nstride),
                         (const int64_t*)nullptr, R, ovf, NW));
    else
      CHOPPER_HIP(launch("agg_fast_reduce_records",
                         k_agg_fast_reduce<kMD, FromRecords, false, true>,
                         grid, dim3(kBlock), s, fr, NG, li, D, M, tb,
                         (const uint32_t*)nullptr, (const int64_t*)nullptr,
                         R, ovf, NW));
    return CHOPPER_OK;
  };
  // the level the records reduce to (with li0 - 1 when two0)
  const int li0 = level == CHOPPER_LEVEL_ALL
                      ? (D > 0 ? D - 1 : D)
                      : (level == CHOPPER_LEVEL_GPU ? D : level);
  const bool two0 = level == CHOPPER_LEVEL_ALL && D >= 2;
  bool spec = false;   // the natural-tile records reduction is queued
  // the fast-path flags and the level offsets (row counts per level size
  // the launches of the coarser levels); with `speculate` the natural-tile
  // records reduction, which needs none of them, is queued before the wait
  // and exits on the device unless the flags let it run
  uint32_t hf[3] = {1u, 0u, 1u};
  int64_t lo_h[kMaxLevels + 1];
  auto fetch_stage = [&](bool speculate) -> int {
    int64_t st[3 + kMaxLevels + 1];
    ReadBack rb;
    CHOPPER_HIP(read_back_start(L.stage,
                                sizeof(int64_t) * (size_t)(3 + Lv + 1), s,
                                &rb));
    // gap and ovl are read from here on: the caller's event first (the
    // read-back above does not wait for it)
    if (ready) CHOPPER_HIP(hipStreamWaitEvent(s, ready, 0));
    if (speculate) {
      NatGeom NS = N;
      NS.fflags = L.hflags;
      const int r = nat_records(NS, li0, two0);
      if (r != CHOPPER_OK) return r;
      spec = true;
    }
    CHOPPER_HIP(read_back_finish(&rb, st));
    for (int i = 0; i < 3; ++i) hf[i] = (uint32_t)st[i];
    for (int i = 0; i <= Lv; ++i) lo_h[i] = st[3 + i];
    return CHOPPER_OK;
  };
  CHOPPER_HIP(launch("agg_nat_init", k_nat_init, dim3(1), dim3(kBlock), s,
                     L.hflags, L.gs, G));
  CHOPPER_HIP(launch("agg_nat_pre", k_nat_pre,
                     dim3((unsigned)ceil_div(Th, (int64_t)kWavesPerBlock)),
                     dim3(kBlock), s, S.n, G, S.gpu, S.cls, S.start, Th,
                     L.lps, L.lpraw, L.gs, L.hflags + 2));
  CHOPPER_HIP(launch("agg_nat_tiles", k_nat_tiles,
                     dim3((unsigned)(1 + ceil_div(Th, kLpSpan))), dim3(1024), s,
                     S.n, G, Th, L.lps, (const int32_t*)L.lpraw, L.lp,
                     (const uint32_t*)L.gs, L.ge, L.gtb, L.tg,
                     (const uint32_t*)(L.hflags + 2)));
  CHOPPER_HIP(launch("agg_heads_nat", k_agg_heads_nat<kMD>,
                     dim3((unsigned)ceil_div(NW, (int64_t)kWavesPerBlock)),
                     dim3(kBlock), s, S, N, act, 0, Lv - 1, D, M, L.nstride,
                     L.ntc, L.hflags, status));
  CHOPPER_HIP(exclusive_scan<uint32_t>(L.ntc, L.ntb, (int64_t)Lv * L.nstride,
                                       L.nscan, L.htotal, s));
  CHOPPER_HIP(launch("agg_offsets", k_agg_offsets_fast, dim3(1), dim3(64),
                     s, Lv, L.nstride, (const uint32_t*)L.ntb,
                     (const uint32_t*)L.htotal, (const uint32_t*)L.hflags,
                     want_workload, rows->cap, rows->level_offset, L.stage,
                     status));
  rc = fetch_stage(true);
  if (rc != CHOPPER_OK) return rc;
  const bool nat = hf[2] == 0;
  if (!nat) {
    CHOPPER_HIP(launch("agg_zero", k_zero_u32, dim3(1), dim3(64), s,
                       L.hflags, 3));
    CHOPPER_HIP(launch("agg_heads_records", k_agg_heads<kMD, FromRecords>,
                       dim3((unsigned)ceil_div(Th, (int64_t)kWavesPerBlock)),
                       dim3(kBlock), s, fr, act, 0, Lv - 1, D, M, Th, L.htc,
                       L.hflags, status));
    CHOPPER_HIP(exclusive_scan<uint32_t>(L.htc, L.htb, (int64_t)Lv * Th,
                                         L.hscan, L.htotal, s));
    CHOPPER_HIP(launch("agg_offsets", k_agg_offsets_fast, dim3(1), dim3(64),
                       s, Lv, Th, (const uint32_t*)L.htb,
                       (const uint32_t*)L.htotal, (const uint32_t*)L.hflags,
                       want_workload, rows->cap, rows->level_offset, L.stage,
                       status));
    rc = fetch_stage(false);
    if (rc != CHOPPER_OK) return rc;
  }
  auto level_rows = [&](int li) -> int64_t {
    int64_t a = lo_h[li], b = lo_h[li + 1];
    if (b > rows->cap) b = rows->cap;
    return b > a ? b - a : 0;
  };
  if (hf[0] != 0) return 1;
  // finer < 0: from the records (two levels, li and li - 1, when `two`)
  auto fast_level = [&](int li, int finer, bool two) -> int {
    if (finer < 0) {
      int64_t ns;
      if (nat) {
        // (queued before the flags were read, when they allowed it)
        if (!(spec && li == li0 && two == two0)) {
          const int r = nat_records(N, li, two);
          if (r != CHOPPER_OK) return r;
        }
        ns = (two ? 4 : 2) * NW;
      } else {
        const uint32_t* tb = L.htb + (int64_t)li * Th;
        if (two)
          CHOPPER_HIP(launch("agg_fast_reduce_records",
                             k_agg_fast_reduce<kMD, FromRecords, true, false>,
                             dim3((unsigned)T), dim3(kBlock), s, fr, none, li,
                             D, M, tb, (const uint32_t*)(tb - Th),
                             (const int64_t*)nullptr, R, ovf, Th));
        else
          CHOPPER_HIP(launch("agg_fast_reduce_records",
                             k_agg_fast_reduce<kMD, FromRecords, false, false>,
                             dim3((unsigned)T), dim3(kBlock), s, fr, none, li,
                             D, M, tb, (const uint32_t*)nullptr,
                             (const int64_t*)nullptr, R, ovf, Th));
        ns = two ? 2 * Th : Th;
      }
      CHOPPER_HIP(launch("agg_apply_overflow", k_agg_apply_overflow,
                         grid_for(ns, kBlock), dim3(kBlock), s, ovf, R,
                         nfields, ns, L.hflags2));
    } else {
      // launches sized by the finer level's row count; with `two` also the
      // level li - 1 (heads of li - 1 first in the table, then li)
      const int64_t cnt = level_rows(finer);
      if (cnt == 0) return CHOPPER_OK;
      const int64_t nw = ceil_div(cnt, (int64_t)kWaveTile);
      const unsigned gr = (unsigned)ceil_div(nw, (int64_t)kWavesPerBlock);
      FromRows src{R, M, rows->level_offset, finer};
      const int lv0 = two ? li - 1 : li;
      const uint32_t lact = two ? (3u << (li - 1)) : (1u << li);
      // (the flags were zeroed by the previous overflow pass)
      CHOPPER_HIP(launch("agg_heads_rows", k_agg_heads<kMD, FromRows>,
                         dim3(gr), dim3(kBlock), s, src, lact, lv0, li, D, M,
                         nw, L.htc2, L.hflags2, status));
      CHOPPER_HIP(exclusive_scan<uint32_t>(L.htc2, L.htb2,
                                           (two ? 2 : 1) * nw, L.hscan,
                                           L.htotal + 1, s));
      const int64_t* r0 = rows->level_offset + li;
      if (two)
        CHOPPER_HIP(launch("agg_fast_reduce_rows",
                           k_agg_fast_reduce<kMD, FromRows, true, false>,
                           dim3(gr), dim3(kBlock), s, src, none, li, D, M,
                           (const uint32_t*)(L.htb2 + nw),
                           (const uint32_t*)L.htb2, r0, R, ovf, nw));
      else
        CHOPPER_HIP(launch("agg_fast_reduce_rows",
                           k_agg_fast_reduce<kMD, FromRows, false, false>,
                           dim3(gr), dim3(kBlock), s, src, none, li, D, M,
                           (const uint32_t*)L.htb2, (const uint32_t*)nullptr,
                           r0, R, ovf, nw));
      const int64_t ns = (two ? 2 : 1) * nw;
      CHOPPER_HIP(launch("agg_apply_overflow", k_agg_apply_overflow,
                         grid_for(ns, kBlock), dim3(kBlock), s, ovf, R,
                         nfields, ns, L.hflags2));
    }
    return CHOPPER_OK;
  };
  if (level == CHOPPER_LEVEL_ALL) {
    // the records give the two finest levels, coarser marker levels come
    // in pairs from the rows of the level below, the GPU rows from the
    // level-0 rows
    const bool two = D >= 2;
    rc = fast_level(D > 0 ? D - 1 : D, -1, two);
    if (rc != CHOPPER_OK) return rc;
    for (int li = D - (two ? 3 : 2); li >= 0; li -= 2) {
      rc = fast_level(li, li + 1, li >= 1);
      if (rc != CHOPPER_OK) return rc;
    }
    CHOPPER_HIP(launch("agg_gpu_rows", k_agg_gpu_sums,
                       dim3((unsigned)(2 * L.G)), dim3(kBlock), s,
                       (const int64_t*)rows->level_offset, R, nfields,
                       L.pair));
    CHOPPER_HIP(launch("agg_workload_from_gpu", k_agg_gpu_finish, dim3(1),
                       dim3(1024), s, (const int64_t*)rows->level_offset, D,
                       R, nfields, 2 * L.G, (const uint64_t*)L.pair));
  } else {
    rc = fast_level(level == CHOPPER_LEVEL_GPU ? D : level, -1, false);
    if (rc != CHOPPER_OK) return rc;
  }
  return CHOPPER_OK;
}

extern "C" int chopper_aggregate(const chopper_records* rec,
                                 const int64_t* start_al,
                                 const int64_t* end_al, const uint32_t* korder,
                                 const uint32_t* idx, int32_t depth,
                                 const int64_t* gap, const int64_t* ovl,
                                 const chopper_markers* mk, int32_t level,
                                 const chopper_filter* filter,
                                 chopper_rows* rows, void* scratch,
                                 size_t* scratch_bytes, uint32_t* status,
                                 void* ready, void* stream) {
  if (!validate_records(rec) || !validate_markers(mk) || !rows ||
      !scratch_bytes)
    return CHOPPER_EINVAL;
  const int64_t n = rec->n;
  const int D = depth;
  if (D < 0 || D > 8) return CHOPPER_EINVAL;
  if (mk && mk->depth != D) return CHOPPER_EINVAL;
  const int64_t M = mk ? mk->n : 0;
  if (filter && filter->use_iter && (!mk || (M > 0 && !mk->label)))
    return CHOPPER_EINVAL;
  if (n > 0 && (!start_al || !end_al || !korder || !gap || !ovl ||
                (D > 0 && !idx)))
    return CHOPPER_EINVAL;
  if (rows->cap < 0 || !rows->level_offset) return CHOPPER_EINVAL;
  if (rows->cap > 0 && (!rows->gpu || !rows->kind || !rows->n || !rows->dur ||
                        !rows->gap || !rows->ovl || !rows->tmin ||
                        !rows->tmax || !rows->first ||
                        (D > 0 && !rows->path) ||
                        (rec->n_counters > 0 && !rows->ctr)))
    return CHOPPER_EINVAL;
  uint32_t act = 0;
  if (level == CHOPPER_LEVEL_ALL) act = (1u << (D + 2)) - 1u;
  else if (level >= 0 && level < D) act = 1u << level;
  else if (level == CHOPPER_LEVEL_GPU) act = 1u << D;
  else if (level == CHOPPER_LEVEL_WORKLOAD) act = 1u << (D + 1);
  else return CHOPPER_EINVAL;

  Scratch probe(nullptr);
  agg_layout(probe, n, D, M, rows->cap, act, rec->n_gpus);
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  AggLayout L = agg_layout(sc, n, D, M, rows->cap, act, rec->n_gpus);
  const int Lv = L.L;
  const int64_t T = L.ntiles;
  const int nc = rec->n_counters;
  const int nfields = 6 + nc;

  RecSrc S;
  S.n = n;
  S.D = D;
  S.M = M;
  S.korder = korder;
  S.gpu = rec->gpu;
  S.cls = rec->cls;
  S.start = start_al;
  S.end = end_al;
  S.idx = idx;
  S.gap = gap;
  S.ovl = ovl;
  S.ctr = rec->counters;
  S.nc = nc;
  S.mlabel = mk ? mk->label : nullptr;
  memset(&S.f, 0, sizeof(S.f));
  S.gk = nullptr;
  S.ipath = nullptr;
  S.igk = nullptr;
  if (filter) {
    for (int q = 0; q < 4; ++q) S.f.gpu_mask[q] = filter->gpu_mask[q];
    S.f.class_mask = filter->class_mask;
    S.f.use_iter = filter->use_iter;
    S.f.iter_lo = filter->iter_lo;
    S.f.iter_hi = filter->iter_hi;
    S.f.active = 1;
  }
  RowsDev R;
  R.cap = rows->cap;
  R.path = rows->path;
  R.gpu = rows->gpu;
  R.kind = rows->kind;
  R.n = rows->n;
  R.dur = rows->dur;
  R.gap = rows->gap;
  R.ovl = rows->ovl;
  R.tmin = rows->tmin;
  R.tmax = rows->tmax;
  R.first = rows->first;
  R.ctr = rows->ctr;
  R.firstpos = L.firstpos;
  R.D = D;
  R.nc = nc;

  Overflow ovf{L.ovf_count, L.ovf_count + 1, L.ovf_row, L.ovf_val, L.ovf_cap};
  const bool want_workload = (act >> (D + 1)) & 1u;

  // ---- fast path: every group is one run of consecutive records
  // (the fast path addresses columns with 32-bit byte offsets)
  if (n > 0 && !filter && level != CHOPPER_LEVEL_WORKLOAD &&
      n < ((int64_t)1 << 29) && rows->cap < ((int64_t)1 << 29)) {
    rc = D <= 4 ? agg_fast<4>(L, S, R, ovf, T, Lv, act, D, M, nfields, rows,
                              level, want_workload, status,
                              (hipEvent_t)ready, s)
                : agg_fast<8>(L, S, R, ovf, T, Lv, act, D, M, nfields, rows,
                              level, want_workload, status,
                              (hipEvent_t)ready, s);
    if (rc != 1) return rc;
  }

  // ---- general path: per-level owner election (it reads gap and ovl)
  if (ready) CHOPPER_HIP(hipStreamWaitEvent(s, (hipEvent_t)ready, 0));
  // pointer tables for the per-level owner / row maps
  CHOPPER_HIP(hipMemcpyAsync(L.own_tab, L.own, sizeof(L.own),
                             hipMemcpyHostToDevice, s));
  CHOPPER_HIP(hipMemcpyAsync(L.rowof_tab, L.rowof, sizeof(L.rowof),
                             hipMemcpyHostToDevice, s));
  CHOPPER_HIP(hipMemcpyAsync(L.ks_dev, L.ks, sizeof(L.ks),
                             hipMemcpyHostToDevice, s));
  int64_t maxks = 1;
  for (int li = 0; li < Lv; ++li) maxks = L.ks[li] > maxks ? L.ks[li] : maxks;
  unsigned fx = (unsigned)ceil_div(maxks, kBlock);
  if (fx > 4096) fx = 4096;
  CHOPPER_HIP(launch("agg_fill_owner", k_fill_u32_many, dim3(fx, Lv),
                     dim3(kBlock), s, L.own_tab, (const int64_t*)L.ks_dev, Lv,
                     act));
  const uint32_t atomic_levels = (1u << D) | (1u << (D + 1));
  if (n > 0) {
    // the items once, in korder order, for the passes below
    CHOPPER_HIP(launch("agg_items", k_agg_items, grid_for(n, kBlock),
                       dim3(kBlock), s, S, L.ipath, L.igk));
    S.ipath = L.ipath;
    S.igk = L.igk;
    CHOPPER_HIP(launch("agg_elect", k_agg_elect, dim3((unsigned)T),
                       dim3(kBlock), s, S, act, L.own_tab));
    CHOPPER_HIP(launch("agg_count", k_agg_count, dim3((unsigned)T),
                       dim3(kBlock), s, S, act, L.own_tab, T, L.tilecnt));
  }
  CHOPPER_HIP(exclusive_scan<uint32_t>(L.tilecnt, L.tilebase, (int64_t)Lv * T,
                                       L.scantmp, L.total, s));
  CHOPPER_HIP(launch("agg_offsets", k_agg_offsets, dim3(1), dim3(64), s, Lv, T,
                     (const uint32_t*)L.tilebase, (const uint32_t*)L.total,
                     rows->cap, rows->level_offset, status));
  if (n == 0) return CHOPPER_OK;
  CHOPPER_HIP(launch("agg_assign", k_agg_assign, dim3((unsigned)T),
                     dim3(kBlock), s, S, act, atomic_levels, L.own_tab,
                     L.rowof_tab, T, (const uint32_t*)L.tilebase, R));
  CHOPPER_HIP(launch("agg_zero", k_zero_u32, dim3(1), dim3(64), s,
                     L.ovf_count, 2));
  CHOPPER_HIP(launch("agg_zero", k_zero_u32, dim3(1), dim3(64), s,
                     L.xflag, 1));

  // order of work: finest marker level from records, coarser marker levels
  // from the rows below, GPU rows from level-0 rows, workload from GPU rows
  auto run_level = [&](int li, bool atomic_mode) -> int {
    int finer = -1;                       // level whose rows feed this one
    if (level == CHOPPER_LEVEL_ALL) {
      if (li < D - 1) finer = li + 1;
      else if (li == D && D > 0) finer = 0;
      else if (li == D + 1) finer = D;
    }
    if (!atomic_mode)
      CHOPPER_HIP(launch("agg_zero", k_zero_u32, dim3(1), dim3(64), s,
                         L.ovf_count, 1));
    if (finer < 0) {
      FromRecords src{S};
      CHOPPER_HIP(launch("agg_reduce_records", k_agg_reduce<FromRecords>,
                         dim3((unsigned)T), dim3(kBlock), s, src, li, D, M,
                         atomic_mode, (const uint32_t*)L.own[li],
                         (const uint32_t*)L.rowof[li], R, ovf, nfields,
                         status, L.xflag));
    } else {
      FromRows src{R, M, rows->level_offset, finer, S.gk, n};
      // rows of the finer level never outnumber the records
      CHOPPER_HIP(launch("agg_reduce_rows", k_agg_reduce<FromRows>,
                         dim3((unsigned)T), dim3(kBlock), s, src, li, D, M,
                         atomic_mode, (const uint32_t*)L.own[li],
                         (const uint32_t*)L.rowof[li], R, ovf, nfields,
                         status, L.xflag));
    }
    if (!atomic_mode)
      CHOPPER_HIP(launch("agg_apply_overflow", k_agg_apply_overflow,
                         grid_for(L.ovf_cap, kBlock), dim3(kBlock), s, ovf, R,
                         nfields, (int64_t)-1, (uint32_t*)nullptr));
    if (li == D + 1) {
      if (finer < 0) {
        FromRecords src{S};
        CHOPPER_HIP(launch("agg_workload_first",
                           k_agg_workload_first<FromRecords>,
                           grid_for(n, kBlock), dim3(kBlock), s, src, D, M,
                           (const uint32_t*)L.rowof[li], R));
      } else {
        FromRows src{R, M, rows->level_offset, finer, S.gk, n};
        CHOPPER_HIP(launch("agg_workload_first", k_agg_workload_first<FromRows>,
                           grid_for(n, kBlock), dim3(kBlock), s, src, D, M,
                           (const uint32_t*)L.rowof[li], R));
      }
    }
    return CHOPPER_OK;
  };
  int order_levels[kMaxLevels];
  int nl = 0;
  for (int li = D - 1; li >= 0; --li)
    if ((act >> li) & 1u) order_levels[nl++] = li;
  if ((act >> D) & 1u) order_levels[nl++] = D;
  if ((act >> (D + 1)) & 1u) order_levels[nl++] = D + 1;
  for (int q = 0; q < nl; ++q) {
    const int li = order_levels[q];
    rc = run_level(li, (atomic_levels >> li) & 1u);
    if (rc != CHOPPER_OK) return rc;
  }
  // markers not nested (a record's path differed from its row's): group by
  // the whole path, with exact group ids, and run the levels again
  uint32_t conflict = 0;
  CHOPPER_HIP(read_back(L.xflag, &conflict, sizeof(uint32_t), s));
  int lmax = -1;
  for (int li = 0; li < D; ++li)
    if ((act >> li) & 1u) lmax = li;
  if (conflict && lmax >= 0 && S.gk == nullptr) {
    rc = exact_group_ids(L, S, lmax, s);
    if (rc != CHOPPER_OK) return rc;
    S.gk = L.gk;
    CHOPPER_HIP(launch("agg_fill_owner", k_fill_u32_many, dim3(fx, Lv),
                       dim3(kBlock), s, L.own_tab, (const int64_t*)L.ks_dev,
                       Lv, act));
    CHOPPER_HIP(launch("agg_elect", k_agg_elect, dim3((unsigned)T),
                       dim3(kBlock), s, S, act, L.own_tab));
    CHOPPER_HIP(launch("agg_count", k_agg_count, dim3((unsigned)T),
                       dim3(kBlock), s, S, act, L.own_tab, T, L.tilecnt));
    CHOPPER_HIP(exclusive_scan<uint32_t>(L.tilecnt, L.tilebase,
                                         (int64_t)Lv * T, L.scantmp, L.total,
                                         s));
    CHOPPER_HIP(launch("agg_offsets", k_agg_offsets, dim3(1), dim3(64), s, Lv,
                       T, (const uint32_t*)L.tilebase,
                       (const uint32_t*)L.total, rows->cap,
                       rows->level_offset, status));
    CHOPPER_HIP(launch("agg_assign", k_agg_assign, dim3((unsigned)T),
                       dim3(kBlock), s, S, act, atomic_levels, L.own_tab,
                       L.rowof_tab, T, (const uint32_t*)L.tilebase, R));
    CHOPPER_HIP(launch("agg_zero", k_zero_u32, dim3(1), dim3(64), s,
                       L.ovf_count, 2));
    for (int q = 0; q < nl; ++q) {
      const int li = order_levels[q];
      rc = run_level(li, (atomic_levels >> li) & 1u);
      if (rc != CHOPPER_OK) return rc;
    }
  }
  // an overflow list that did not fit: redo the marker levels with atomics
  uint32_t lost = 0;
  CHOPPER_HIP(read_back(L.ovf_count + 1, &lost, sizeof(uint32_t), s));
  if (lost) {
    for (int q = 0; q < nl; ++q) {
      const int li = order_levels[q];
      CHOPPER_HIP(launch("agg_zero_rows", k_agg_zero_rows, dim3(1024),
                         dim3(kBlock), s, (const int64_t*)rows->level_offset,
                         li, li + 1, R));
      rc = run_level(li, true);
      if (rc != CHOPPER_OK) return rc;
    }
  }
  return CHOPPER_OK;
}
