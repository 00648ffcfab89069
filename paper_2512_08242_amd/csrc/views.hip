// Re-keyed views of the aggregated run and their medians (caption of Fig.
// end_to_end: duration and launch overhead per phase and kernel class,
// medians across iterations and GPUs, throughput from the largest duration
// plus launch overhead across GPUs; Section V-B / Fig. operation_time:
// operation duration summed across layers with its bubbles; Section IV:
// warm-up iterations are not sampled).
//
// Units (one GPU's iteration marker) get dense numbers from a scan of the
// marker levels.  The class view reads the records once in wave tiles: per
// distinct (unit, phase) of a tile the lanes sum their items per class and
// one wave reduction per class and field feeds one atomic add; a tile with
// more distinct pairs than a few (records out of time order) adds the rest
// item by item.  The
// operation view re-keys the rows of the operation level the same way,
// through a per-wave LDS table of (operation, kind) sums.  Medians take one
// 1024-thread block per group: a radix selection of the two middle order
// statistics, eight bits per pass from the highest bit in which the group's
// values differ, with the counts of each digit in LDS.
#include "common.h"
#include "wave.h"

namespace chopper {

bool validate_records(const chopper_records* r);
bool validate_markers(const chopper_markers* m);

namespace {

constexpr int kViewClasses = 8;
constexpr int kMaxPhases = 16;
constexpr int kMaxOps = 128;
constexpr int kMedThreads = 1024;
constexpr int kMedIpt = 8;       // items per thread held in registers
constexpr int kWaveGroups = 4;   // groups a record wave sums before per-item adds
constexpr uint64_t kSign = 1ull << 63;

__global__ void k_view_fill(uint64_t* p, int64_t n, uint64_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

constexpr int kRankThreads = 1024;
constexpr int kRankIpt = 8;
constexpr int64_t kRankTile = (int64_t)kRankThreads * kRankIpt;

// level == iter_level flags of thread t's kRankIpt consecutive markers
__device__ inline uint32_t unit_bits(const uint8_t* level, int64_t nm,
                                     int64_t m0, int iter_level) {
  uint32_t b = 0;
  if (m0 + kRankIpt <= nm && ((uintptr_t)(level + m0) & 7) == 0) {
    const uint64_t w = *(const uint64_t*)(level + m0);
#pragma unroll
    for (int j = 0; j < kRankIpt; ++j)
      if (((w >> (8 * j)) & 0xFFu) == (uint64_t)(uint8_t)iter_level)
        b |= 1u << j;
  } else {
#pragma unroll
    for (int j = 0; j < kRankIpt; ++j)
      if (m0 + j < nm && level[m0 + j] == (uint8_t)iter_level) b |= 1u << j;
  }
  return b;
}

template <typename T>
__device__ inline T block_sum_1024(T v, T* s_w) {
  const int lane = lane_id(), w = (int)(threadIdx.x / kWave);
  v = lane63(wave_incl(v, OpAdd(), (T)0));
  if (lane == 0) s_w[w] = v;
  __syncthreads();
  T s = 0;
  for (int i = 0; i < kRankThreads / kWave; ++i) s += s_w[i];
  __syncthreads();
  return s;
}

// units per tile of kRankTile markers
__global__ __launch_bounds__(kRankThreads) void k_view_count(
    const uint8_t* level, int64_t nm, int iter_level, uint32_t* tilecnt) {
  __shared__ uint32_t s_w[kRankThreads / kWave];
  const int64_t m0 = (int64_t)blockIdx.x * kRankTile +
                     (int64_t)threadIdx.x * kRankIpt;
  const uint32_t c = (uint32_t)__popc(unit_bits(level, nm, m0, iter_level));
  const uint32_t tot = block_sum_1024(c, s_w);
  if (threadIdx.x == 0) tilecnt[blockIdx.x] = tot;
}

// Unit numbers: block b adds up the counts of the tiles before it itself,
// then numbers its units in marker order (unit_of is written for the units
// only); the last block writes the count.
__global__ __launch_bounds__(kRankThreads) void k_view_rank(
    const uint8_t* level, int64_t nm, int iter_level, const uint32_t* tilecnt,
    int64_t cap, uint32_t* unit_of, uint32_t* unit_marker, uint32_t* total,
    int64_t* n_units, uint32_t* status) {
  __shared__ uint32_t s_w[kRankThreads / kWave];
  uint32_t p = 0;
  for (int64_t i = threadIdx.x; i < (int64_t)blockIdx.x; i += kRankThreads)
    p += tilecnt[i];
  const uint32_t before = block_sum_1024(p, s_w);
  const int64_t m0 = (int64_t)blockIdx.x * kRankTile +
                     (int64_t)threadIdx.x * kRankIpt;
  const uint32_t b = unit_bits(level, nm, m0, iter_level);
  const uint32_t c = (uint32_t)__popc(b);
  const int lane = lane_id(), w = (int)(threadIdx.x / kWave);
  const uint32_t incl = wave_incl(c, OpAdd(), 0u);
  if (lane == kWave - 1) s_w[w] = incl;
  __syncthreads();
  uint32_t r = before + incl - c, tot = before;
  for (int i = 0; i < kRankThreads / kWave; ++i) {
    if (i < w) r += s_w[i];
    tot += s_w[i];
  }
#pragma unroll
  for (int j = 0; j < kRankIpt; ++j)
    if ((b >> j) & 1u) {
      unit_of[m0 + j] = r;
      if ((int64_t)r < cap) unit_marker[r] = (uint32_t)(m0 + j);
      ++r;
    }
  if (threadIdx.x == 0 && (int64_t)(blockIdx.x + 1) * kRankTile >= nm) {
    *total = tot;
    *n_units = (int64_t)tot;
    if ((int64_t)tot > cap) atomicOr(status, CHOPPER_ST_ROWS_OVERFLOW);
  }
}

__global__ void k_view_zero(uint32_t* p, int64_t* n_units) {
  *p = 0;
  *n_units = 0;
}

__device__ inline uint64_t wave_sum(uint64_t v) {
  return lane63(wave_incl(v, OpAdd(), (uint64_t)0));
}

// The key of the first pending item of the first lane that has one; every
// lane then marks its pending items with that key in `hit`.  Returns false
// when no item is pending.
__device__ inline bool next_group(uint32_t pend,
                                  const uint64_t (&key)[kTileIpt],
                                  uint64_t& k, uint32_t& hit) {
  const uint64_t act = __ballot(pend != 0u);
  if (act == 0) return false;
  const int leader = __ffsll((long long)act) - 1;
  // this lane's first pending key (no indexing, so the keys stay in
  // registers)
  uint64_t mine = 0;
  bool found = false;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j)
    if (!found && ((pend >> j) & 1u)) {
      mine = key[j];
      found = true;
    }
  k = (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)mine,
                                                    leader) |
      ((uint64_t)(uint32_t)__builtin_amdgcn_readlane(
           (int)(uint32_t)(mine >> 32), leader) << 32);
  hit = 0;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j)
    if (((pend >> j) & 1u) && key[j] == k) hit |= 1u << j;
  return true;
}

// Unit of an iteration marker m (kNone if m is not one or does not fit).
__device__ inline uint32_t unit_of_marker(uint32_t m, int64_t nm,
                                          const uint8_t* level, int iter_level,
                                          const uint32_t* unit_of,
                                          int64_t ucap) {
  if ((int64_t)m >= nm) return kNone;
  const uint8_t lv = level[m];
  const uint32_t u = unit_of[m];   // meaningful for iteration markers only
  return lv == (uint8_t)iter_level && (int64_t)u < ucap ? u : kNone;
}

// Class view and busy time from the records; one wave per kWaveTile records.
// Items are grouped by their (iteration marker, phase marker) pair; the unit
// and the phase label are looked up once per group.
__global__ __launch_bounds__(kBlock) void k_view_records(
    int64_t n, const uint8_t* cls, const int64_t* start, const int64_t* end,
    const int64_t* gap, const uint32_t* idx_iter, const uint32_t* idx_phase,
    const uint8_t* level, int iter_level, const uint32_t* unit_of,
    const uint32_t* label, int64_t nm, const uint32_t* units, int64_t cap,
    int P, uint64_t* cls_tab, int64_t* busy) {
  __shared__ uint64_t s_acc[kWavesPerBlock][2 * kViewClasses * kWave];
  __shared__ uint32_t s_cnt[kWavesPerBlock][kViewClasses * kWave];
  const int lane = lane_id();
  const int wv = (int)(threadIdx.x / kWave);
  const int64_t w = (int64_t)blockIdx.x * kWavesPerBlock + wv;
  const int64_t base = w * kWaveTile;
  if (base >= n) return;
  int64_t ucap = (int64_t)*units;
  ucap = ucap < cap ? ucap : cap;
  uint64_t ikey[kTileIpt], key[kTileIpt], d[kTileIpt], g[kTileIpt];
  uint32_t c[kTileIpt];
  uint32_t pb = 0, pc = 0;   // pending items: busy, class view
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const int64_t r = base + (int64_t)j * kWave + lane;
    const bool valid = r < n;
    const uint32_t mi = valid ? idx_iter[r] : kNone;
    const uint32_t mp = valid ? idx_phase[r] : kNone;
    c[j] = valid ? (uint32_t)cls[r] : 255u;
    d[j] = valid ? (uint64_t)(end[r] - start[r]) : 0ull;
    g[j] = valid ? (uint64_t)gap[r] : 0ull;
    ikey[j] = mi;
    key[j] = (uint64_t)mi << 32 | mp;
    if (mi != kNone && !kind_of(c[j])) pb |= 1u << j;
    if (mi != kNone && mp != kNone && c[j] < (uint32_t)kViewClasses)
      pc |= 1u << j;
  }
  uint64_t k;
  uint32_t hit;
  // busy: compute records by iteration marker; after kWaveGroups groups the
  // rest of the tile (an input out of time order) adds item by item
  for (int grp = 0; grp < kWaveGroups && next_group(pb, ikey, k, hit);
       ++grp) {
    const uint32_t u = unit_of_marker((uint32_t)k, nm, level, iter_level,
                                      unit_of, ucap);
    uint64_t x = 0;
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j)
      if ((hit >> j) & 1u) x += d[j] + g[j];
    x = wave_sum(x);
    if (lane == 0 && u != kNone) atomicAdd((unsigned long long*)&busy[u], x);
    pb &= ~hit;
  }
  if (__ballot(pb != 0u) != 0) {
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j)
      if ((pb >> j) & 1u) {
        const uint32_t u = unit_of_marker((uint32_t)ikey[j], nm, level,
                                          iter_level, unit_of, ucap);
        if (u != kNone)
          atomicAdd((unsigned long long*)&busy[u], d[j] + g[j]);
      }
  }
  // class view by (iteration marker, phase marker): each lane adds its items
  // into its own LDS column per class (dur and gap rows, and a count row),
  // then groups of lanes add the rows up
  uint64_t* acc = s_acc[wv];
  uint32_t* cnt = s_cnt[wv];
  const int64_t ncls = cap * P * kViewClasses;
  for (int grp = 0; grp < kWaveGroups && next_group(pc, key, k, hit);
       ++grp) {
    const uint32_t u = unit_of_marker((uint32_t)(k >> 32), nm, level,
                                      iter_level, unit_of, ucap);
    const uint32_t mp = (uint32_t)k;
    const uint32_t p = (int64_t)mp < nm ? label[mp] : kNone;
    pc &= ~hit;
    if (u == kNone || p >= (uint32_t)P) continue;
#pragma unroll
    for (int r = 0; r < 2 * kViewClasses; ++r) acc[r * kWave + lane] = 0;
#pragma unroll
    for (int r = 0; r < kViewClasses; ++r) cnt[r * kWave + lane] = 0;
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j)
      if ((hit >> j) & 1u) {
        acc[c[j] * kWave + lane] += d[j];
        acc[(kViewClasses + c[j]) * kWave + lane] += g[j];
        cnt[c[j] * kWave + lane] += 1u;
      }
    wave_sync();
    // lanes 4r .. 4r + 3 add up row r of the dur / gap rows, lanes
    // 8c .. 8c + 7 the count row of class c
    const int r = lane >> 2, q = lane & 3;
    uint64_t sv = 0;
#pragma unroll
    for (int i = 0; i < kWave / 4; ++i) sv += acc[r * kWave + q * 16 + i];
    sv += __shfl_xor(sv, 1, kWave);
    sv += __shfl_xor(sv, 2, kWave);
    const int cn = lane >> 3, qn = lane & 7;
    uint32_t sn = 0;
#pragma unroll
    for (int i = 0; i < kWave / 8; ++i) sn += cnt[cn * kWave + qn * 8 + i];
    sn += __shfl_xor(sn, 1, kWave);
    sn += __shfl_xor(sn, 2, kWave);
    sn += __shfl_xor(sn, 4, kWave);
    const int cr = r & (kViewClasses - 1);
    const uint32_t ncr = (uint32_t)__shfl((int)sn, cr * 8, kWave);
    const int64_t col = ((int64_t)p * kViewClasses) * cap + u;
    if (q == 0 && ncr != 0)
      atomicAdd((unsigned long long*)&cls_tab[(1 + (r >> 3)) * ncls + col +
                                              (int64_t)cr * cap],
                sv);
    if (qn == 0 && sn != 0)
      atomicAdd((unsigned long long*)&cls_tab[col + (int64_t)cn * cap],
                (uint64_t)sn);
    wave_sync();
  }
  if (__ballot(pc != 0u) == 0) return;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j)
    if ((pc >> j) & 1u) {
      const uint32_t u = unit_of_marker((uint32_t)(key[j] >> 32), nm, level,
                                        iter_level, unit_of, ucap);
      const uint32_t mp = (uint32_t)key[j];
      const uint32_t p = (int64_t)mp < nm ? label[mp] : kNone;
      if (u == kNone || p >= (uint32_t)P) continue;
      const int64_t col = ((int64_t)p * kViewClasses + c[j]) * cap + u;
      atomicAdd((unsigned long long*)&cls_tab[col], 1ull);
      atomicAdd((unsigned long long*)&cls_tab[ncls + col], d[j]);
      atomicAdd((unsigned long long*)&cls_tab[2 * ncls + col], g[j]);
    }
}

// Operation view: the rows of the operation level re-keyed by (unit, phase
// label, operation label, kind); one wave per kWaveTile rows, per distinct
// (unit, phase) of the tile a per-wave LDS table of the (operation, kind)
// sums, flushed with one atomic add per field of each entry used.
struct RowCols {
  const int64_t* level_offset;
  const uint32_t* path;     // [depth][cap]
  const uint8_t* kind;
  const uint64_t* n;
  const int64_t* dur;
  const int64_t* gap;
  const int64_t* ovl;
  int64_t cap;
};

__global__ __launch_bounds__(kBlock) void k_view_rows(
    RowCols R, int lv_iter, int lv_phase, int lv_op, const uint8_t* level,
    const uint32_t* unit_of, const uint32_t* label, int64_t nm,
    const uint32_t* units, int64_t cap, int P, int O, uint64_t* op_tab) {
  __shared__ uint64_t s_tab[kWavesPerBlock][kMaxOps * 2 * 4];
  const int lane = lane_id();
  const int wv = (int)(threadIdx.x / kWave);
  int64_t lo = R.level_offset[lv_op], hi = R.level_offset[lv_op + 1];
  if (hi > R.cap) hi = R.cap;
  if (lo > hi) lo = hi;
  const int64_t base =
      lo + ((int64_t)blockIdx.x * kWavesPerBlock + wv) * kWaveTile;
  if (base >= hi) return;
  int64_t ucap = (int64_t)*units;
  ucap = ucap < cap ? ucap : cap;
  uint64_t* tab = s_tab[wv];
  const int ne = O * 2;
  uint64_t key[kTileIpt], v[kTileIpt][4];
  uint32_t sub[kTileIpt];
  uint32_t pend = 0;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const int64_t row = base + (int64_t)j * kWave + lane;
    const bool valid = row < hi;
    const uint32_t p0 =
        valid ? R.path[(int64_t)lv_iter * R.cap + row] : kNone;
    const uint32_t p1 =
        valid ? R.path[(int64_t)lv_phase * R.cap + row] : kNone;
    const uint32_t p3 = valid ? R.path[(int64_t)lv_op * R.cap + row] : kNone;
    const uint32_t op = (int64_t)p3 < nm ? label[p3] : kNone;
    key[j] = (uint64_t)p0 << 32 | p1;
    sub[j] = op * 2u + (valid && R.kind[row] ? 1u : 0u);
    v[j][0] = valid ? R.n[row] : 0ull;
    v[j][1] = valid ? (uint64_t)R.dur[row] : 0ull;
    v[j][2] = valid ? (uint64_t)R.gap[row] : 0ull;
    v[j][3] = valid ? (uint64_t)R.ovl[row] : 0ull;
    if (p0 != kNone && p1 != kNone && op < (uint32_t)O) pend |= 1u << j;
  }
  const int64_t nop = cap * P * O * 2;
  uint64_t k;
  uint32_t hit;
  while (next_group(pend, key, k, hit)) {
    pend &= ~hit;
    const uint32_t u = unit_of_marker((uint32_t)(k >> 32), nm, level,
                                      lv_iter, unit_of, ucap);
    const uint32_t mp = (uint32_t)k;
    const uint32_t ph = (int64_t)mp < nm ? label[mp] : kNone;
    if (u == kNone || ph >= (uint32_t)P) continue;
    for (int e = lane; e < ne * 4; e += kWave) tab[e] = 0;
    wave_sync();
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j)
      if ((hit >> j) & 1u) {
#pragma unroll
        for (int f = 0; f < 4; ++f)
          atomicAdd((unsigned long long*)&tab[sub[j] * 4 + f], v[j][f]);
      }
    wave_sync();
    const int64_t g0 = (int64_t)ph * O * 2;
    for (int e = lane; e < ne; e += kWave) {
      if (tab[e * 4] == 0) continue;
      const int64_t at = (g0 + e) * cap + u;
#pragma unroll
      for (int f = 0; f < 4; ++f)
        atomicAdd((unsigned long long*)&op_tab[f * nop + at], tab[e * 4 + f]);
    }
    wave_sync();
  }
}

__global__ void k_view_iter_max(const uint32_t* units, int64_t cap,
                                const uint32_t* unit_marker,
                                const uint32_t* label, const int64_t* busy,
                                int NI, int64_t* iter_max) {
  int64_t U = (int64_t)*units;
  U = U < cap ? U : cap;
  const int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= U) return;
  const uint32_t lab = label[unit_marker[u]];
  if (lab < (uint32_t)NI)
    atomicMax((long long*)&iter_max[lab], (long long)busy[u]);
}

// ---------------------------------------------------------------------------
// Medians.  Group g < P * 8: class view entry g; then the operation view
// entries; the last group: the iteration maxima.
struct MedArgs {
  const uint32_t* units;
  int64_t cap;
  const uint32_t* unit_marker;
  const uint32_t* label;
  uint32_t warmup;
  int P, O, NI;
  const uint64_t* cls_tab;
  const uint64_t* op_tab;
  const int64_t* iter_max;
  double* cls_med;
  int64_t* cls_cnt;
  double* op_med;
  int64_t* op_cnt;
  double* iter_med;
  int64_t* iter_cnt;
};

struct MedSrc {
  const uint64_t* n;      // entry counts (null: the iteration maxima)
  const uint64_t* d;
  const uint64_t* g;
  int64_t stride;         // between units
  int64_t items;
};

__global__ __launch_bounds__(kMedThreads) void k_view_medians(MedArgs A) {
  __shared__ uint32_t s_hist[2][256];
  __shared__ uint64_t s_red[kMedThreads / kWave];
  __shared__ uint64_t s_sel[4];
  const int t = (int)threadIdx.x;
  const int lane = lane_id(), wv = t / kWave;
  const int64_t gi = blockIdx.x;
  const int64_t ncg = (int64_t)A.P * kViewClasses;
  const int64_t nog = (int64_t)A.P * A.O * 2;
  int64_t U = (int64_t)*A.units;
  U = U < A.cap ? U : A.cap;
  MedSrc S;
  double* med;
  int64_t* cnt;
  int64_t off, mstride;
  int nstat;
  if (gi < ncg) {
    const int64_t col = A.cap * ncg, at = gi * A.cap;
    S = MedSrc{A.cls_tab + at, A.cls_tab + col + at, A.cls_tab + 2 * col + at,
               1, U};
    med = A.cls_med;
    cnt = A.cls_cnt;
    off = gi;
    mstride = ncg;
    nstat = 3;
  } else if (gi < ncg + nog) {
    const int64_t o = gi - ncg, col = A.cap * nog, at = o * A.cap;
    S = MedSrc{A.op_tab + at, A.op_tab + col + at, A.op_tab + 2 * col + at, 1,
               U};
    med = A.op_med;
    cnt = A.op_cnt;
    off = o;
    mstride = nog;
    nstat = 3;
  } else {
    S = MedSrc{nullptr, (const uint64_t*)A.iter_max, nullptr, 1,
               (int64_t)A.NI};
    med = A.iter_med;
    cnt = A.iter_cnt;
    off = 0;
    mstride = 1;
    nstat = 1;
  }
  // item i is in the group when its unit is past the warm-up and its entry
  // is not empty (iteration maxima: i >= warmup and a unit had label i)
  auto member = [&](int64_t i) -> bool {
    if (i >= S.items) return false;
    if (!S.n) return i >= (int64_t)A.warmup && (int64_t)S.d[i] >= 0;
    return A.label[A.unit_marker[i]] >= A.warmup && S.n[i * S.stride] != 0;
  };
  // order-preserving unsigned key of statistic st of item i
  auto key_of = [&](int64_t i, int st) -> uint64_t {
    const uint64_t d = S.d[i * S.stride];
    if (st == 0) return d ^ kSign;
    const uint64_t g = S.g[i * S.stride];
    return (st == 1 ? g : d + g) ^ kSign;
  };
  // the first kMedIpt items of each thread are held in registers, items
  // past kMedIpt * kMedThreads are read again in every pass
  uint32_t mine = 0;
  int64_t m = 0;
#pragma unroll
  for (int q = 0; q < kMedIpt; ++q)
    if (member(t + (int64_t)q * kMedThreads)) {
      mine |= 1u << q;
      ++m;
    }
  for (int64_t i = t + (int64_t)kMedIpt * kMedThreads; i < S.items;
       i += kMedThreads)
    if (member(i)) ++m;
  m = (int64_t)lane63(wave_incl((uint64_t)m, OpAdd(), (uint64_t)0));
  if (lane == 0) s_red[wv] = (uint64_t)m;
  __syncthreads();
  m = 0;
  for (int i = 0; i < kMedThreads / kWave; ++i) m += (int64_t)s_red[i];
  __syncthreads();
  if (t == 0) cnt[off] = m;
  for (int st = 0; st < nstat; ++st) {
    if (m == 0) {
      if (t == 0) med[st * mstride + off] = __builtin_nan("");
      continue;
    }
    uint64_t key[kMedIpt];
#pragma unroll
    for (int q = 0; q < kMedIpt; ++q)
      key[q] = ((mine >> q) & 1u) ? key_of(t + (int64_t)q * kMedThreads, st)
                                  : 0ull;
    // fn(key, is_member) for every item slot; whole waves take part
    auto each = [&](auto&& fn) {
#pragma unroll
      for (int q = 0; q < kMedIpt; ++q) fn(key[q], ((mine >> q) & 1u) != 0);
      for (int64_t i0 = (int64_t)kMedIpt * kMedThreads; i0 < S.items;
           i0 += kMedThreads) {
        const int64_t i = i0 + t;
        const bool ok = member(i);
        fn(ok ? key_of(i, st) : 0ull, ok);
      }
    };
    // smallest and largest key: the bits above the highest one in which
    // they differ are common to every member
    uint64_t lo = ~0ull, hi = 0;
    each([&](uint64_t k, bool ok) {
      if (!ok) return;
      lo = k < lo ? k : lo;
      hi = k > hi ? k : hi;
    });
    lo = lane63(wave_incl(
        lo, [](uint64_t a, uint64_t b) { return a < b ? a : b; },
        ~(uint64_t)0));
    hi = lane63(wave_incl(
        hi, [](uint64_t a, uint64_t b) { return a > b ? a : b; },
        (uint64_t)0));
    if (lane == 0) {
      s_red[wv] = lo;
      s_hist[0][wv * 2] = (uint32_t)hi;
      s_hist[0][wv * 2 + 1] = (uint32_t)(hi >> 32);
    }
    __syncthreads();
    lo = ~0ull;
    hi = 0;
    for (int i = 0; i < kMedThreads / kWave; ++i) {
      const uint64_t a = s_red[i];
      const uint64_t b = (uint64_t)s_hist[0][2 * i] |
                         ((uint64_t)s_hist[0][2 * i + 1] << 32);
      lo = a < lo ? a : lo;
      hi = b > hi ? b : hi;
    }
    __syncthreads();
    uint64_t res[2];
    if (lo == hi) {
      res[0] = res[1] = lo;
    } else {
      const int top = 63 - __clzll((long long)(lo ^ hi));
      const int s0 = (top / 8) * 8;
      uint64_t pre[2];
      int64_t rank[2] = {(m - 1) / 2, m / 2};
      pre[0] = pre[1] = s0 + 8 >= 64 ? 0ull : (lo >> (s0 + 8)) << (s0 + 8);
      for (int sh = s0; sh >= 0; sh -= 8) {
        for (int b = t; b < 512; b += kMedThreads) (&s_hist[0][0])[b] = 0;
        __syncthreads();
        const int hs = sh + 8;
        each([&](uint64_t k, bool ok) {
          const uint32_t dig = (uint32_t)(k >> sh) & 255u;
#pragma unroll
          for (int r = 0; r < 2; ++r) {
            const bool cand = ok && (hs >= 64 || (k >> hs) == (pre[r] >> hs));
            // one add per wave when its candidates share the digit (the
            // usual case in the high digits), else one per candidate
            const uint64_t act = __ballot(cand);
            if (act == 0) continue;
            const int ld = __ffsll((long long)act) - 1;
            const uint32_t d0 =
                (uint32_t)__builtin_amdgcn_readlane((int)dig, ld);
            if (__ballot(cand && dig == d0) == act) {
              if (lane == ld)
                atomicAdd(&s_hist[r][d0], (uint32_t)__popcll(act));
            } else if (cand) {
              atomicAdd(&s_hist[r][dig], 1u);
            }
          }
        });
        __syncthreads();
        if (t < 2 * kWave) {
          // wave r finds the digit that holds rank r
          const int r = t / kWave;
          uint32_t h[4], sum = 0;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            h[q] = s_hist[r][lane * 4 + q];
            sum += h[q];
          }
          const uint32_t incl = wave_incl(sum, OpAdd(), 0u);
          const uint64_t past = __ballot((int64_t)incl > rank[r]);
          const int ln = __ffsll((long long)past) - 1;
          if (lane == ln) {
            int64_t below = incl - sum;
            int dsel = lane * 4 + 3;
#pragma unroll
            for (int q = 3; q >= 0; --q)
              if (below + (int64_t)h[0] + (q > 0 ? h[1] : 0) +
                      (q > 1 ? h[2] : 0) + (q > 2 ? h[3] : 0) >
                  rank[r])
                dsel = lane * 4 + q;
            int64_t under = below;
            for (int q = 0; q < dsel - lane * 4; ++q) under += h[q];
            s_sel[2 * r] = (uint64_t)dsel;
            s_sel[2 * r + 1] = (uint64_t)under;
          }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          pre[r] |= s_sel[2 * r] << sh;
          rank[r] -= (int64_t)s_sel[2 * r + 1];
        }
        __syncthreads();
      }
      res[0] = pre[0];
      res[1] = pre[1];
    }
    if (t == 0) {
      const int64_t a = (int64_t)(res[0] ^ kSign);
      const int64_t b = (int64_t)(res[1] ^ kSign);
      med[st * mstride + off] = ((double)a + (double)b) / 2.0;
    }
  }
}

}  // namespace

extern "C" int chopper_views(const chopper_records* rec,
                             const int64_t* start_al, const int64_t* end_al,
                             const uint32_t* idx, int32_t depth,
                             const int64_t* gap, const chopper_markers* mk,
                             const chopper_rows* rows,
                             const chopper_view_spec* spec,
                             const chopper_view_out* out, void* scratch,
                             size_t* scratch_bytes, uint32_t* status,
                             void* stream) {
  if (!validate_records(rec) || !validate_markers(mk) || !mk || !rows ||
      !spec || !out || !scratch_bytes)
    return CHOPPER_EINVAL;
  const int64_t n = rec->n, nm = mk->n;
  const int P = spec->n_phases, O = spec->n_ops, NI = spec->n_iters;
  const int64_t cap = out->unit_cap;
  if (depth < 1 || depth > mk->depth || spec->iter_level < 0 ||
      spec->iter_level >= depth || spec->phase_level < 0 ||
      spec->phase_level >= depth || spec->op_level < 0 ||
      spec->op_level >= depth || P < 1 || P > kMaxPhases || O < 1 ||
      O > kMaxOps || NI < 0 || cap < 0 || cap * P >= ((int64_t)1 << 32))
    return CHOPPER_EINVAL;
  if (n > 0 && (!rec->cls || !start_al || !end_al || !idx || !gap))
    return CHOPPER_EINVAL;
  if (nm > 0 && (!mk->level || !mk->label)) return CHOPPER_EINVAL;
  if (!rows->level_offset || (rows->cap > 0 &&
      (!rows->path || !rows->kind || !rows->n || !rows->dur || !rows->gap ||
       !rows->ovl)))
    return CHOPPER_EINVAL;
  if (!out->n_units || !out->cls_med || !out->cls_cnt || !out->op_med ||
      !out->op_cnt || !out->iter_med || !out->iter_cnt ||
      (NI > 0 && !out->iter_max) ||
      (cap > 0 && (!out->unit_marker || !out->cls_tab || !out->op_tab ||
                   !out->busy)))
    return CHOPPER_EINVAL;
  const int64_t ntiles = ceil_div(nm, kRankTile);
  Scratch probe(nullptr);
  auto layout = [&](Scratch& sc, uint32_t*& tilecnt, uint32_t*& unit_of,
                    uint32_t*& total) {
    tilecnt = sc.take<uint32_t>(ntiles);
    unit_of = sc.take<uint32_t>(nm);
    total = sc.take<uint32_t>(1);
  };
  uint32_t *tilecnt, *unit_of, *total;
  layout(probe, tilecnt, unit_of, total);
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  layout(sc, tilecnt, unit_of, total);

  // units: the iteration markers numbered in marker order
  if (nm > 0) {
    CHOPPER_HIP(launch("view_units", k_view_count, dim3((unsigned)ntiles),
                       dim3(kRankThreads), s, mk->level, nm, spec->iter_level,
                       tilecnt));
    CHOPPER_HIP(launch("view_units", k_view_rank, dim3((unsigned)ntiles),
                       dim3(kRankThreads), s, mk->level, nm, spec->iter_level,
                       (const uint32_t*)tilecnt, cap, unit_of,
                       out->unit_marker, total, out->n_units, status));
  } else {
    CHOPPER_HIP(launch("view_units", k_view_zero, dim3(1), dim3(1), s, total,
                       out->n_units));
  }
  // cleared tables
  const int64_t ncls = cap * P * kViewClasses, nop = cap * P * O * 2;
  auto fill = [&](void* p, int64_t cnt, uint64_t v) -> int {
    if (cnt <= 0) return CHOPPER_OK;
    int64_t blocks = ceil_div(cnt, (int64_t)kBlock * 4);
    blocks = blocks < 4096 ? blocks : 4096;
    CHOPPER_HIP(launch("view_fill", k_view_fill, dim3((unsigned)blocks),
                       dim3(kBlock), s, (uint64_t*)p, cnt, v));
    return CHOPPER_OK;
  };
  if ((rc = fill(out->cls_tab, 3 * ncls, 0ull)) != CHOPPER_OK) return rc;
  if ((rc = fill(out->op_tab, 4 * nop, 0ull)) != CHOPPER_OK) return rc;
  if ((rc = fill(out->busy, cap, 0ull)) != CHOPPER_OK) return rc;
  if ((rc = fill(out->iter_max, NI, ~0ull)) != CHOPPER_OK) return rc;
  // class view and busy time
  if (n > 0 && nm > 0 && cap > 0) {
    CHOPPER_HIP(launch(
        "view_records", k_view_records,
        dim3((unsigned)ceil_div(n, (int64_t)kWaveTile * kWavesPerBlock)),
        dim3(kBlock), s, n, rec->cls, start_al, end_al, gap,
        idx + (int64_t)spec->iter_level * n,
        idx + (int64_t)spec->phase_level * n, mk->level, spec->iter_level,
        (const uint32_t*)unit_of, mk->label, nm, (const uint32_t*)total, cap,
        P, out->cls_tab, out->busy));
  }
  // operation view from the rows
  if (rows->cap > 0 && nm > 0 && cap > 0) {
    RowCols R{rows->level_offset, rows->path, rows->kind, rows->n,
              rows->dur, rows->gap, rows->ovl, rows->cap};
    CHOPPER_HIP(launch(
        "view_rows", k_view_rows,
        dim3((unsigned)ceil_div(rows->cap,
                                (int64_t)kWaveTile * kWavesPerBlock)),
        dim3(kBlock), s, R, spec->iter_level, spec->phase_level,
        spec->op_level, mk->level, (const uint32_t*)unit_of, mk->label, nm,
        (const uint32_t*)total, cap, P, O, out->op_tab));
  }
  if (NI > 0 && cap > 0)
    CHOPPER_HIP(launch("view_iter_max", k_view_iter_max,
                       grid_for(cap, kBlock), dim3(kBlock), s,
                       (const uint32_t*)total, cap,
                       (const uint32_t*)out->unit_marker, mk->label,
                       (const int64_t*)out->busy, NI, out->iter_max));
  MedArgs A{(const uint32_t*)total, cap, out->unit_marker, mk->label,
            spec->warmup, P, O, NI, out->cls_tab, out->op_tab,
            out->iter_max, out->cls_med, out->cls_cnt, out->op_med,
            out->op_cnt, out->iter_med, out->iter_cnt};
  CHOPPER_HIP(launch("view_medians", k_view_medians,
                     dim3((unsigned)(P * kViewClasses + P * O * 2 + 1)),
                     dim3(kMedThreads), s, A));
  return CHOPPER_OK;
}

}  // namespace chopper
