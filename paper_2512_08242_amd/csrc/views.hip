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
// one wave reduction per class and field feeds one atomic add.  The
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
constexpr int kMedIpt = 16;      // items per thread of a group's pass
constexpr uint64_t kSign = 1ull << 63;

__global__ void k_view_fill(uint64_t* p, int64_t n, uint64_t v) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

__global__ void k_view_zero(uint32_t* p) { *p = 0; }

__global__ void k_view_flags(int64_t nm, const uint8_t* level, int iter_level,
                             uint32_t* flags) {
  const int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (m < nm) flags[m] = level[m] == (uint8_t)iter_level ? 1u : 0u;
}

// unit_marker of every unit that fits and the unit count
__global__ void k_view_units(int64_t nm, const uint32_t* flags,
                             const uint32_t* unit_of, const uint32_t* total,
                             int64_t cap, uint32_t* unit_marker,
                             int64_t* n_units, uint32_t* status) {
  const int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (m == 0) {
    *n_units = (int64_t)*total;
    if ((int64_t)*total > cap) atomicOr(status, CHOPPER_ST_ROWS_OVERFLOW);
  }
  if (m < nm && flags[m] && (int64_t)unit_of[m] < cap)
    unit_marker[unit_of[m]] = (uint32_t)m;
}

__device__ inline uint64_t wave_sum(uint64_t v) {
  return lane63(wave_incl(v, OpAdd(), (uint64_t)0));
}

// Value of a per-lane item array at a lane-varying index (a select chain
// keeps the array in registers).
template <typename T>
__device__ inline T pick(const T (&a)[kTileIpt], int j) {
  T r = a[0];
#pragma unroll
  for (int q = 1; q < kTileIpt; ++q)
    if (q == j) r = a[q];
  return r;
}

// The key of the first pending item of the first lane that has one; every
// lane then marks its pending items with that key in `hit`.  Returns false
// when no item is pending.
__device__ inline bool next_group(uint32_t pend,
                                  const uint32_t (&key)[kTileIpt],
                                  uint32_t& k, uint32_t& hit) {
  const uint64_t act = __ballot(pend != 0u);
  if (act == 0) return false;
  const int leader = __ffsll((long long)act) - 1;
  const uint32_t mine = pend ? pick(key, __ffs((int)pend) - 1) : 0u;
  k = (uint32_t)__builtin_amdgcn_readlane((int)mine, leader);
  hit = 0;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j)
    if (((pend >> j) & 1u) && key[j] == k) hit |= 1u << j;
  return true;
}

// Class view and busy time from the records; one wave per kWaveTile records.
__global__ __launch_bounds__(kBlock) void k_view_records(
    int64_t n, const uint8_t* cls, const int64_t* start, const int64_t* end,
    const int64_t* gap, const uint32_t* idx_iter, const uint32_t* idx_phase,
    const uint32_t* unit_of, const uint32_t* label, int64_t nm,
    const uint32_t* units, int64_t cap, int P, uint64_t* cls_tab,
    int64_t* busy) {
  const int lane = lane_id();
  const int64_t w =
      (int64_t)blockIdx.x * kWavesPerBlock + (int64_t)(threadIdx.x / kWave);
  const int64_t base = w * kWaveTile;
  if (base >= n) return;
  int64_t ucap = (int64_t)*units;
  ucap = ucap < cap ? ucap : cap;
  uint32_t ukey[kTileIpt], key[kTileIpt], c[kTileIpt];
  uint64_t d[kTileIpt], g[kTileIpt];
  uint32_t pb = 0, pc = 0;   // pending items: busy, class view
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const int64_t r = base + (int64_t)j * kWave + lane;
    const bool valid = r < n;
    const uint32_t mi = valid ? idx_iter[r] : kNone;
    uint32_t u = (int64_t)mi < nm ? unit_of[mi] : kNone;
    if ((int64_t)u >= ucap) u = kNone;
    const uint32_t mp = u != kNone ? idx_phase[r] : kNone;
    const uint32_t p = (int64_t)mp < nm ? label[mp] : kNone;
    c[j] = valid ? (uint32_t)cls[r] : 255u;
    d[j] = valid ? (uint64_t)(end[r] - start[r]) : 0ull;
    g[j] = valid ? (uint64_t)gap[r] : 0ull;
    ukey[j] = u;
    key[j] = (u != kNone && p < (uint32_t)P && c[j] < (uint32_t)kViewClasses)
                 ? u * (uint32_t)P + p : kNone;
    if (u != kNone && !kind_of(c[j])) pb |= 1u << j;
    if (key[j] != kNone) pc |= 1u << j;
  }
  uint32_t k, hit;
  // busy: compute records by unit
  while (next_group(pb, ukey, k, hit)) {
    uint64_t x = 0;
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j)
      if ((hit >> j) & 1u) x += d[j] + g[j];
    x = wave_sum(x);
    if (lane == 0) atomicAdd((unsigned long long*)&busy[k], x);
    pb &= ~hit;
  }
  // class view by (unit, phase), one class at a time
  const int64_t ncls = cap * P * kViewClasses;
  while (next_group(pc, key, k, hit)) {
    for (uint32_t cc = 0; cc < (uint32_t)kViewClasses; ++cc) {
      uint64_t xn = 0, xd = 0, xg = 0;
#pragma unroll
      for (int j = 0; j < kTileIpt; ++j)
        if (((hit >> j) & 1u) && c[j] == cc) {
          xn += 1;
          xd += d[j];
          xg += g[j];
        }
      if (__ballot(xn != 0) == 0) continue;
      xn = wave_sum(xn);
      xd = wave_sum(xd);
      xg = wave_sum(xg);
      const int64_t e = (int64_t)k * kViewClasses + cc;
      if (lane == 0) {
        atomicAdd((unsigned long long*)&cls_tab[e], xn);
        atomicAdd((unsigned long long*)&cls_tab[ncls + e], xd);
        atomicAdd((unsigned long long*)&cls_tab[2 * ncls + e], xg);
      }
    }
    pc &= ~hit;
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
    RowCols R, int lv_iter, int lv_phase, int lv_op, const uint32_t* unit_of,
    const uint32_t* label, int64_t nm, const uint32_t* units, int64_t cap,
    int P, int O, uint64_t* op_tab) {
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
  uint32_t key[kTileIpt], sub[kTileIpt];
  uint64_t v[kTileIpt][4];
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
    uint32_t u = (int64_t)p0 < nm ? unit_of[p0] : kNone;
    if ((int64_t)u >= ucap) u = kNone;
    const uint32_t ph = (int64_t)p1 < nm ? label[p1] : kNone;
    const uint32_t op = (int64_t)p3 < nm ? label[p3] : kNone;
    key[j] = (u != kNone && ph < (uint32_t)P && op < (uint32_t)O)
                 ? u * (uint32_t)P + ph : kNone;
    sub[j] = key[j] != kNone ? op * 2u + (R.kind[row] ? 1u : 0u) : 0u;
    v[j][0] = key[j] != kNone ? R.n[row] : 0ull;
    v[j][1] = key[j] != kNone ? (uint64_t)R.dur[row] : 0ull;
    v[j][2] = key[j] != kNone ? (uint64_t)R.gap[row] : 0ull;
    v[j][3] = key[j] != kNone ? (uint64_t)R.ovl[row] : 0ull;
    if (key[j] != kNone) pend |= 1u << j;
  }
  const int64_t nop = cap * P * O * 2;
  uint32_t k, hit;
  while (next_group(pend, key, k, hit)) {
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
    const int64_t row0 = (int64_t)k * O * 2;
    for (int e = lane; e < ne; e += kWave) {
      if (tab[e * 4] == 0) continue;
#pragma unroll
      for (int f = 0; f < 4; ++f)
        atomicAdd((unsigned long long*)&op_tab[f * nop + row0 + e],
                  tab[e * 4 + f]);
    }
    wave_sync();
    pend &= ~hit;
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

__device__ inline int64_t block_sum_i64(int64_t v, int64_t* s_red) {
  const int lane = lane_id(), w = (int)(threadIdx.x / kWave);
  v = (int64_t)wave_sum((uint64_t)v);
  if (lane == 0) s_red[w] = v;
  __syncthreads();
  int64_t t = 0;
  for (int i = 0; i < kMedThreads / kWave; ++i) t += s_red[i];
  __syncthreads();
  return t;
}

__device__ inline uint64_t block_or_u64(uint64_t v, uint64_t* s_red) {
  const int lane = lane_id(), w = (int)(threadIdx.x / kWave);
  v = lane63(wave_incl(v, [](uint64_t a, uint64_t b) { return a | b; },
                       (uint64_t)0));
  if (lane == 0) s_red[w] = v;
  __syncthreads();
  uint64_t t = 0;
  for (int i = 0; i < kMedThreads / kWave; ++i) t |= s_red[i];
  __syncthreads();
  return t;
}

__global__ __launch_bounds__(kMedThreads) void k_view_medians(MedArgs A) {
  __shared__ uint32_t s_hist[2][256];
  __shared__ uint64_t s_red[kMedThreads / kWave];
  __shared__ uint64_t s_sel[4];
  const int t = (int)threadIdx.x;
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
    const int64_t col = A.cap * ncg;
    S = MedSrc{A.cls_tab + gi, A.cls_tab + col + gi, A.cls_tab + 2 * col + gi,
               ncg, U};
    med = A.cls_med;
    cnt = A.cls_cnt;
    off = gi;
    mstride = ncg;
    nstat = 3;
  } else if (gi < ncg + nog) {
    const int64_t o = gi - ncg, col = A.cap * nog;
    S = MedSrc{A.op_tab + o, A.op_tab + col + o, A.op_tab + 2 * col + o, nog,
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
  auto value = [&](int64_t i, int st) -> uint64_t {
    const uint64_t d = S.d[i * S.stride];
    if (st == 0) return d;
    const uint64_t g = S.g[i * S.stride];
    return st == 1 ? g : d + g;
  };
  // membership of this thread's first kMedIpt items, kept as bits
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
  m = block_sum_i64(m, (int64_t*)s_red);
  if (t == 0) cnt[off] = m;
  auto is_member = [&](int64_t q, int64_t i) -> bool {
    return q < kMedIpt ? ((mine >> q) & 1u) != 0 : member(i);
  };
  const int64_t nq = (S.items + kMedThreads - 1) / kMedThreads;
  for (int st = 0; st < nstat; ++st) {
    if (m == 0) {
      if (t == 0) med[st * mstride + off] = __builtin_nan("");
      continue;
    }
    // highest bit in which the members' keys differ from the first one's
    uint64_t first = 0, diff = 0;
    bool have = false;
    for (int64_t q = 0; q < nq; ++q) {
      const int64_t i = t + q * kMedThreads;
      if (i < S.items && is_member(q, i)) {
        first = value(i, st) ^ kSign;
        have = true;
        break;
      }
    }
    // a common reference: the key of the first member of the lowest thread
    // that holds one
    {
      const uint64_t cand = have ? (uint64_t)t : ~0ull;
      const int lane = lane_id(), w = t / kWave;
      uint64_t mn = lane63(wave_incl(
          cand, [](uint64_t a, uint64_t b) { return a < b ? a : b; },
          ~(uint64_t)0));
      if (lane == 0) s_red[w] = mn;
      __syncthreads();
      uint64_t best = ~0ull;
      for (int i = 0; i < kMedThreads / kWave; ++i)
        best = s_red[i] < best ? s_red[i] : best;
      __syncthreads();
      if ((uint64_t)t == best) s_sel[0] = first;
      __syncthreads();
      first = s_sel[0];
      __syncthreads();
    }
    for (int64_t q = 0; q < nq; ++q) {
      const int64_t i = t + q * kMedThreads;
      if (i < S.items && is_member(q, i))
        diff |= (value(i, st) ^ kSign) ^ first;
    }
    diff = block_or_u64(diff, s_red);
    uint64_t res[2];
    if (diff == 0) {
      res[0] = res[1] = first;
    } else {
      const int top = 63 - __clzll((long long)diff);
      const int s0 = (top / 8) * 8;
      // candidates share the bits above s0 + 8 with `first`
      uint64_t pre[2];
      int64_t rank[2] = {(m - 1) / 2, m / 2};
      pre[0] = pre[1] = s0 + 8 >= 64 ? 0ull : (first >> (s0 + 8)) << (s0 + 8);
      for (int sh = s0; sh >= 0; sh -= 8) {
        for (int b = t; b < 512; b += kMedThreads) (&s_hist[0][0])[b] = 0;
        __syncthreads();
        const int hs = sh + 8;
        for (int64_t q = 0; q < nq; ++q) {
          const int64_t i = t + q * kMedThreads;
          if (!(i < S.items && is_member(q, i))) continue;
          const uint64_t key = value(i, st) ^ kSign;
          const uint32_t dig = (uint32_t)(key >> sh) & 255u;
#pragma unroll
          for (int r = 0; r < 2; ++r)
            if (hs >= 64 || (key >> hs) == (pre[r] >> hs))
              atomicAdd(&s_hist[r][dig], 1u);
        }
        __syncthreads();
        if (t < 2 * kWave) {
          // wave r finds the digit holding rank[r]
          const int r = t / kWave, lane = lane_id();
          uint32_t h[4], sum = 0;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            h[q] = s_hist[r][lane * 4 + q];
            sum += h[q];
          }
          const uint32_t incl = wave_incl(sum, OpAdd(), 0u);
          const uint32_t excl = incl - sum;
          const uint64_t past = __ballot((int64_t)incl > rank[r]);
          const int ln = __ffsll((long long)past) - 1;
          if (lane == ln) {
            int64_t below = excl;
            int dsel = lane * 4;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
              if (below + h[q] > rank[r]) {
                dsel = lane * 4 + q;
                break;
              }
              below += h[q];
            }
            s_sel[2 * r] = (uint64_t)dsel;
            s_sel[2 * r + 1] = (uint64_t)below;
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
      const int64_t lo = (int64_t)(res[0] ^ kSign);
      const int64_t hi = (int64_t)(res[1] ^ kSign);
      med[st * mstride + off] = ((double)lo + (double)hi) / 2.0;
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
  Scratch probe(nullptr);
  auto layout = [&](Scratch& sc, uint32_t*& flags, uint32_t*& unit_of,
                    uint32_t*& tmp, uint32_t*& total) {
    flags = sc.take<uint32_t>(nm);
    unit_of = sc.take<uint32_t>(nm);
    tmp = sc.take<uint32_t>(scan_scratch_elems(nm));
    total = sc.take<uint32_t>(1);
  };
  uint32_t *flags, *unit_of, *tmp, *total;
  layout(probe, flags, unit_of, tmp, total);
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  layout(sc, flags, unit_of, tmp, total);

  // units
  if (nm > 0) {
    CHOPPER_HIP(launch("view_flags", k_view_flags, grid_for(nm, kBlock),
                       dim3(kBlock), s, nm, mk->level, spec->iter_level,
                       flags));
    CHOPPER_HIP(exclusive_scan<uint32_t>(flags, unit_of, nm, tmp, total, s));
  } else {
    CHOPPER_HIP(launch("view_units", k_view_zero, dim3(1), dim3(1), s, total));
  }
  CHOPPER_HIP(launch("view_units", k_view_units,
                     grid_for(nm > 0 ? nm : 1, kBlock), dim3(kBlock), s, nm,
                     (const uint32_t*)flags, (const uint32_t*)unit_of,
                     (const uint32_t*)total, cap, out->unit_marker,
                     out->n_units, status));
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
        idx + (int64_t)spec->phase_level * n, (const uint32_t*)unit_of,
        mk->label, nm, (const uint32_t*)total, cap, P, out->cls_tab,
        out->busy));
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
        spec->op_level, (const uint32_t*)unit_of, mk->label, nm,
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
