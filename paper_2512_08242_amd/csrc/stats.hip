// chopper_op_stats: overlap statistics and overhead breakdown of operations
// (Fig. gemm_overlap: overlap ratio against operation duration, their
// correlation, 25-75 % and min-max fills; Section VI duration breakdown,
// eqs. 6-10).
//
// The instances (compute rows of the operation level) are partitioned by
// (phase, operation) group; one 1024-thread block per group then adds the
// exact moments of (overlap ratio in Q30, duration) in 128-bit integers --
// integer sums do not depend on their order, so the derived doubles are the
// same IEEE operations on the same values as anywhere else -- and selects
// the quantiles of the ratio by radix, eight bits per pass.
#include "common.h"
#include "wave.h"

namespace chopper {

bool validate_markers(const chopper_markers* m);

namespace {

constexpr int kMaxGroups = 16 * 128;
constexpr int kStatT = 1024;
constexpr int kStats = 17;
typedef __int128 i128;
typedef unsigned __int128 u128;

struct StatArgs {
  const int64_t* level_offset;
  const uint32_t* path;
  const uint8_t* kind;
  const int64_t* dur;
  const int64_t* gap;
  const int64_t* ovl;
  const uint64_t* ctr;
  int64_t cap;
  int nc;
  int lv_phase, lv_op;
  const uint32_t* label;
  int64_t nm;
  int P, O;
};

__device__ inline void level_range(const StatArgs& A, int64_t& lo,
                                   int64_t& hi) {
  lo = A.level_offset[A.lv_op];
  hi = A.level_offset[A.lv_op + 1];
  if (hi > A.cap) hi = A.cap;
  if (lo > hi) lo = hi;
}

// group of an operation-level row, or kNone when it is no instance
__device__ inline uint32_t group_of(const StatArgs& A, int64_t r) {
  if (A.kind[r] != 0 || A.dur[r] <= 0) return kNone;
  const uint32_t mp = A.path[(int64_t)A.lv_phase * A.cap + r];
  const uint32_t mo = A.path[(int64_t)A.lv_op * A.cap + r];
  if ((int64_t)mp >= A.nm || (int64_t)mo >= A.nm) return kNone;
  const uint32_t p = A.label[mp], o = A.label[mo];
  if (p >= (uint32_t)A.P || o >= (uint32_t)A.O) return kNone;
  return p * (uint32_t)A.O + o;
}

__global__ void k_stats_clear(uint32_t* cnt, int G) {
  const int g = (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (g < G) cnt[g] = 0;
}

// group of every row and the instances per group
__global__ __launch_bounds__(kBlock) void k_stats_keys(StatArgs A,
                                                       uint32_t* key,
                                                       uint32_t* cnt) {
  __shared__ uint32_t s_h[kMaxGroups];
  const int G = A.P * A.O;
  for (int g = threadIdx.x; g < G; g += kBlock) s_h[g] = 0;
  __syncthreads();
  int64_t lo, hi;
  level_range(A, lo, hi);
  const int64_t r = lo + (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (r < hi) {
    const uint32_t g = group_of(A, r);
    key[r - lo] = g;
    if (g != kNone) atomicAdd(&s_h[g], 1u);
  }
  __syncthreads();
  for (int g = threadIdx.x; g < G; g += kBlock)
    if (s_h[g]) atomicAdd(&cnt[g], s_h[g]);
}

// group offsets (one block) and the fill cursors
__global__ __launch_bounds__(kStatT) void k_stats_offsets(const uint32_t* cnt,
                                                          int G, uint32_t* off,
                                                          uint32_t* cur) {
  __shared__ uint32_t s_w[kStatT / kWave];
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  uint32_t carry = 0;
  for (int b0 = 0; b0 < G; b0 += kStatT) {
    const int g = b0 + t;
    const uint32_t v = g < G ? cnt[g] : 0u;
    const uint32_t incl = wave_incl(v, OpAdd(), 0u);
    if (lane == kWave - 1) s_w[w] = incl;
    __syncthreads();
    uint32_t pre = carry, tot = carry;
    for (int q = 0; q < kStatT / kWave; ++q) {
      if (q < w) pre += s_w[q];
      tot += s_w[q];
    }
    if (g < G) {
      off[g] = pre + incl - v;
      cur[g] = pre + incl - v;
    }
    carry = tot;
    __syncthreads();
  }
  if (t == 0) off[G] = carry;
}

// rows into their group's slots (the order inside a group is immaterial:
// its sums are exact and its quantiles are order statistics)
__global__ void k_stats_scatter(StatArgs A, const uint32_t* key,
                                uint32_t* cur, uint32_t* list) {
  int64_t lo, hi;
  level_range(A, lo, hi);
  const int64_t r = lo + (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= hi) return;
  const uint32_t g = key[r - lo];
  if (g == kNone) return;
  list[atomicAdd(&cur[g], 1u)] = (uint32_t)r;
}

// nearest double to a 128-bit integer (round half to even): a magnitude
// below 2^63 converts directly; else its top 64 bits with every lower bit
// folded into the last one (below the double's precision there) convert
// and are scaled back exactly
__device__ inline double i128_to_double(i128 v) {
  const bool neg = v < 0;
  const u128 a = neg ? (u128)0 - (u128)v : (u128)v;
  double d;
  if ((a >> 63) == 0) {
    d = (double)(uint64_t)a;
  } else {
    const uint64_t hi64 = (uint64_t)(a >> 64);
    const int len = hi64 ? 128 - __clzll((long long)hi64) : 64;
    const int sh = len - 64;
    uint64_t top = (uint64_t)(a >> sh);
    if (sh > 0 && (a & (((u128)1 << sh) - 1)) != 0) top |= 1u;
    d = ldexp((double)top, sh);
  }
  return neg ? -d : d;
}

// block-wide sum of a 128-bit value (tree in LDS)
__device__ inline u128 block_sum_u128(u128 v, u128* s) {
  const int t = threadIdx.x;
  s[t] = v;
  __syncthreads();
  for (int d = kStatT / 2; d > 0; d >>= 1) {
    if (t < d) s[t] += s[t + d];
    __syncthreads();
  }
  const u128 r = s[0];
  __syncthreads();
  return r;
}

struct StatOut {
  double* out;
  int64_t* cnt;
  double freq_peak, tpt_peak;
  int have_f;
  double f_gemm[128];
};

__global__ __launch_bounds__(kStatT) void k_stats_group(
    StatArgs A, const uint32_t* off, const uint32_t* list, uint32_t* xs,
    StatOut S, uint32_t* status) {
  __shared__ u128 s_v[kStatT];
  __shared__ uint32_t s_hist[2][256];
  __shared__ uint32_t s_sel[4];
  const int t = threadIdx.x;
  const int G = A.P * A.O;
  const int g = blockIdx.x;
  const int64_t b = off[g], m = (int64_t)off[g + 1] - b;
  const double nan = __builtin_nan("");
  if (m == 0) {
    if (t < kStats) S.out[(int64_t)t * G + g] = nan;
    if (t == 0) S.cnt[g] = 0;
    return;
  }
  // exact moments; the ratio of every instance into xs
  u128 sx = 0, sy = 0, sxx = 0, syy = 0, sxy = 0;
  uint64_t cyc = 0, busy = 0, flops = 0;
  bool big = false;
  for (int64_t i = t; i < m; i += kStatT) {
    const uint32_t r = list[b + i];
    const uint64_t d = (uint64_t)A.dur[r];
    const uint64_t ov = (uint64_t)A.ovl[r];
    const uint64_t x = (ov << 30) / d;
    const uint64_t y = d + (uint64_t)A.gap[r];
    if (y >> 34) big = true;
    xs[b + i] = (uint32_t)x;
    sx += x;
    sy += y;
    sxx += (u128)x * x;
    syy += (u128)y * y;
    sxy += (u128)x * y;
    if (A.nc >= 16) {
      cyc += A.ctr[0 * A.cap + r];
      busy += A.ctr[1 * A.cap + r];
      flops += A.ctr[11 * A.cap + r];
    }
  }
  if (__ballot(big) != 0 && lane_id() == 0)
    atomicOr(status, CHOPPER_ST_RANGE);
  sx = block_sum_u128(sx, s_v);
  sy = block_sum_u128(sy, s_v);
  sxx = block_sum_u128(sxx, s_v);
  syy = block_sum_u128(syy, s_v);
  sxy = block_sum_u128(sxy, s_v);
  cyc = (uint64_t)block_sum_u128(cyc, s_v);
  busy = (uint64_t)block_sum_u128(busy, s_v);
  flops = (uint64_t)block_sum_u128(flops, s_v);
  // order statistics of the ratio: the smallest, v[(m-1)/4], v[(m-1)/2],
  // v[m/2], v[3(m-1)/4] and the largest, two ranks per radix selection
  const int64_t want[6] = {0, (m - 1) / 4, (m - 1) / 2, m / 2,
                           3 * (m - 1) / 4, m - 1};
  uint32_t got[6];
  for (int pair = 0; pair < 3; ++pair) {
    int64_t rank[2] = {want[2 * pair], want[2 * pair + 1]};
    uint32_t pre[2] = {0, 0};
    for (int sh = 24; sh >= 0; sh -= 8) {
      for (int q = t; q < 512; q += kStatT) (&s_hist[0][0])[q] = 0;
      __syncthreads();
      const int hs = sh + 8;
      for (int64_t i = t; i < m; i += kStatT) {
        const uint32_t k = xs[b + i];
        const uint32_t dig = (k >> sh) & 255u;
#pragma unroll
        for (int rr = 0; rr < 2; ++rr)
          if (hs >= 32 || (k >> hs) == (pre[rr] >> hs))
            atomicAdd(&s_hist[rr][dig], 1u);
      }
      __syncthreads();
      if (t < 2 * kWave) {
        const int rr = t / kWave, lane = lane_id();
        uint32_t h[4], sum = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          h[q] = s_hist[rr][lane * 4 + q];
          sum += h[q];
        }
        const uint32_t incl = wave_incl(sum, OpAdd(), 0u);
        const uint64_t past = __ballot((int64_t)incl > rank[rr]);
        const int ln = __ffsll((long long)past) - 1;
        if (lane == ln) {
          int64_t under = incl - sum;
          int dsel = lane * 4 + 3;
          for (int q = 0; q < 4; ++q) {
            if (under + (int64_t)h[q] > rank[rr]) {
              dsel = lane * 4 + q;
              break;
            }
            under += h[q];
          }
          s_sel[2 * rr] = (uint32_t)dsel;
          s_sel[2 * rr + 1] = (uint32_t)under;   // candidates below it
        }
      }
      __syncthreads();
#pragma unroll
      for (int rr = 0; rr < 2; ++rr) {
        pre[rr] |= s_sel[2 * rr] << sh;
        rank[rr] -= (int64_t)s_sel[2 * rr + 1];
      }
      __syncthreads();
    }
    got[2 * pair] = pre[0];
    got[2 * pair + 1] = pre[1];
  }
  if (t != 0) return;
  // the derived values, in the same IEEE operations as their definition
  double* o = S.out;
  for (int k = 0; k < kStats; ++k) o[(int64_t)k * G + g] = nan;
  S.cnt[g] = m;
  const i128 im = (i128)m;
  const i128 cov = im * (i128)sxy - (i128)sx * (i128)sy;
  const i128 vx = im * (i128)sxx - (i128)sx * (i128)sx;
  const i128 vy = im * (i128)syy - (i128)sy * (i128)sy;
  const double dm = (double)m;
  if (m >= 2 && vx != 0 && vy != 0)
    o[0 * G + g] = i128_to_double(cov) /
                   sqrt(i128_to_double(vx) * i128_to_double(vy));
  double slope = nan, a = nan;
  if (vx != 0) {
    slope = i128_to_double(cov) / i128_to_double(vx);
    a = (i128_to_double((i128)sy) - slope * i128_to_double((i128)sx)) / dm;
  }
  o[1 * G + g] = slope;
  o[2 * G + g] = a;
  const double d0 = a, d50 = a + slope * 536870912.0;
  o[3 * G + g] = d0;
  o[4 * G + g] = d50;
  const double q = 1.0 / 1073741824.0;
  o[5 * G + g] = (double)got[0] * q;
  o[6 * G + g] = (double)got[1] * q;
  o[7 * G + g] = ((double)got[2] + (double)got[3]) / 2.0 * q;
  o[8 * G + g] = (double)got[4] * q;
  o[9 * G + g] = (double)got[5] * q;
  const double dact = i128_to_double((i128)sy) / dm;
  o[10 * G + g] = dact;
  const double ovr_ov = d50 / d0;
  o[14 * G + g] = ovr_ov;
  const double fg = S.have_f ? S.f_gemm[g % A.O] : nan;
  if (A.nc >= 16) {
    const double dpeak = (double)cyc * 1000.0 / S.freq_peak / dm;
    o[11 * G + g] = dpeak;
    o[12 * G + g] = 1.0 / ((double)busy / (double)cyc);
    o[13 * G + g] = ((double)flops / dm) / fg;
    o[15 * G + g] = dact / dpeak / ovr_ov;
  }
  o[16 * G + g] = fg / S.tpt_peak;
}

}  // namespace

extern "C" int chopper_op_stats(const chopper_rows* rows, int32_t depth,
                                int32_t n_counters,
                                const chopper_markers* mk,
                                const chopper_stats_spec* spec, double* out,
                                int64_t* cnt, void* scratch,
                                size_t* scratch_bytes, uint32_t* status,
                                void* stream) {
  if (!rows || !spec || !mk || !validate_markers(mk) || !scratch_bytes ||
      !out || !cnt)
    return CHOPPER_EINVAL;
  const int P = spec->n_phases, O = spec->n_ops;
  if (depth < 1 || depth > mk->depth || spec->phase_level < 0 ||
      spec->phase_level >= depth || spec->op_level < 0 ||
      spec->op_level >= depth || P < 1 || P > 16 || O < 1 || O > 128 ||
      n_counters < 0 || n_counters > 16 || rows->cap < 0 ||
      rows->cap >= (int64_t)0xFFFFFFFF || !rows->level_offset)
    return CHOPPER_EINVAL;
  if (rows->cap > 0 && (!rows->path || !rows->kind || !rows->dur ||
                        !rows->gap || !rows->ovl ||
                        (n_counters > 0 && !rows->ctr)))
    return CHOPPER_EINVAL;
  if (mk->n > 0 && !mk->label) return CHOPPER_EINVAL;
  const int G = P * O;
  const int64_t cap = rows->cap;
  auto layout = [&](Scratch& sc, uint32_t*& key, uint32_t*& gcnt,
                    uint32_t*& off, uint32_t*& cur, uint32_t*& list,
                    uint32_t*& xs) {
    key = sc.take<uint32_t>(cap);
    gcnt = sc.take<uint32_t>(G);
    off = sc.take<uint32_t>(G + 1);
    cur = sc.take<uint32_t>(G);
    list = sc.take<uint32_t>(cap);
    xs = sc.take<uint32_t>(cap);
  };
  uint32_t *key, *gcnt, *off, *cur, *list, *xs;
  Scratch probe(nullptr);
  layout(probe, key, gcnt, off, cur, list, xs);
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  layout(sc, key, gcnt, off, cur, list, xs);
  StatArgs A{rows->level_offset, rows->path, rows->kind, rows->dur,
             rows->gap, rows->ovl, rows->ctr, cap, n_counters,
             spec->phase_level, spec->op_level, mk->label, mk->n, P, O};
  StatOut S{out, cnt, spec->freq_peak_mhz, spec->tpt_peak,
            spec->f_gemm != nullptr, {0}};
  for (int o = 0; o < O && spec->f_gemm; ++o) S.f_gemm[o] = spec->f_gemm[o];
  CHOPPER_HIP(launch("stats_clear", k_stats_clear, grid_for(G, kBlock),
                     dim3(kBlock), s, gcnt, G));
  const unsigned rb = (unsigned)ceil_div(cap > 0 ? cap : 1, (int64_t)kBlock);
  CHOPPER_HIP(launch("stats_keys", k_stats_keys, dim3(rb), dim3(kBlock), s,
                     A, key, gcnt));
  CHOPPER_HIP(launch("stats_offsets", k_stats_offsets, dim3(1),
                     dim3(kStatT), s, (const uint32_t*)gcnt, G, off, cur));
  CHOPPER_HIP(launch("stats_scatter", k_stats_scatter, dim3(rb), dim3(kBlock),
                     s, A, (const uint32_t*)key, cur, list));
  CHOPPER_HIP(launch("stats_group", k_stats_group, dim3((unsigned)G),
                     dim3(kStatT), s, A, (const uint32_t*)off,
                     (const uint32_t*)list, xs, S, status));
  return CHOPPER_OK;
}

}  // namespace chopper
