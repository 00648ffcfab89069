// chopper_op_stats: overlap statistics and overhead breakdown of operations
// (Fig. gemm_overlap: overlap ratio against operation duration, their
// correlation, 25-75 % and min-max fills; Section VI duration breakdown,
// eqs. 6-10).
//
// The instances (compute rows of the operation level) are partitioned by
// (phase, operation) group into compact columns of the overlap ratio (Q30)
// and the time (the grouping pass adds the three counters of every group in
// LDS on the way).  Blocks of 8192 instances of one group then
// add the exact moments in 64-bit words (halves of the products that would
// overflow) -- integer sums do not depend on their order, so the derived
// doubles are the same IEEE operations on the same values as anywhere else
// -- and build the histograms of a radix selection of six order statistics
// of the ratio per group, eight bits per pass, all groups at once.
#include "common.h"
#include "sort.h"
#include "wave.h"

namespace chopper {

bool validate_markers(const chopper_markers* m);

namespace {

constexpr int kMaxGroups = 16 * 128;
constexpr int kStatT = 1024;
constexpr int kStatIpt = 8;
constexpr int kRowSpan = kStatT * kStatIpt;   // rows per block
constexpr int kChunk = kStatT * kStatIpt;     // instances per block
constexpr int kRanks = 6;                     // order statistics per group
constexpr int kSums = 8;                      // exact moment words per group
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

// add 1 for every active lane to h[bin] and return the lane's slot among
// the adds (the old value plus its rank): one LDS atomic per wave when the
// active lanes share the bin, else one per lane
__device__ inline uint32_t lds_claim(uint32_t* h, uint32_t bin, bool act) {
  const uint64_t m = __ballot(act);
  if (m == 0) return 0;
  const int ld = __ffsll((long long)m) - 1;
  const uint32_t b0 = (uint32_t)__builtin_amdgcn_readlane((int)bin, ld);
  if (__ballot(act && bin == b0) == m) {
    uint32_t base = 0;
    if (lane_id() == ld) base = atomicAdd(&h[b0], (uint32_t)__popcll(m));
    base = (uint32_t)__builtin_amdgcn_readlane((int)base, ld);
    return base + lanes_below(m);
  }
  return act ? atomicAdd(&h[bin], 1u) : 0u;
}

__global__ void k_stats_clear_cdf(int64_t NGG, uint32_t* cnt,
                                  uint64_t* ymin) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < NGG) {
    cnt[i] = 0;
    ymin[i] = ~0ull;
  }
}

__global__ void k_stats_clear(uint32_t* cnt, int G, uint32_t* hist,
                              int64_t nh, uint64_t* csum) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < G) cnt[i] = 0;
  if (i < 3 * (int64_t)G) csum[i] = 0;
  if (i < nh) hist[i] = 0;
}

// group of every row of the operation level (kNone when it is no
// instance: not a compute row, zero length, or a label out of range) and
// the instances per group
__global__ __launch_bounds__(kStatT) void k_stats_keys(StatArgs A,
                                                       uint32_t* key,
                                                       uint32_t* cnt,
                                                       uint64_t* csum) {
  __shared__ uint32_t s_h[kMaxGroups];
  __shared__ uint64_t s_cs[3][kMaxGroups];   // counter sums (wrap mod 2^64)
  const int G = A.P * A.O;
  const bool ctr = A.nc >= 16;
  for (int g = threadIdx.x; g < G; g += kStatT) {
    s_h[g] = 0;
    s_cs[0][g] = s_cs[1][g] = s_cs[2][g] = 0;
  }
  __syncthreads();
  int64_t lo, hi;
  level_range(A, lo, hi);
  const int64_t r0 = lo + (int64_t)blockIdx.x * kRowSpan + threadIdx.x;
  // the rows' fields of all eight rows in flight at once, then the labels
  uint8_t kd[kStatIpt];
  int64_t du[kStatIpt];
  uint32_t mp[kStatIpt], mo[kStatIpt];
#pragma unroll
  for (int k = 0; k < kStatIpt; ++k) {
    const int64_t r = r0 + (int64_t)k * kStatT;
    const bool ok = r < hi;
    kd[k] = ok ? A.kind[r] : (uint8_t)1;
    du[k] = ok ? A.dur[r] : 0;
    mp[k] = ok ? A.path[(int64_t)A.lv_phase * A.cap + r] : kNone;
    mo[k] = ok ? A.path[(int64_t)A.lv_op * A.cap + r] : kNone;
  }
#pragma unroll
  for (int k = 0; k < kStatIpt; ++k) {
    const int64_t r = r0 + (int64_t)k * kStatT;
    uint32_t g = kNone;
    if (kd[k] == 0 && du[k] > 0 && (int64_t)mp[k] < A.nm &&
        (int64_t)mo[k] < A.nm) {
      const uint32_t p = A.label[mp[k]], o = A.label[mo[k]];
      if (p < (uint32_t)A.P && o < (uint32_t)A.O) g = p * (uint32_t)A.O + o;
    }
    if (r < hi) key[r - lo] = g;
    lds_claim(s_h, g, g != kNone);
    // GPU cycles, MFMA-busy cycles and FLOPs of the instance (eqs. 7, 8, 10)
    if (ctr && g != kNone) {
      atomicAdd((unsigned long long*)&s_cs[0][g],
                (unsigned long long)A.ctr[0 * A.cap + r]);
      atomicAdd((unsigned long long*)&s_cs[1][g],
                (unsigned long long)A.ctr[1 * A.cap + r]);
      atomicAdd((unsigned long long*)&s_cs[2][g],
                (unsigned long long)A.ctr[11 * A.cap + r]);
    }
  }
  __syncthreads();
  for (int g = threadIdx.x; g < G; g += kStatT)
    if (s_h[g]) {
      atomicAdd(&cnt[g], s_h[g]);
      if (ctr)
        for (int f = 0; f < 3; ++f)
          atomicAdd((unsigned long long*)&csum[3 * g + f],
                    (unsigned long long)s_cs[f][g]);
    }
}

// group offsets, fill cursors, chunk offsets and the ranks to select (one
// block)
__global__ __launch_bounds__(kStatT) void k_stats_offsets(
    const uint32_t* cnt, int G, uint32_t* off, uint32_t* cur, uint32_t* coff,
    uint32_t* spre, int64_t* srank) {
  __shared__ uint32_t s_w[2][kStatT / kWave];
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  uint32_t carry = 0, ccarry = 0;
  for (int b0 = 0; b0 < G; b0 += kStatT) {
    const int g = b0 + t;
    const uint32_t v = g < G ? cnt[g] : 0u;
    const uint32_t c = (uint32_t)ceil_div(v, kChunk);
    const uint32_t incl = wave_incl(v, OpAdd(), 0u);
    const uint32_t cincl = wave_incl(c, OpAdd(), 0u);
    if (lane == kWave - 1) {
      s_w[0][w] = incl;
      s_w[1][w] = cincl;
    }
    __syncthreads();
    uint32_t pre = carry, tot = carry, cpre = ccarry, ctot = ccarry;
    for (int q = 0; q < kStatT / kWave; ++q) {
      if (q < w) {
        pre += s_w[0][q];
        cpre += s_w[1][q];
      }
      tot += s_w[0][q];
      ctot += s_w[1][q];
    }
    if (g < G) {
      off[g] = pre + incl - v;
      cur[g] = pre + incl - v;
      coff[g] = cpre + cincl - c;
      // v[0], v[(m-1)/4], v[(m-1)/2], v[m/2], v[3(m-1)/4], v[m-1]
      const int64_t m = v;
      const int64_t want[kRanks] = {0, (m - 1) / 4, (m - 1) / 2, m / 2,
                                    3 * (m - 1) / 4, m - 1};
#pragma unroll
      for (int r = 0; r < kRanks; ++r) {
        spre[g * kRanks + r] = 0;
        srank[g * kRanks + r] = want[r];
      }
    }
    carry = tot;
    ccarry = ctot;
    __syncthreads();
  }
  if (t == 0) {
    off[G] = carry;
    coff[G] = ccarry;
  }
}

// every instance into its group's slots with its ratio x (Q30), its time y
// and three counters: a block claims its slots of a group with one atomic
// (the order inside a group is immaterial: sums are exact and quantiles are
// order statistics)
__global__ __launch_bounds__(kStatT) void k_stats_scatter(
    StatArgs A, const uint32_t* key, uint32_t* cur, uint32_t* xs,
    uint64_t* ys, uint32_t* status) {
  __shared__ uint32_t s_n[kMaxGroups];
  __shared__ uint32_t s_base[kMaxGroups];
  const int G = A.P * A.O;
  for (int g = threadIdx.x; g < G; g += kStatT) s_n[g] = 0;
  __syncthreads();
  int64_t lo, hi;
  level_range(A, lo, hi);
  const int64_t r0 = lo + (int64_t)blockIdx.x * kRowSpan + threadIdx.x;
  uint32_t g[kStatIpt], slot[kStatIpt];
  int64_t du[kStatIpt], ol[kStatIpt], gp[kStatIpt];
#pragma unroll
  for (int k = 0; k < kStatIpt; ++k) {
    const int64_t r = r0 + (int64_t)k * kStatT;
    const bool ok = r < hi;
    g[k] = ok ? key[r - lo] : kNone;
    du[k] = ok ? A.dur[r] : 1;
    ol[k] = ok ? A.ovl[r] : 0;
    gp[k] = ok ? A.gap[r] : 0;
  }
#pragma unroll
  for (int k = 0; k < kStatIpt; ++k)
    slot[k] = lds_claim(s_n, g[k], g[k] != kNone);
  __syncthreads();
  for (int q = threadIdx.x; q < G; q += kStatT)
    if (s_n[q]) s_base[q] = atomicAdd(&cur[q], s_n[q]);
  __syncthreads();
  bool big = false;
#pragma unroll
  for (int k = 0; k < kStatIpt; ++k) {
    if (g[k] == kNone) continue;
    const uint64_t d = (uint64_t)du[k];
    const uint64_t ov = (uint64_t)ol[k];
    const uint64_t y = d + (uint64_t)gp[k];
    const uint64_t x = (ov << 30) / d;
    if ((y >> 34) != 0 || x > (1ull << 30)) big = true;
    const uint32_t pos = s_base[g[k]] + slot[k];
    xs[pos] = (uint32_t)x;
    ys[pos] = y;
  }
  if (__ballot(big) != 0 && lane_id() == 0)
    atomicOr(status, CHOPPER_ST_RANGE);
}

// the group and chunk of this block (false past the last chunk)
__device__ inline bool chunk_of(const uint32_t* coff, const uint32_t* off,
                                int G, int64_t& b, int64_t& e, int& g) {
  const uint32_t c = blockIdx.x;
  if (c >= coff[G]) return false;
  int lo = 0, hi = G;        // the last g with coff[g] <= c
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (coff[mid] <= c) lo = mid;
    else hi = mid;
  }
  g = lo;
  b = (int64_t)off[g] + (int64_t)(c - coff[g]) * kChunk;
  e = b + kChunk;
  if (e > (int64_t)off[g + 1]) e = off[g + 1];
  return true;
}

// sum of v over the block into s_part (kSums words), exact in 64 bits
__device__ inline void block_sums(uint64_t (&v)[kSums],
                                  uint64_t (*s_w)[kSums], uint64_t* dst) {
  const int w = threadIdx.x / kWave;
#pragma unroll
  for (int k = 0; k < kSums; ++k) {
    const uint64_t s = lane63(wave_incl(v[k], OpAdd(), (uint64_t)0));
    if (lane_id() == 0) s_w[w][k] = s;
  }
  __syncthreads();
  if (threadIdx.x < kSums) {
    uint64_t s = 0;
    for (int q = 0; q < (int)(blockDim.x / kWave); ++q)
      s += s_w[q][threadIdx.x];
    dst[threadIdx.x] = s;
  }
}

// One radix pass over a chunk of one group: the histogram of digit
// (x >> sh) & 255 of the candidates of every rank (those whose higher
// digits equal the rank's selected prefix) into the group's global
// histograms.  The first pass has one histogram (no prefix yet) and also
// writes the chunk's sums of x, y, x^2, y^2, xy (in 32-bit halves where they
// would overflow); the counter sums come from the grouping pass.
template <bool First>
__global__ __launch_bounds__(kStatT) void k_stats_pass(
    const uint32_t* off, const uint32_t* coff, int G, const uint32_t* xs,
    const uint64_t* ys,
    const uint32_t* spre, int sh, uint32_t* ghist, uint64_t* part) {
  __shared__ uint32_t s_h[kRanks * 256];
  __shared__ uint64_t s_w[kStatT / kWave][kSums];
  int64_t b, e;
  int g;
  if (!chunk_of(coff, off, G, b, e, g)) return;
  const int t = threadIdx.x;
  for (int q = t; q < kRanks * 256; q += kStatT) s_h[q] = 0;
  uint32_t pre[kRanks];
#pragma unroll
  for (int r = 0; r < kRanks; ++r) pre[r] = spre[g * kRanks + r];
  __syncthreads();
  const int hs = sh + 8;
  uint64_t acc[kSums];
#pragma unroll
  for (int k = 0; k < kSums; ++k) acc[k] = 0;
#pragma unroll
  for (int k = 0; k < kStatIpt; ++k) {
    const int64_t i = b + (int64_t)k * kStatT + t;
    const bool ok = i < e;
    const uint32_t x = ok ? xs[i] : 0u;
    const uint32_t dig = (x >> sh) & 255u;
    if (First) {
      lds_claim(s_h, dig, ok);
      if (ok) {
        const uint64_t y = ys[i];
        const uint64_t xx = (uint64_t)x * x;
        const u128 yy = (u128)y * y;
        const uint64_t xy = (uint64_t)x * y;
        acc[0] += x;
        acc[1] += y;
        acc[2] += xx & 0xFFFFFFFFull;
        acc[3] += xx >> 32;
        acc[4] += (uint64_t)yy & 0xFFFFFFFFull;
        acc[5] += (uint64_t)(yy >> 32);
        acc[6] += xy & 0xFFFFFFFFull;
        acc[7] += xy >> 32;
      }
    } else {
#pragma unroll
      for (int r = 0; r < kRanks; ++r)
        lds_claim(&s_h[r * 256], dig, ok && (x >> hs) == (pre[r] >> hs));
    }
  }
  if (First) block_sums(acc, s_w, part + (int64_t)blockIdx.x * kSums);
  __syncthreads();
  uint32_t* gh = ghist + (int64_t)g * kRanks * 256;
  for (int q = t; q < (First ? 256 : kRanks * 256); q += kStatT)
    if (s_h[q]) atomicAdd(&gh[q], s_h[q]);
}

// the digit of every rank of a group from its histogram; the prefix and
// the rank within the remaining candidates move on, and the histograms are
// cleared for the next pass
__global__ __launch_bounds__(kRanks * kWave) void k_stats_select(
    const uint32_t* cnt, int sh, bool first, uint32_t* ghist, uint32_t* spre,
    int64_t* srank) {
  const int g = blockIdx.x, w = threadIdx.x / kWave, lane = lane_id();
  if (cnt[g] == 0) return;
  uint32_t* gh = ghist + (int64_t)g * kRanks * 256;
  const uint32_t* h4 = gh + (first ? 0 : w * 256) + lane * 4;
  uint32_t h[4], sum = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    h[q] = h4[q];
    sum += h[q];
  }
  const int64_t rank = srank[g * kRanks + w];
  const uint32_t incl = wave_incl(sum, OpAdd(), 0u);
  const uint64_t past = __ballot((int64_t)incl > rank);
  const int ln = __ffsll((long long)past) - 1;
  if (lane == ln) {
    int64_t under = (int64_t)incl - sum;
    int dsel = lane * 4 + 3;
    for (int q = 0; q < 4; ++q) {
      if (under + (int64_t)h[q] > rank) {
        dsel = lane * 4 + q;
        break;
      }
      under += h[q];
    }
    spre[g * kRanks + w] |= (uint32_t)dsel << sh;
    srank[g * kRanks + w] = rank - under;
  }
  __syncthreads();
  for (int q = threadIdx.x; q < (first ? 256 : kRanks * 256);
       q += kRanks * kWave)
    gh[q] = 0;
}

struct StatOut {
  double* out;
  int64_t* cnt;
  double freq_peak, tpt_peak;
  int have_f;
  double f_gemm[128];
};

// the exact sums of a group from its chunks and the derived values, in the
// same IEEE operations as their definition
__global__ __launch_bounds__(kBlock) void k_stats_final(
    const uint32_t* cnt, const uint32_t* coff, int G, int O, int nc,
    const uint64_t* part, const uint64_t* csum, const uint32_t* spre,
    StatOut S) {
  __shared__ uint64_t s_w[kBlock / kWave][kSums];
  __shared__ uint64_t s_tot[kSums];
  const int g = blockIdx.x, t = threadIdx.x;
  const int64_t m = cnt[g];
  const double nan = __builtin_nan("");
  double* o = S.out;
  if (m == 0) {
    if (t < kStats) o[(int64_t)t * G + g] = nan;
    if (t == 0) S.cnt[g] = 0;
    return;
  }
  uint64_t acc[kSums];
#pragma unroll
  for (int k = 0; k < kSums; ++k) acc[k] = 0;
  for (uint32_t c = coff[g] + t; c < coff[g + 1]; c += kBlock)
#pragma unroll
    for (int k = 0; k < kSums; ++k) acc[k] += part[(int64_t)c * kSums + k];
  block_sums(acc, s_w, s_tot);
  __syncthreads();
  if (t != 0) return;
  for (int k = 0; k < kStats; ++k) o[(int64_t)k * G + g] = nan;
  S.cnt[g] = m;
  const i128 sx = (i128)s_tot[0], sy = (i128)s_tot[1];
  const i128 sxx = ((i128)s_tot[3] << 32) + (i128)s_tot[2];
  const i128 syy = ((i128)s_tot[5] << 32) + (i128)s_tot[4];
  const i128 sxy = ((i128)s_tot[7] << 32) + (i128)s_tot[6];
  const uint64_t cyc = csum[3 * g], busy = csum[3 * g + 1],
                 flops = csum[3 * g + 2];
  const i128 im = (i128)m;
  const i128 cov = im * sxy - sx * sy;
  const i128 vx = im * sxx - sx * sx;
  const i128 vy = im * syy - sy * sy;
  const double dm = (double)m;
  if (m >= 2 && vx != 0 && vy != 0)
    o[0 * G + g] = i128_to_double(cov) /
                   sqrt(i128_to_double(vx) * i128_to_double(vy));
  double slope = nan, a = nan;
  if (vx != 0) {
    slope = i128_to_double(cov) / i128_to_double(vx);
    a = (i128_to_double(sy) - slope * i128_to_double(sx)) / dm;
  }
  o[1 * G + g] = slope;
  o[2 * G + g] = a;
  const double d0 = a, d50 = a + slope * 536870912.0;
  o[3 * G + g] = d0;
  o[4 * G + g] = d50;
  const uint32_t* v = spre + g * kRanks;
  const double q = 1.0 / 1073741824.0;
  o[5 * G + g] = (double)v[0] * q;
  o[6 * G + g] = (double)v[1] * q;
  o[7 * G + g] = ((double)v[2] + (double)v[3]) / 2.0 * q;
  o[8 * G + g] = (double)v[4] * q;
  o[9 * G + g] = (double)v[5] * q;
  const double dact = i128_to_double(sy) / dm;
  o[10 * G + g] = dact;
  const double ovr_ov = d50 / d0;
  o[14 * G + g] = ovr_ov;
  const double fg = S.have_f ? S.f_gemm[g % O] : nan;
  if (nc >= 16) {
    const double dpeak = (double)cyc * 1000.0 / S.freq_peak / dm;
    o[11 * G + g] = dpeak;
    o[12 * G + g] = 1.0 / ((double)busy / (double)cyc);
    o[13 * G + g] = ((double)flops / dm) / fg;
    o[15 * G + g] = dact / dpeak / ovr_ov;
  }
  o[16 * G + g] = fg / S.tpt_peak;
}

// ------------------------------------------------------ per-GPU overlap CDF
// Instances of (phase, operation) group g on GPU h form CDF group
// c = g * NG + h.  Every row slot of the rows output gets the sort key
// c << 31 | x (x = overlap ratio in Q30), or `sentinel` (above every key)
// when it is no instance; its value is the slot.  After a stable sort by
// key each CDF group is a run in CDF order: ascending x, equal x in row
// order, which is time order on a GPU.
struct CdfArgs {
  StatArgs A;
  const uint8_t* gpu;
  int NG;
};

// Counts and smallest durations of the CDF groups: a block takes kCdfSpan
// row slots (rows of one gpu are consecutive, so nearly all of a block's
// instances are on its first row's gpu) and adds those per (phase,
// operation) in LDS, with one global atomic per group and block; instances
// of other gpus go to the global tables directly.
constexpr int kCdfIpt = 8;
constexpr int kCdfSpan = kBlock * kCdfIpt;

__global__ __launch_bounds__(kBlock) void k_cdf_keys(CdfArgs C,
                                                     uint64_t sentinel,
                                                     uint64_t* key,
                                                     uint32_t* val,
                                                     uint32_t* gcnt,
                                                     uint64_t* ymin) {
  __shared__ uint32_t s_cnt[kMaxGroups];
  __shared__ unsigned long long s_min[kMaxGroups];
  const StatArgs& A = C.A;
  const int G = A.P * A.O;
  for (int g = threadIdx.x; g < G; g += kBlock) {
    s_cnt[g] = 0;
    s_min[g] = ~0ull;
  }
  int64_t lo, hi;
  level_range(A, lo, hi);
  const int64_t b0 = (int64_t)blockIdx.x * kCdfSpan;
  const int64_t f = b0 > lo ? b0 : lo;     // the block's first row in range
  const uint32_t h0 = f < hi ? (uint32_t)C.gpu[f] : 0xFFFFFFFFu;
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kCdfIpt; ++q) {
    const int64_t r = b0 + (int64_t)q * kBlock + threadIdx.x;
    if (r >= A.cap) break;
    uint64_t k = sentinel;
    if (r >= lo && r < hi && A.kind[r] == 0 && A.dur[r] > 0) {
      const uint32_t mp = A.path[(int64_t)A.lv_phase * A.cap + r];
      const uint32_t mo = A.path[(int64_t)A.lv_op * A.cap + r];
      const uint32_t h = C.gpu[r];
      if ((int64_t)mp < A.nm && (int64_t)mo < A.nm && (int)h < C.NG) {
        const uint32_t p = A.label[mp], o = A.label[mo];
        if (p < (uint32_t)A.P && o < (uint32_t)A.O) {
          const uint32_t g = p * (uint32_t)A.O + o;
          const uint64_t c = (uint64_t)g * C.NG + h;
          const uint64_t d = (uint64_t)A.dur[r];
          uint64_t x = ((uint64_t)A.ovl[r] << 30) / d;
          if (x > 0x7FFFFFFFull) x = 0x7FFFFFFFull;   // (RANGE, set elsewhere)
          k = c << 31 | x;
          const uint64_t y = d + (uint64_t)A.gap[r];
          if (h == h0) {
            atomicAdd(&s_cnt[g], 1u);
            atomicMin(&s_min[g], (unsigned long long)y);
          } else {
            atomicAdd(&gcnt[c], 1u);
            atomicMin((unsigned long long*)&ymin[c], (unsigned long long)y);
          }
        }
      }
    }
    key[r] = k;
    val[r] = (uint32_t)r;
  }
  __syncthreads();
  if (h0 == 0xFFFFFFFFu || (int)h0 >= C.NG) return;
  for (int g = threadIdx.x; g < G; g += kBlock)
    if (s_cnt[g]) {
      const int64_t c = (int64_t)g * C.NG + h0;
      atomicAdd(&gcnt[c], s_cnt[g]);
      atomicMin((unsigned long long*)&ymin[c], s_min[g]);
    }
}

// one thread per CDF group: quantiles of x, y_min, D_0%, D_50% and their
// ratio, in the same IEEE operations as their definition
__global__ __launch_bounds__(kBlock) void k_cdf_final(
    CdfArgs C, int64_t NGG, const uint32_t* gcnt, const uint32_t* goff,
    const uint64_t* skey, const uint32_t* sval, const uint64_t* ymin,
    double* gout, int64_t* gcnt_out) {
  const int64_t c = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (c >= NGG) return;
  const int64_t m = gcnt[c];
  gcnt_out[c] = m;
  const double nan = __builtin_nan("");
  if (m == 0) {
    for (int z = 0; z < 9; ++z) gout[(int64_t)z * NGG + c] = nan;
    return;
  }
  const int64_t b = goff[c];
  auto xq = [&](int64_t k) {
    return (double)(uint32_t)(skey[b + k] & 0x7FFFFFFFull);
  };
  auto yk = [&](int64_t k) {
    const uint32_t r = sval[b + k];
    return (double)(C.A.dur[r] + C.A.gap[r]);
  };
  const double q = 1.0 / 1073741824.0, dy = (double)ymin[c];
  gout[0 * NGG + c] = xq(0) * q;
  gout[1 * NGG + c] = xq((m - 1) / 4) * q;
  gout[2 * NGG + c] = (xq((m - 1) / 2) + xq(m / 2)) / 2.0 * q;
  gout[3 * NGG + c] = xq(3 * (m - 1) / 4) * q;
  gout[4 * NGG + c] = xq(m - 1) * q;
  gout[5 * NGG + c] = dy;
  const double c0 = yk(0) / dy;
  const double c50 = (yk((m - 1) / 2) / dy + yk(m / 2) / dy) / 2.0;
  gout[6 * NGG + c] = c0;
  gout[7 * NGG + c] = c50;
  gout[8 * NGG + c] = c50 / c0;
}

// eq. 9 per (phase, operation): the median over its GPUs with instances of
// their D_50% / D_0%; eq. 10 divides by it (overwrites columns 14 and 15 of
// k_stats_final)
__global__ __launch_bounds__(kBlock) void k_cdf_pool(int G, int NG, int nc,
                                                     const int64_t* gcnt,
                                                     const double* gout,
                                                     int64_t NGG,
                                                     double* out) {
  const int g = (int)(blockIdx.x * kBlock + threadIdx.x);
  if (g >= G) return;
  double v[256];
  int k = 0;
  for (int h = 0; h < NG; ++h) {
    const int64_t c = (int64_t)g * NG + h;
    if (gcnt[c] == 0) continue;
    // insertion into ascending order
    const double x = gout[8 * NGG + c];
    int j = k++;
    while (j > 0 && v[j - 1] > x) {
      v[j] = v[j - 1];
      --j;
    }
    v[j] = x;
  }
  const double ovr = k > 0 ? (v[(k - 1) / 2] + v[k / 2]) / 2.0
                           : __builtin_nan("");
  out[14 * (int64_t)G + g] = ovr;
  if (nc >= 16)
    out[15 * (int64_t)G + g] =
        out[10 * (int64_t)G + g] / out[11 * (int64_t)G + g] / ovr;
}

}  // namespace

extern "C" int chopper_op_stats(const chopper_rows* rows, int32_t depth,
                                int32_t n_counters,
                                const chopper_markers* mk,
                                const chopper_stats_spec* spec, double* out,
                                int64_t* cnt, double* gpu_out,
                                int64_t* gpu_cnt, void* scratch,
                                size_t* scratch_bytes, uint32_t* status,
                                void* stream) {
  if (!rows || !spec || !mk || !validate_markers(mk) || !scratch_bytes ||
      !out || !cnt)
    return CHOPPER_EINVAL;
  const int P = spec->n_phases, O = spec->n_ops, NG = spec->n_gpus;
  if (NG < 1 || NG > 256) return CHOPPER_EINVAL;
  if (depth < 1 || depth > mk->depth || spec->phase_level < 0 ||
      spec->phase_level >= depth || spec->op_level < 0 ||
      spec->op_level >= depth || P < 1 || P > 16 || O < 1 || O > 128 ||
      n_counters < 0 || n_counters > 16 || rows->cap < 0 ||
      rows->cap >= (int64_t)0xFFFFFFFF || !rows->level_offset)
    return CHOPPER_EINVAL;
  if (rows->cap > 0 && (!rows->path || !rows->kind || !rows->dur ||
                        !rows->gap || !rows->ovl || !rows->gpu ||
                        (n_counters > 0 && !rows->ctr)))
    return CHOPPER_EINVAL;
  if (mk->n > 0 && !mk->label) return CHOPPER_EINVAL;
  const int G = P * O;
  const int64_t cap = rows->cap;
  const int64_t nchunk = ceil_div(cap, kChunk) + G;
  const int64_t nh = (int64_t)G * kRanks * 256;
  const int64_t NGG = (int64_t)G * NG;      // CDF groups
  const int64_t capn = cap > 0 ? cap : 1;
  struct Bufs {
    uint32_t *key, *gcnt, *off, *cur, *coff, *xs, *ghist, *spre;
    uint64_t *ys, *csum, *part;
    int64_t* srank;
    uint32_t *ccnt, *coffs, *cscan, *ctot, *sval;
    uint64_t *ymin, *skey;
    double* gout;
    int64_t* gcnt_out;
    ClassSortLayout sort;
  } B;
  auto layout = [&](Scratch& sc) {
    B.key = sc.take<uint32_t>(cap);
    B.gcnt = sc.take<uint32_t>(G);
    B.off = sc.take<uint32_t>(G + 1);
    B.cur = sc.take<uint32_t>(G);
    B.coff = sc.take<uint32_t>(G + 1);
    B.xs = sc.take<uint32_t>(cap);
    B.ys = sc.take<uint64_t>(cap);
    B.csum = sc.take<uint64_t>(3 * (int64_t)G);
    B.part = sc.take<uint64_t>(nchunk * kSums);
    B.ghist = sc.take<uint32_t>(nh);
    B.spre = sc.take<uint32_t>((int64_t)G * kRanks);
    B.srank = sc.take<int64_t>((int64_t)G * kRanks);
    B.ccnt = sc.take<uint32_t>(NGG);
    B.coffs = sc.take<uint32_t>(NGG + 1);
    B.cscan = sc.take<uint32_t>(scan_scratch_elems(NGG));
    B.ctot = sc.take<uint32_t>(1);
    B.ymin = sc.take<uint64_t>(NGG);
    B.skey = sc.take<uint64_t>(capn);
    B.sval = sc.take<uint32_t>(capn);
    // (per-GPU results in scratch when the caller passes no arrays)
    B.gout = gpu_out ? gpu_out : sc.take<double>(9 * NGG);
    B.gcnt_out = gpu_cnt ? gpu_cnt : sc.take<int64_t>(NGG);
    B.sort = class_sort_layout(sc, capn, 256);
  };
  Scratch probe(nullptr);
  layout(probe);
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  layout(sc);
  StatArgs A{rows->level_offset, rows->path, rows->kind, rows->dur,
             rows->gap, rows->ovl, rows->ctr, cap, n_counters,
             spec->phase_level, spec->op_level, mk->label, mk->n, P, O};
  StatOut S{out, cnt, spec->freq_peak_mhz, spec->tpt_peak,
            spec->f_gemm != nullptr, {0}};
  for (int o = 0; o < O && spec->f_gemm; ++o) S.f_gemm[o] = spec->f_gemm[o];
  CHOPPER_HIP(launch("stats_clear", k_stats_clear, grid_for(nh, kBlock),
                     dim3(kBlock), s, B.gcnt, G, B.ghist, nh, B.csum));
  const dim3 rb((unsigned)ceil_div(cap > 0 ? cap : 1, (int64_t)kRowSpan));
  CHOPPER_HIP(launch("stats_keys", k_stats_keys, rb, dim3(kStatT), s, A,
                     B.key, B.gcnt, B.csum));
  CHOPPER_HIP(launch("stats_offsets", k_stats_offsets, dim3(1), dim3(kStatT),
                     s, (const uint32_t*)B.gcnt, G, B.off, B.cur, B.coff,
                     B.spre, B.srank));
  CHOPPER_HIP(launch("stats_scatter", k_stats_scatter, rb, dim3(kStatT), s,
                     A, (const uint32_t*)B.key, B.cur, B.xs, B.ys, status));
  for (int pass = 0; pass < 4; ++pass) {
    const int sh = 24 - 8 * pass;
    CHOPPER_HIP(launch("stats_pass",
                       pass == 0 ? k_stats_pass<true> : k_stats_pass<false>,
                       dim3((unsigned)nchunk), dim3(kStatT), s,
                       (const uint32_t*)B.off, (const uint32_t*)B.coff, G,
                       (const uint32_t*)B.xs, (const uint64_t*)B.ys,
                       (const uint32_t*)B.spre, sh, B.ghist, B.part));
    CHOPPER_HIP(launch("stats_select", k_stats_select, dim3((unsigned)G),
                       dim3(kRanks * kWave), s, (const uint32_t*)B.gcnt, sh,
                       pass == 0, B.ghist, B.spre, B.srank));
  }
  CHOPPER_HIP(launch("stats_final", k_stats_final, dim3((unsigned)G),
                     dim3(kBlock), s, (const uint32_t*)B.gcnt,
                     (const uint32_t*)B.coff, G, O, n_counters,
                     (const uint64_t*)B.part, (const uint64_t*)B.csum,
                     (const uint32_t*)B.spre, S));
  // per-GPU overlap CDFs, and eq. 9 / eq. 10 from them
  const CdfArgs C{A, rows->gpu, NG};
  const uint64_t sentinel = (uint64_t)NGG << 31;
  int bits = 0;
  while (bits < 64 && (sentinel >> bits) != 0) ++bits;
  CHOPPER_HIP(launch("stats_cdf", k_stats_clear_cdf, grid_for(NGG, kBlock),
                     dim3(kBlock), s, NGG, B.ccnt, B.ymin));
  if (cap > 0) {
    CHOPPER_HIP(launch("stats_cdf", k_cdf_keys,
                       dim3((unsigned)ceil_div(cap, (int64_t)kCdfSpan)),
                       dim3(kBlock), s, C, sentinel, B.sort.key0, B.sort.val0,
                       B.ccnt, B.ymin));
    ClassSortLayout L = B.sort;
    L.n = cap;
    L.ntiles = sort_tiles(cap);
    rc = radix_sort_pairs(L, bits, B.sval, B.skey, s);
    if (rc != CHOPPER_OK) return rc;
  }
  CHOPPER_HIP(exclusive_scan<uint32_t>(B.ccnt, B.coffs, NGG, B.cscan, B.ctot,
                                       s));
  CHOPPER_HIP(launch("stats_cdf", k_cdf_final, grid_for(NGG, kBlock),
                     dim3(kBlock), s, C, NGG, (const uint32_t*)B.ccnt,
                     (const uint32_t*)B.coffs, (const uint64_t*)B.skey,
                     (const uint32_t*)B.sval, (const uint64_t*)B.ymin, B.gout,
                     B.gcnt_out));
  CHOPPER_HIP(launch("stats_cdf", k_cdf_pool, grid_for(G, kBlock),
                     dim3(kBlock), s, G, NG, n_counters,
                     (const int64_t*)B.gcnt_out, (const double*)B.gout, NGG,
                     out));
  return CHOPPER_OK;
}

}  // namespace chopper
