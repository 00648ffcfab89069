// chopper_align: clock fit (host), fused per-GPU clock transform of every
// record and marker timestamp (one 64x64->128-bit product per timestamp), and
// the two stable record orders.  Paper: Section III-B (alignment of traces so
// that counters attach to operations, layers and iterations).
#include <algorithm>
#include <vector>

#include "clock.h"
#include "sort.h"
#include "wave.h"

namespace chopper {

typedef __int128 int128;
typedef unsigned __int128 uint128;

// ---------------------------------------------------------------------------
// Host clock fit
// ---------------------------------------------------------------------------
// floor(p / q) and the remainder, q > 0
static void floor_divmod(int128 p, int128 q, int128* f, int128* r) {
  int128 a = p / q, b = p % q;
  if (b < 0) { a -= 1; b += q; }
  *f = a;
  *r = b;
}

// nearest integer to p / q (q > 0), ties to even
static int128 round_even(int128 p, int128 q) {
  int128 f, r;
  floor_divmod(p, q, &f, &r);
  int128 twice = r + r;
  if (twice > q) return f + 1;
  if (twice == q) return (f & 1) ? f + 1 : f;
  return f;
}

// nearest integer to |num| * 2^48 / den for 0 < den < 2^126, ties to even;
// the quotient is produced one bit at a time so no intermediate exceeds
// 2 * den.  Returns false when the result would reach 2^38.
static bool q48_quotient(uint128 num, uint128 den, uint128* out) {
  uint128 q = num / den;
  uint128 r = num % den;
  if (q >> 38) return false;
  for (int i = 0; i < 48; ++i) {
    r <<= 1;
    q <<= 1;
    if (r >= den) {
      r -= den;
      q |= 1;
    }
  }
  uint128 r2 = r << 1;
  if (r2 > den || (r2 == den && (q & 1))) q += 1;
  if (q >> 38) return false;
  *out = q;
  return true;
}

static int fit_clocks(const chopper_anchors* anc, int n_gpus,
                      chopper_clock* out) {
  for (int g = 0; g < n_gpus; ++g) out[g] = chopper_clock{0, 0, 0};
  if (!anc || anc->n == 0) return CHOPPER_OK;
  std::vector<std::vector<std::pair<int64_t, int64_t>>> per(n_gpus);
  for (int64_t j = 0; j < anc->n; ++j) {
    int g = anc->gpu[j];
    if (g >= n_gpus) return CHOPPER_EINVAL;
    per[g].push_back({anc->local_ns[j], anc->ref_ns[j]});
  }
  const int128 lim_u = (int128)1 << 42, lim_w = (int128)1 << 40;
  for (int g = 0; g < n_gpus; ++g) {
    auto& v = per[g];
    if (v.empty()) continue;
    if (v.size() > ((size_t)1 << 20)) return CHOPPER_EOVERFLOW;
    std::sort(v.begin(), v.end());
    const int64_t x0 = v[0].first;
    int128 su = 0, sw = 0, suu = 0, suw = 0;
    for (auto& p : v) {
      int128 u = (int128)p.first - x0;
      int128 w = (int128)p.second - p.first;
      if (u >= lim_u || w >= lim_w || w <= -lim_w) return CHOPPER_EOVERFLOW;
      su += u;
      sw += w;
      suu += u * u;
      suw += u * w;
    }
    const int128 cnt = (int128)v.size();
    const int128 den = cnt * suu - su * su;
    const int128 num = cnt * suw - su * sw;
    int128 d = 0;
    if (cnt > 1 && den > 0) {
      uint128 mag;
      bool neg = num < 0;
      if (!q48_quotient((uint128)(neg ? -num : num), (uint128)den, &mag))
        return CHOPPER_EOVERFLOW;
      d = neg ? -(int128)mag : (int128)mag;
    }
    const int128 one48 = (int128)1 << 48;
    int128 c = round_even(sw * one48 - d * su, cnt * one48);
    out[g] = chopper_clock{x0, (int64_t)c, (int64_t)d};
  }
  return CHOPPER_OK;
}

// ---------------------------------------------------------------------------
// Device transform (clock.h)
// ---------------------------------------------------------------------------
__device__ inline void status_or(uint32_t* status, uint32_t bits) {
  // one atomic per wave that has anything to report
  uint32_t v = bits;
  for (int d = kWave / 2; d > 0; d >>= 1) v |= __shfl_xor(v, d, kWave);
  if ((threadIdx.x & (kWave - 1)) == 0 && v) atomicOr(status, v);
}

// Presence of (gpu, stream) and (gpu, kind) pairs as byte flags written with
// plain stores (no read-modify-write on the few hot lines); within a wave
// only the lanes whose pair differs from the previous lane's store.
__device__ inline void mark_present(uint8_t* flags, uint32_t idx) {
  const uint32_t prev = __shfl_up(idx, 1, kWave);
  const int lane = threadIdx.x & (kWave - 1);
  if (lane == 0 || prev != idx) flags[idx] = 1;
}

__global__ __launch_bounds__(kBlock) void k_transform_records(
    int64_t n, int n_gpus, const uint8_t* gpu, const uint8_t* stream,
    const uint8_t* cls, const int64_t* start, const int64_t* end,
    const ClockDev* clk, int64_t* s_out, int64_t* e_out, uint8_t* pres_s,
    uint8_t* pres_k, uint32_t* unsorted, uint32_t* status,
    WaveClasses* wcls) {
  // each lane owns eight consecutive records (a wave 512)
  const int lane = lane_id(), wv = (int)(threadIdx.x / kWave);
  const int64_t base =
      ((int64_t)blockIdx.x * kWavesPerBlock + wv) * (int64_t)kWaveTile;
  if (base >= n) return;
  const int64_t k0 = base + (int64_t)lane * kTileIpt;
  const bool full = base + kWaveTile <= n;
  const bool vec = full && (((uintptr_t)gpu | (uintptr_t)stream |
                             (uintptr_t)cls) & 7) == 0 &&
                   (((uintptr_t)start | (uintptr_t)end | (uintptr_t)s_out |
                     (uintptr_t)e_out) & 15) == 0;
  uint8_t g8[kTileIpt], st8[kTileIpt], c8[kTileIpt];
  int64_t s[kTileIpt], e[kTileIpt];
  if (vec) {
    *reinterpret_cast<uint2*>(g8) = *reinterpret_cast<const uint2*>(gpu + k0);
    *reinterpret_cast<uint2*>(st8) =
        *reinterpret_cast<const uint2*>(stream + k0);
    *reinterpret_cast<uint2*>(c8) = *reinterpret_cast<const uint2*>(cls + k0);
#pragma unroll
    for (int q = 0; q < kTileIpt / 2; ++q) {
      *reinterpret_cast<int4*>(&s[2 * q]) =
          reinterpret_cast<const int4*>(start + k0)[q];
      *reinterpret_cast<int4*>(&e[2 * q]) =
          reinterpret_cast<const int4*>(end + k0)[q];
    }
  } else {
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j) {
      const int64_t k = k0 + j;
      const bool v = k < n;
      g8[j] = v ? gpu[k] : 0;
      st8[j] = v ? stream[k] : 0;
      c8[j] = v ? cls[k] : 0;
      s[j] = v ? start[k] : 0;
      e[j] = v ? end[k] : 0;
    }
  }
  uint32_t st = 0;
  int64_t s2[kTileIpt], e2[kTileIpt];
  uint32_t gl = 0xFFFFFFFFu;     // gpu of the clock held
  ClockDev kc{0, 0, 0};
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const uint32_t g = g8[j];
    if (k0 + j >= n) {
      s2[j] = e2[j] = 0;
      continue;
    }
    if (g != gl) {
      gl = g;
      kc = (int)g < n_gpus ? clk[g] : ClockDev{0, 0, 0};
    }
    if ((int)g >= n_gpus) st |= CHOPPER_ST_BAD_GPU;
    if (c8[j] >= 8) st |= CHOPPER_ST_BAD_CLASS;
    if (e[j] < s[j]) st |= CHOPPER_ST_NEG_DURATION;
    s2[j] = align_time(s[j], kc);
    e2[j] = align_time(e[j], kc);
    if (out_of_range(s[j]) || out_of_range(e[j]) || out_of_range(s2[j]) ||
        out_of_range(e2[j]))
      st |= CHOPPER_ST_RANGE;
  }
  if (vec) {
#pragma unroll
    for (int q = 0; q < kTileIpt / 2; ++q) {
      reinterpret_cast<int4*>(s_out + k0)[q] =
          *reinterpret_cast<const int4*>(&s2[2 * q]);
      reinterpret_cast<int4*>(e_out + k0)[q] =
          *reinterpret_cast<const int4*>(&e2[2 * q]);
    }
  } else {
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j)
      if (k0 + j < n) {
        s_out[k0 + j] = s2[j];
        e_out[k0 + j] = e2[j];
      }
  }
  // The wave's classes in both keys, for the class histogram: the first
  // record's, then the first other one met, counted by ballots per row
  // (uniform control: the ballots are the wave's).  They also give the
  // presence of the (gpu, stream) and (gpu, kind) pairs: lane 0 marks them,
  // and only a wave with more classes marks them record by record (one
  // plain byte store per run of equal pairs in the lane).
  {
    uint32_t ks[kTileIpt], kk[kTileIpt];
#pragma unroll
    for (int j = 0; j < kTileIpt; ++j) {
      ks[j] = (uint32_t)g8[j] * 256u + st8[j];
      kk[j] = (uint32_t)g8[j] * 2u + (uint32_t)kind_of(c8[j]);
    }
    WaveClasses wc;
    auto classes = [&](const uint32_t (&key)[kTileIpt], uint8_t* pres,
                       uint32_t& c0, uint32_t& n0, uint32_t& c1,
                       uint32_t& n1) {
      c0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)key[0]);
      c1 = kNone;
      n0 = n1 = 0;
      bool many = false;
#pragma unroll
      for (int j = 0; j < kTileIpt; ++j) {
        const bool v = k0 + j < n;
        const uint64_t m0 = __ballot(v && key[j] == c0);
        const uint64_t rest = __ballot(v && key[j] != c0);
        n0 += (uint32_t)__popcll(m0);
        if (rest) {
          if (c1 == kNone)
            c1 = (uint32_t)__builtin_amdgcn_readlane(
                (int)key[j], __ffsll((long long)rest) - 1);
          const uint64_t m1 = __ballot(v && key[j] == c1);
          n1 += (uint32_t)__popcll(m1);
          many = many || (rest & ~m1) != 0;
        }
      }
      if (many) {
        c1 = kManyClasses;
        uint32_t pv = kNone;
#pragma unroll
        for (int j = 0; j < kTileIpt; ++j) {
          if (k0 + j >= n) break;
          if (key[j] != pv) pres[key[j]] = 1;
          pv = key[j];
        }
      } else if (lane == 0) {
        pres[c0] = 1;
        if (c1 != kNone) pres[c1] = 1;
      }
    };
    classes(ks, pres_s, wc.a0, wc.na0, wc.a1, wc.na1);
    classes(kk, pres_k, wc.b0, wc.nb0, wc.b1, wc.nb1);
    if (lane == 0) wcls[base / kWaveTile] = wc;
  }
  // is the input ordered by (gpu, start')?  Then every (gpu, stream) and
  // (gpu, kind) subsequence is time-ordered and one stable class pass sorts.
  bool bad = false;
#pragma unroll
  for (int j = 1; j < kTileIpt; ++j)
    if (k0 + j < n)
      bad = bad || g8[j - 1] > g8[j] || (g8[j - 1] == g8[j] && s2[j - 1] > s2[j]);
  // the lane below's last record (lane 0: the record before the tile)
  uint32_t pg = wave_shr1_u32(0u, (uint32_t)g8[kTileIpt - 1]);
  int64_t pst = wave_shr1((uint64_t)0, (uint64_t)s2[kTileIpt - 1]);
  bool have = lane > 0;
  if (lane == 0 && base > 0) {
    pg = gpu[base - 1];
    const ClockDev kp = (int)pg < n_gpus ? clk[pg] : ClockDev{0, 0, 0};
    pst = align_time(start[base - 1], kp);
    have = true;
  }
  if (have && k0 < n)
    bad = bad || pg > g8[0] || (pg == g8[0] && pst > s2[0]);
  if (__ballot(bad) != 0 && lane == 0) atomicOr(unsorted, 1u);
  status_or(status, st);
}

__global__ __launch_bounds__(kBlock) void k_transform_markers(
    int64_t n, int n_gpus, int depth, const uint8_t* gpu, const uint8_t* level,
    const int64_t* start, const int64_t* end, const ClockDev* clk,
    int64_t* s_out, int64_t* e_out, uint32_t* status) {
  const int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  uint32_t st = 0;
  if (i < n) {
    const uint32_t g = gpu[i];
    const int64_t s = start[i], e = end[i];
    ClockDev k{0, 0, 0};
    if ((int)g < n_gpus) k = clk[g];
    else st |= CHOPPER_ST_BAD_GPU;
    if ((int)level[i] >= depth) st |= CHOPPER_ST_BAD_LEVEL;
    if (e < s) st |= CHOPPER_ST_NEG_DURATION;
    const int64_t s2 = align_time(s, k), e2 = align_time(e, k);
    if (out_of_range(s) || out_of_range(e) || out_of_range(s2) ||
        out_of_range(e2))
      st |= CHOPPER_ST_RANGE;
    s_out[i] = s2;
    e_out[i] = e2;
  }
  status_or(status, st);
}

// Dense class ids in (gpu, stream) and (gpu, kind) order from the presence
// flags (65536 + 512 bytes), one block of 1024 threads: every thread counts
// 64 consecutive (gpu, stream) flags (and at most one (gpu, kind) flag), a
// block scan numbers them, and every thread writes its own ids with
// 16-byte stores.
constexpr int kDenseThreads = 1024;

__device__ inline uint32_t block1024_exclusive(uint32_t v, uint32_t* s_w,
                                               uint32_t* total) {
  const int lane = lane_id(), w = (int)(threadIdx.x / kWave);
  const uint32_t incl = wave_incl(v, OpAdd(), 0u);
  if (lane == kWave - 1) s_w[w] = incl;
  __syncthreads();
  uint32_t pre = 0, tot = 0;
  for (int q = 0; q < kDenseThreads / kWave; ++q) {
    if (q < w) pre += s_w[q];
    tot += s_w[q];
  }
  __syncthreads();
  *total = tot;
  return pre + incl - v;
}

__global__ __launch_bounds__(kDenseThreads) void k_dense_classes(
    const uint8_t* pres_s, uint16_t* cmap_s, const uint8_t* pres_k,
    uint16_t* cmap_k, uint32_t* counts) {
  __shared__ uint32_t s_w[kDenseThreads / kWave];
  const int t = threadIdx.x;
  uint4 f[4];
  const uint4* src = reinterpret_cast<const uint4*>(pres_s) + t * 4;
#pragma unroll
  for (int q = 0; q < 4; ++q) f[q] = src[q];
  const uint8_t* fb = reinterpret_cast<const uint8_t*>(f);
  uint32_t c = 0;
#pragma unroll
  for (int b = 0; b < 64; ++b) c += fb[b] ? 1u : 0u;
  uint32_t tot;
  uint32_t id = block1024_exclusive(c, s_w, &tot);
  uint16_t ids[64];
#pragma unroll
  for (int b = 0; b < 64; ++b) {
    ids[b] = (uint16_t)(fb[b] ? id : 0u);
    id += fb[b] ? 1u : 0u;
  }
  uint4* dst = reinterpret_cast<uint4*>(cmap_s) + t * 8;
  const uint4* iv = reinterpret_cast<const uint4*>(ids);
#pragma unroll
  for (int q = 0; q < 8; ++q) dst[q] = iv[q];
  if (t == 0) counts[0] = tot;
  // (gpu, kind) flags: one per thread
  const uint32_t on = t < 512 && pres_k[t] ? 1u : 0u;
  uint32_t totk;
  const uint32_t k = block1024_exclusive(on, s_w, &totk);
  if (t < 512) cmap_k[t] = (uint16_t)(on ? k : 0u);
  if (t == 0) counts[1] = totk;
}

// presence flags (65536 + 512 bytes) and the class counts to zero
__global__ __launch_bounds__(kBlock) void k_align_clear(uint32_t* pres,
                                                        uint32_t* counts) {
  const int i = (int)(blockIdx.x * kBlock + threadIdx.x);
  if (i < 16384 + 128) pres[i] = 0;
  if (i < 4) counts[i] = 0;
}

// ---------------------------------------------------------------------------
// Entry point
// ---------------------------------------------------------------------------
struct AlignLayout {
  ClockDev* clk;
  uint8_t* pres_s;    // 65536 + 512 byte flags, cleared together
  uint8_t* pres_k;
  uint16_t* cmap_s;
  uint16_t* cmap_k;
  uint32_t* counts;
  uint32_t* coff;
  WaveClasses* wcls;   // classes of every wave tile of the records
  ClassSortLayout sort;
};

static AlignLayout align_layout(Scratch& sc, int64_t n, int n_gpus) {
  AlignLayout L;
  L.clk = sc.take<ClockDev>(n_gpus);
  L.pres_s = sc.take<uint8_t>(65536 + 512);
  L.pres_k = L.pres_s ? L.pres_s + 65536 : nullptr;
  L.cmap_s = sc.take<uint16_t>(65536);
  L.cmap_k = sc.take<uint16_t>(512);
  L.counts = sc.take<uint32_t>(4);
  L.coff = sc.take<uint32_t>(65536 + 1);
  L.wcls = sc.take<WaveClasses>(ceil_div(n, (int64_t)kWaveTile));
  L.sort = class_sort_layout(sc, n, 65536);
  return L;
}

static bool records_ok(const chopper_records* r) {
  if (!r || r->n < 0 || r->n >= (int64_t)0xFFFFFFFF) return false;
  if (r->n_gpus < 1 || r->n_gpus > 256) return false;
  if (r->n_counters < 0 || r->n_counters > 16) return false;
  if (r->n > 0 && (!r->gpu || !r->stream || !r->cls || !r->start_ns ||
                   !r->end_ns))
    return false;
  if (r->n > 0 && r->n_counters > 0 && !r->counters) return false;
  return true;
}

static bool markers_ok(const chopper_markers* m) {
  if (!m) return true;
  if (m->n < 0 || m->n >= (int64_t)0xFFFFFFFF) return false;
  if (m->depth < 1 || m->depth > 8) return false;
  if (m->n > 0 && (!m->gpu || !m->level || !m->start_ns || !m->end_ns))
    return false;
  return true;
}

bool validate_records(const chopper_records* r) { return records_ok(r); }
bool validate_markers(const chopper_markers* m) { return markers_ok(m); }

}  // namespace chopper

using namespace chopper;

extern "C" int chopper_align(const chopper_records* rec,
                             const chopper_markers* mk,
                             const chopper_anchors* anc,
                             chopper_clock* clocks_out, int64_t* start_out,
                             int64_t* end_out, int64_t* mstart_out,
                             int64_t* mend_out, uint32_t* order_out,
                             uint32_t* korder_out, void* scratch,
                             size_t* scratch_bytes, uint32_t* status,
                             void* stream) {
  if (!records_ok(rec) || !markers_ok(mk) || !clocks_out || !scratch_bytes)
    return CHOPPER_EINVAL;
  if (anc && anc->n < 0) return CHOPPER_EINVAL;
  if (anc && anc->n > 0 && (!anc->gpu || !anc->local_ns || !anc->ref_ns))
    return CHOPPER_EINVAL;
  const int64_t n = rec->n;
  const int64_t nm = mk ? mk->n : 0;
  const int G = rec->n_gpus;
  if (n > 0 && (!start_out || !end_out || !order_out || !korder_out))
    return CHOPPER_EINVAL;
  if (nm > 0 && (!mstart_out || !mend_out)) return CHOPPER_EINVAL;
  Scratch probe(nullptr);
  align_layout(probe, n, G);
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;

  std::vector<chopper_clock> clocks(G);
  rc = fit_clocks(anc, G, clocks.data());
  if (rc != CHOPPER_OK) return rc;
  for (int g = 0; g < G; ++g) clocks_out[g] = clocks[g];

  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  AlignLayout L = align_layout(sc, n, G);
  std::vector<ClockDev> cd(G);
  for (int g = 0; g < G; ++g)
    cd[g] = ClockDev{clocks[g].x0, clocks[g].c, clocks[g].d_q48};
  CHOPPER_HIP(hipMemcpyAsync(L.clk, cd.data(), sizeof(ClockDev) * G,
                             hipMemcpyHostToDevice, s));
  auto markers = [&]() -> int {
    if (nm > 0)
      CHOPPER_HIP(launch("align_transform_markers", k_transform_markers,
                         grid_for(nm, kBlock), dim3(kBlock), s, nm, G,
                         mk->depth, mk->gpu, mk->level, mk->start_ns,
                         mk->end_ns, (const ClockDev*)L.clk, mstart_out,
                         mend_out, status));
    return CHOPPER_OK;
  };
  if (n == 0) return markers();
  CHOPPER_HIP(launch("align_fill", k_align_clear,
                     grid_for(16384 + 128, kBlock), dim3(kBlock), s,
                     reinterpret_cast<uint32_t*>(L.pres_s), L.counts));
  CHOPPER_HIP(launch("align_transform_records", k_transform_records,
                     dim3((unsigned)ceil_div(n, (int64_t)kWaveTile *
                                                    kWavesPerBlock)),
                     dim3(kBlock), s, n, G, rec->gpu,
                     rec->stream, rec->cls, rec->start_ns, rec->end_ns,
                     (const ClockDev*)L.clk, start_out, end_out, L.pres_s,
                     L.pres_k, L.counts + 2, status, L.wcls));
  CHOPPER_HIP(launch("align_dense_classes", k_dense_classes, dim3(1),
                     dim3(kDenseThreads), s, (const uint8_t*)L.pres_s, L.cmap_s,
                     (const uint8_t*)L.pres_k, L.cmap_k, L.counts));
  // the markers are transformed while the host waits for the class counts
  uint32_t counts[3];
  ReadBack rb;
  CHOPPER_HIP(read_back_start(L.counts, sizeof(counts), s, &rb));
  rc = markers();
  if (rc != CHOPPER_OK) {
    (void)read_back_finish(&rb, counts);
    return rc;
  }
  CHOPPER_HIP(read_back_finish(&rb, counts));
  // counts[2] != 0: the input is not ordered by (gpu, start')
  const int known = counts[2] ? -1 : 1;
  bool range_err = false, r2 = false;
  KeyRecStream ks{rec->gpu, rec->stream, start_out, L.cmap_s, (int)counts[0]};
  KeyRecKind kk{rec->gpu, rec->cls, start_out, L.cmap_k, (int)counts[1]};
  if (known == 1 && counts[0] + counts[1] <= 256) {
    // input in (gpu, start') order: both orders are class partitions,
    // computed together
    rc = class_sort2(ks, kk, L.sort, order_out, L.coff, korder_out,
                     L.coff + counts[0] + 1, s, (const WaveClasses*)L.wcls);
    if (rc != CHOPPER_OK) return rc;
  } else {
    rc = class_sort(ks, L.sort, order_out, L.coff, &range_err, s, known);
    if (rc != CHOPPER_OK) return rc;
    rc = class_sort(kk, L.sort, korder_out, L.coff, &r2, s, known);
    if (rc != CHOPPER_OK) return rc;
  }
  if (range_err || r2) {
    // fold the host-detected condition into the device status word
    CHOPPER_HIP(launch("status_set", k_status_set, dim3(1), dim3(1), s,
                       (uint32_t)CHOPPER_ST_RANGE, status));
  }
  return CHOPPER_OK;
}
