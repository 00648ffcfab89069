// Wave64 primitives for CDNA (gfx9 family): DPP lane moves, segmented scans
// inside one wavefront, lane-prefix counts from ballots.  Kernels built on
// these treat each wavefront as an independent worker with its own slice of
// LDS, so no block-wide barrier is needed.
#pragma once

#include "common.h"

namespace chopper {

// DPP controls (GCN3 / CDNA encoding)
constexpr int kDppRowShr1 = 0x111;
constexpr int kDppRowShr2 = 0x112;
constexpr int kDppRowShr4 = 0x114;
constexpr int kDppRowShr8 = 0x118;
constexpr int kDppWaveShr1 = 0x138;   // lane i takes lane i-1; lane 0 old
constexpr int kDppWaveRor1 = 0x13C;   // lane i takes lane i-1; lane 0 lane 63
constexpr int kDppRowBcast15 = 0x142; // lane 15 of a row to the next row
constexpr int kDppRowBcast31 = 0x143; // lane 31 to rows 2 and 3

// Lanes whose source is out of range or whose row is masked keep `old`.
template <int Ctrl, int RowMask = 0xF>
__device__ inline uint32_t dpp32(uint32_t old, uint32_t src) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)src, Ctrl,
                                               RowMask, 0xF, false);
}

template <int Ctrl, int RowMask = 0xF>
__device__ inline uint64_t dpp64(uint64_t old, uint64_t src) {
  const uint32_t lo = dpp32<Ctrl, RowMask>((uint32_t)old, (uint32_t)src);
  const uint32_t hi =
      dpp32<Ctrl, RowMask>((uint32_t)(old >> 32), (uint32_t)(src >> 32));
  return ((uint64_t)hi << 32) | lo;
}

// Compiler barrier plus LDS ordering for one wavefront: a wave's LDS
// operations complete in issue order, so this is all that is needed between
// writes and reads of the wave's own LDS slice by different lanes.
__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ inline int lane_id() { return (int)(threadIdx.x & (kWave - 1)); }

// Relaxed device-scope read of a flag word that other waves of the running
// kernel may set (it bypasses the non-coherent vector L1).
__device__ inline uint32_t flag_read(const uint32_t* f) {
  return __hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// OR `bits` into *f when some lane of the wave has `cond`: one atomic per
// wave, and none once the bits are set (a word that most waves set would
// otherwise serialize them all on one address).
__device__ inline void wave_flag_or(uint32_t* f, bool cond, uint32_t bits) {
  if (__ballot(cond) != 0 && lane_id() == 0 && (flag_read(f) & bits) != bits)
    atomicOr(f, bits);
}

// number of set bits of m in lanes below this one
__device__ inline uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Exclusive prefix over lanes of small counts c in [0, 2^bits).
template <int Bits>
__device__ inline uint32_t wave_prefix_small(uint32_t c) {
  uint32_t s = 0;
#pragma unroll
  for (int b = 0; b < Bits; ++b)
    s += lanes_below(__ballot((c >> b) & 1u)) << b;
  return s;
}

// 64-bit combines of the reductions (signed min / max over the same bits)
struct CSum {
  static constexpr uint64_t ident = 0ull;
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const { return a + b; }
};
struct CMin {
  static constexpr uint64_t ident = 0x7FFFFFFFFFFFFFFFull;
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const {
    return (int64_t)a < (int64_t)b ? a : b;
  }
};
struct CMax {
  static constexpr uint64_t ident = 0x8000000000000000ull;
  __device__ uint64_t operator()(uint64_t a, uint64_t b) const {
    return (int64_t)a > (int64_t)b ? a : b;
  }
};

// Flags of a segmented wave scan: bit k of the result is the lane's flag
// before step k (a lane whose flag is set takes nothing from below).  They
// depend only on where segments start, so one computation serves every
// field scanned with the same segments.
struct WaveSegMasks {
  uint32_t before[6];
};

__device__ inline WaveSegMasks wave_seg_masks(bool flag) {
  WaveSegMasks m;
  uint32_t f = flag ? 1u : 0u;
  m.before[0] = f;
  f |= dpp32<kDppRowShr1>(0u, f);
  m.before[1] = f;
  f |= dpp32<kDppRowShr2>(0u, f);
  m.before[2] = f;
  f |= dpp32<kDppRowShr4>(0u, f);
  m.before[3] = f;
  f |= dpp32<kDppRowShr8>(0u, f);
  m.before[4] = f;
  f |= dpp32<kDppRowBcast15, 0xA>(0u, f);
  m.before[5] = f;
  return m;
}

// Inclusive segmented scan across the 64 lanes: a lane whose flag is set
// starts a new segment with its own value.  Kogge-Stone inside 16-lane rows,
// then row broadcasts of lanes 15 and 31.
template <typename C>
__device__ inline uint64_t wave_seg_incl(const WaveSegMasks& m, uint64_t v) {
  C c;
  uint64_t o;
  o = dpp64<kDppRowShr1>(C::ident, v);
  if (!m.before[0]) v = c(o, v);
  o = dpp64<kDppRowShr2>(C::ident, v);
  if (!m.before[1]) v = c(o, v);
  o = dpp64<kDppRowShr4>(C::ident, v);
  if (!m.before[2]) v = c(o, v);
  o = dpp64<kDppRowShr8>(C::ident, v);
  if (!m.before[3]) v = c(o, v);
  o = dpp64<kDppRowBcast15, 0xA>(C::ident, v);
  if (!m.before[4]) v = c(o, v);
  o = dpp64<kDppRowBcast31, 0xC>(C::ident, v);
  if (!m.before[5]) v = c(o, v);
  return v;
}

// Generic DPP move of a trivially copyable value, 32 bits at a time.
template <int Ctrl, int RowMask, typename T>
__device__ inline T dpp_any(T old, T v) {
  static_assert(sizeof(T) % 4 == 0, "DPP moves whole dwords");
  constexpr int W = sizeof(T) / 4;
  uint32_t o[W], s[W], r[W];
  __builtin_memcpy(o, &old, sizeof(T));
  __builtin_memcpy(s, &v, sizeof(T));
#pragma unroll
  for (int i = 0; i < W; ++i) r[i] = dpp32<Ctrl, RowMask>(o[i], s[i]);
  T out;
  __builtin_memcpy(&out, r, sizeof(T));
  return out;
}

// Inclusive scan across the wave for an associative op with a two-sided
// identity (lanes with no source in a step combine with the identity).
template <typename T, typename Op>
__device__ inline T wave_incl(T v, Op op, T ident) {
  v = op(dpp_any<kDppRowShr1, 0xF>(ident, v), v);
  v = op(dpp_any<kDppRowShr2, 0xF>(ident, v), v);
  v = op(dpp_any<kDppRowShr4, 0xF>(ident, v), v);
  v = op(dpp_any<kDppRowShr8, 0xF>(ident, v), v);
  v = op(dpp_any<kDppRowBcast15, 0xA>(ident, v), v);
  v = op(dpp_any<kDppRowBcast31, 0xC>(ident, v), v);
  return v;
}

// the inclusive value of the lane below; lane 0 gets `ident`
template <typename T>
__device__ inline T wave_shr1_any(T ident, T v) {
  return dpp_any<kDppWaveShr1, 0xF>(ident, v);
}

template <typename T>
__device__ inline T lane63(T v) {
  static_assert(sizeof(T) % 4 == 0, "readlane moves whole dwords");
  constexpr int W = sizeof(T) / 4;
  uint32_t s[W];
  __builtin_memcpy(s, &v, sizeof(T));
#pragma unroll
  for (int i = 0; i < W; ++i)
    s[i] = (uint32_t)__builtin_amdgcn_readlane((int)s[i], kWave - 1);
  T out;
  __builtin_memcpy(&out, s, sizeof(T));
  return out;
}

// Wave tiles: eight items per lane.  Loads are striped (item j * 64 + lane
// in lane `lane`) and coalesced; scans want the blocked arrangement (items
// lane * 8 + j), so values go through a per-wave LDS slice with one pad
// element per eight, which keeps both patterns free of bank conflicts.
constexpr int kTileIpt = 8;
constexpr int kWaveTile = kWave * kTileIpt;
constexpr int kSlice = kWaveTile + kWaveTile / 8;
__device__ inline int pad8(int q) { return q + (q >> 3); }

template <typename T>
__device__ inline void wave_to_blocked(T* slice, T (&v)[kTileIpt], int lane) {
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) slice[pad8(j * kWave + lane)] = v[j];
  wave_sync();
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) v[j] = slice[pad8(lane * kTileIpt + j)];
  wave_sync();
}

template <typename T>
__device__ inline void wave_to_striped(T* slice, T (&v)[kTileIpt], int lane) {
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) slice[pad8(lane * kTileIpt + j)] = v[j];
  wave_sync();
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) v[j] = slice[pad8(j * kWave + lane)];
  wave_sync();
}

// value of the lane below (lane 0: old)
__device__ inline uint64_t wave_shr1(uint64_t old, uint64_t v) {
  return dpp64<kDppWaveShr1>(old, v);
}
__device__ inline uint32_t wave_shr1_u32(uint32_t old, uint32_t v) {
  return dpp32<kDppWaveShr1>(old, v);
}
// value of the lane below, lane 0 taking lane 63
__device__ inline uint32_t wave_ror1_u32(uint32_t v) {
  return dpp32<kDppWaveRor1>(v, v);
}

// v of a lane that is the same for the whole wave (a lane read, not a
// permute through LDS)
__device__ inline int64_t readlane64(int64_t v, int lane) {
  const uint64_t u = (uint64_t)v;
  const uint32_t lo =
      (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, lane);
  const uint32_t hi =
      (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), lane);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

}  // namespace chopper
