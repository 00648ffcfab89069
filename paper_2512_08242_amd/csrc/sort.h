// Stable (class, time) sorts shared by chopper_align (record orders) and
// chopper_attribute (marker index).
#pragma once

#include "common.h"

namespace chopper {

// Eight consecutive items i0 .. i0 + 7 of a column (b[j] = 0 past n), as one
// 8-byte load when the run is whole and aligned.
__device__ inline void load8_u8(const uint8_t* p, int64_t i0, int64_t n,
                                uint32_t (&b)[8]) {
  if (i0 + 8 <= n && ((uintptr_t)(p + i0) & 7) == 0) {
    const uint64_t w = *reinterpret_cast<const uint64_t*>(p + i0);
#pragma unroll
    for (int j = 0; j < 8; ++j) b[j] = (uint32_t)(w >> (8 * j)) & 0xFFu;
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) b[j] = i0 + j < n ? (uint32_t)p[i0 + j] : 0u;
  }
}

__device__ inline void load8_i64(const int64_t* p, int64_t i0, int64_t n,
                                 int64_t (&x)[8]) {
  if (i0 + 8 <= n && ((uintptr_t)(p + i0) & 15) == 0) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const uint4 v = reinterpret_cast<const uint4*>(p + i0)[k];
      x[2 * k] = (int64_t)((uint64_t)v.x | (uint64_t)v.y << 32);
      x[2 * k + 1] = (int64_t)((uint64_t)v.z | (uint64_t)v.w << 32);
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = i0 + j < n ? p[i0 + j] : 0;
  }
}

// Class ids of the eight items i0 .. i0 + 7 (v[j]: i0 + j < n); accessors
// over plain columns override it with vector loads.
template <typename Acc>
__device__ inline void cls_block(const Acc& acc, int64_t i0, int64_t n,
                                 uint32_t (&d)[8], bool (&v)[8]) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    v[j] = i0 + j < n;
    d[j] = v[j] ? acc.cls(i0 + j) : 0u;
  }
}

// Records keyed by (gpu, stream): dense class ids from a 256 x 256 table.
struct KeyRecStream {
  const uint8_t* gpu;
  const uint8_t* stream;
  const int64_t* t;
  const uint16_t* cmap;   // [256 * 256]
  int C;
  __device__ uint32_t cls(int64_t i) const {
    return cmap[(uint32_t)gpu[i] * 256u + stream[i]];
  }
  // class of the raw code gpu * 256 + stream
  __device__ uint32_t cls_of_raw(uint32_t raw) const { return cmap[raw]; }
  // raw codes of items i0 .. i0 + 7
  __device__ void raw8(int64_t i0, int64_t n, uint32_t (&r)[8]) const {
    uint32_t g[8], s[8];
    load8_u8(gpu, i0, n, g);
    load8_u8(stream, i0, n, s);
#pragma unroll
    for (int j = 0; j < 8; ++j) r[j] = g[j] * 256u + s[j];
  }
  __device__ int64_t time(int64_t i) const { return t[i]; }
  __device__ uint32_t major(int64_t i) const { return gpu[i]; }
  __host__ __device__ int nclass() const { return C; }
  __device__ void cls8(int64_t i0, int64_t n, uint32_t (&d)[8],
                       bool (&v)[8]) const {
    uint32_t g[8], s[8];
    load8_u8(gpu, i0, n, g);
    load8_u8(stream, i0, n, s);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      v[j] = i0 + j < n;
      d[j] = v[j] ? cmap[g[j] * 256u + s[j]] : 0u;
    }
  }
};
__device__ inline void cls_block(const KeyRecStream& a, int64_t i0, int64_t n,
                                 uint32_t (&d)[8], bool (&v)[8]) {
  a.cls8(i0, n, d, v);
}

// Records keyed by (gpu, kind): dense class ids from a 256 x 2 table.
struct KeyRecKind {
  const uint8_t* gpu;
  const uint8_t* cl;
  const int64_t* t;
  const uint16_t* cmap;   // [256 * 2]
  int C;
  __device__ uint32_t cls(int64_t i) const {
    return cmap[(uint32_t)gpu[i] * 2u + (uint32_t)kind_of(cl[i])];
  }
  // class of the raw code gpu * 2 + kind
  __device__ uint32_t cls_of_raw(uint32_t raw) const { return cmap[raw]; }
  // raw codes of items i0 .. i0 + 7
  __device__ void raw8(int64_t i0, int64_t n, uint32_t (&r)[8]) const {
    uint32_t g[8], c[8];
    load8_u8(gpu, i0, n, g);
    load8_u8(cl, i0, n, c);
#pragma unroll
    for (int j = 0; j < 8; ++j) r[j] = g[j] * 2u + (uint32_t)kind_of(c[j]);
  }
  __device__ int64_t time(int64_t i) const { return t[i]; }
  __device__ uint32_t major(int64_t i) const { return gpu[i]; }
  __host__ __device__ int nclass() const { return C; }
  __device__ void cls8(int64_t i0, int64_t n, uint32_t (&d)[8],
                       bool (&v)[8]) const {
    uint32_t g[8], c[8];
    load8_u8(gpu, i0, n, g);
    load8_u8(cl, i0, n, c);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      v[j] = i0 + j < n;
      d[j] = v[j] ? cmap[g[j] * 2u + (uint32_t)kind_of((uint8_t)c[j])] : 0u;
    }
  }
};
__device__ inline void cls_block(const KeyRecKind& a, int64_t i0, int64_t n,
                                 uint32_t (&d)[8], bool (&v)[8]) {
  a.cls8(i0, n, d, v);
}

// Markers keyed by (gpu, level, empty): non-empty markers of a (gpu, level)
// come first; markers with an invalid gpu or level go to the last class.
struct KeyMarker {
  const uint8_t* gpu;
  const uint8_t* level;
  const int64_t* ms;
  const int64_t* me;
  int G, D;
  __device__ uint32_t cls(int64_t i) const {
    uint32_t g = gpu[i], l = level[i];
    if ((int)g >= G || (int)l >= D) return (uint32_t)(G * D * 2);
    return (g * (uint32_t)D + l) * 2u + (me[i] <= ms[i] ? 1u : 0u);
  }
  __device__ int64_t time(int64_t i) const { return ms[i]; }
  __device__ uint32_t major(int64_t i) const { return gpu[i]; }
  __host__ __device__ int nclass() const { return G * D * 2 + 1; }
  __device__ void cls8(int64_t i0, int64_t n, uint32_t (&d)[8],
                       bool (&v)[8]) const {
    uint32_t g[8], l[8];
    int64_t a[8], b[8];
    load8_u8(gpu, i0, n, g);
    load8_u8(level, i0, n, l);
    load8_i64(ms, i0, n, a);
    load8_i64(me, i0, n, b);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      v[j] = i0 + j < n;
      const bool bad = (int)g[j] >= G || (int)l[j] >= D;
      d[j] = !v[j] ? 0u
             : bad ? (uint32_t)(G * D * 2)
                   : (g[j] * (uint32_t)D + l[j]) * 2u + (b[j] <= a[j] ? 1u : 0u);
    }
  }
};
__device__ inline void cls_block(const KeyMarker& a, int64_t i0, int64_t n,
                                 uint32_t (&d)[8], bool (&v)[8]) {
  a.cls8(i0, n, d, v);
}

// What a class partition can write beside the permutation, at each item's
// sorted position p (item index i, class c): nothing by default.
struct NoColumns {
  __device__ void put(int64_t, uint32_t, uint32_t) const {}
};

// The markers' sorted columns: start', end' and input index.
struct MarkerColumns {
  const int64_t* ms;
  const int64_t* me;
  int64_t* sms;
  int64_t* sme;
  uint32_t* sid;
  __device__ void put(int64_t p, uint32_t i, uint32_t) const {
    sms[p] = ms[i];
    sme[p] = me[i];
    sid[p] = i;
  }
};

// Positions of a sequence (position p holds item seq[p]) keyed by (dense
// class of the item's (gpu, stream), the item's label): their stable sort
// brings every label of a class together and keeps the sequence order
// inside it (labels as times; NONE sorts last).
struct KeySeqLabel {
  const uint32_t* seq;
  const uint8_t* gpu;
  const uint8_t* stream;
  const uint32_t* lab;
  const uint16_t* cmap;   // [256 * 256]
  int C;
  __device__ uint32_t cls(int64_t p) const {
    const uint32_t i = seq[p];
    return cmap[(uint32_t)gpu[i] * 256u + stream[i]];
  }
  __device__ int64_t time(int64_t p) const { return (int64_t)lab[seq[p]]; }
  __device__ uint32_t major(int64_t p) const { return cls(p); }
  __host__ __device__ int nclass() const { return C; }
  __device__ void cls8(int64_t p0, int64_t n, uint32_t (&d)[8],
                       bool (&v)[8]) const {
    uint32_t it[8];
    if (p0 + 8 <= n && ((uintptr_t)(seq + p0) & 15) == 0) {
      const uint4 x = reinterpret_cast<const uint4*>(seq + p0)[0];
      const uint4 y = reinterpret_cast<const uint4*>(seq + p0)[1];
      it[0] = x.x; it[1] = x.y; it[2] = x.z; it[3] = x.w;
      it[4] = y.x; it[5] = y.y; it[6] = y.z; it[7] = y.w;
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) it[j] = p0 + j < n ? seq[p0 + j] : 0u;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      v[j] = p0 + j < n;
      d[j] = v[j] ? cmap[(uint32_t)gpu[it[j]] * 256u + stream[it[j]]] : 0u;
    }
  }
};
__device__ inline void cls_block(const KeySeqLabel& a, int64_t i0, int64_t n,
                                 uint32_t (&d)[8], bool (&v)[8]) {
  a.cls8(i0, n, d, v);
}

// (major, time) of the nine items i0 .. i0 + 8 (v[j]: i0 + j < n)
template <typename Acc>
__device__ inline void major_time_block(const Acc& acc, int64_t i0, int64_t n,
                                        uint32_t (&m)[9], int64_t (&t)[9],
                                        bool (&v)[9]) {
#pragma unroll
  for (int j = 0; j < 9; ++j) {
    v[j] = i0 + j < n;
    m[j] = v[j] ? acc.major(i0 + j) : 0u;
    t[j] = v[j] ? acc.time(i0 + j) : 0;
  }
}
__device__ inline void major_time_block(const KeyMarker& a, int64_t i0,
                                        int64_t n, uint32_t (&m)[9],
                                        int64_t (&t)[9], bool (&v)[9]) {
  uint32_t g[8];
  int64_t x[8];
  load8_u8(a.gpu, i0, n, g);
  load8_i64(a.ms, i0, n, x);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    v[j] = i0 + j < n;
    m[j] = g[j];
    t[j] = x[j];
  }
  v[8] = i0 + 8 < n;
  m[8] = v[8] ? a.gpu[i0 + 8] : 0u;
  t[8] = v[8] ? a.ms[i0 + 8] : 0;
}

struct ClassSortLayout {
  int64_t n = 0;
  int C = 0;
  int64_t ntiles = 0;
  uint32_t* tilehist = nullptr;
  uint32_t* tileoff = nullptr;
  uint32_t* scantmp = nullptr;
  uint32_t* total = nullptr;
  uint32_t* flag = nullptr;
  int64_t* mm = nullptr;
  uint64_t* key0 = nullptr;
  uint64_t* key1 = nullptr;
  uint32_t* val0 = nullptr;
  uint32_t* val1 = nullptr;
};

int64_t sort_tiles(int64_t n);
// Sized for up to c_max classes.
ClassSortLayout class_sort_layout(Scratch& sc, int64_t n, int c_max);

// out[n]: stable permutation by (class, time); coff[C + 1]: first position of
// every class and n.  range_error: the packed key would need more than 64
// bits (only possible on the general path).  known_sorted = 1: the caller
// knows the input is ordered by (major, time) -- the gpu of every accessor
// leads its class order -- so each class subsequence is already
// time-ordered; -1: unknown, checked here.  May synchronize `s`.  `cols`
// is written at the sorted positions when the class partition is the sort;
// *cols_done (optional) says whether it was (else the caller gathers them).
template <typename Acc, typename Cols = NoColumns>
int class_sort(const Acc& acc, const ClassSortLayout& L, uint32_t* out,
               uint32_t* coff, bool* range_error, hipStream_t s,
               int known_sorted, const Cols& cols = Cols(),
               bool* cols_done = nullptr);

// The classes of a wave tile of kWaveTile consecutive records in both keys,
// recorded by the pass that reads the records, as raw codes (gpu * 256 +
// stream, gpu * 2 + kind): one or two per key with their counts (na1 = 0:
// one); a1 or b1 is kManyClasses when the wave holds more than two.
struct WaveClasses {
  uint32_t a0, na0, a1, na1, b0, nb0, b1, nb1;
};
constexpr uint32_t kManyClasses = 0xFFFFFFFEu;

// Both class partitions of the same n > 0 items at once, for input ordered
// by (major, time) (so the partitions are the stable sorts); needs
// a.nclass() + b.nclass() <= 256.  `wcls` holds one WaveClasses per wave
// tile of the items: a sort tile whose waves hold at most two classes per
// key in all is counted and partitioned from them and the raw codes, the
// other tiles item by item.
template <typename AccA, typename AccB>
int class_sort2(const AccA& a, const AccB& b, const ClassSortLayout& L,
                uint32_t* outA, uint32_t* coffA, uint32_t* outB,
                uint32_t* coffB, hipStream_t s, const WaveClasses* wcls);

// Stable LSD radix sort of the (L.key0, L.val0) pairs of L.n items by the
// low `bits` bits of the keys (8 bits per pass, through key1 / val1): the
// values in key order go to out, the keys (optional) to keys_out.
int radix_sort_pairs(const ClassSortLayout& L, int bits, uint32_t* out,
                     uint64_t* keys_out, hipStream_t s);

__global__ void k_fill_u32(uint32_t* p, int64_t n, uint32_t v);
__global__ void k_status_set(uint32_t bits, uint32_t* status);

}  // namespace chopper
