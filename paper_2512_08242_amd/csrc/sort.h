// Stable (class, time) sorts shared by chopper_align (record orders) and
// chopper_attribute (marker index).
#pragma once

#include "common.h"

namespace chopper {

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
  __device__ int64_t time(int64_t i) const { return t[i]; }
  __device__ uint32_t major(int64_t i) const { return gpu[i]; }
  __host__ __device__ int nclass() const { return C; }
};

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
  __device__ int64_t time(int64_t i) const { return t[i]; }
  __device__ uint32_t major(int64_t i) const { return gpu[i]; }
  __host__ __device__ int nclass() const { return C; }
};

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
};

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
// time-ordered; -1: unknown, checked here.  May synchronize `s`.
template <typename Acc>
int class_sort(const Acc& acc, const ClassSortLayout& L, uint32_t* out,
               uint32_t* coff, bool* range_error, hipStream_t s,
               int known_sorted);

// Both class partitions of the same n > 0 items at once, for input ordered
// by (major, time) (so the partitions are the stable sorts); needs
// a.nclass() + b.nclass() <= 256.
template <typename AccA, typename AccB>
int class_sort2(const AccA& a, const AccB& b, const ClassSortLayout& L,
                uint32_t* outA, uint32_t* coffA, uint32_t* outB,
                uint32_t* coffB, hipStream_t s);

// Stable LSD radix sort of the (L.key0, L.val0) pairs of L.n items by the
// low `bits` bits of the keys (8 bits per pass, through key1 / val1): the
// values in key order go to out, the keys (optional) to keys_out.
int radix_sort_pairs(const ClassSortLayout& L, int bits, uint32_t* out,
                     uint64_t* keys_out, hipStream_t s);

__global__ void k_fill_u32(uint32_t* p, int64_t n, uint32_t v);
__global__ void k_status_set(uint32_t bits, uint32_t* status);

}  // namespace chopper
