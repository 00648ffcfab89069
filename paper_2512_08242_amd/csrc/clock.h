// Per-GPU clock transform on the device (Section III-B alignment): shared by
// the alignment of records and markers and of kernel dispatch times.
#pragma once

#include "common.h"

namespace chopper {

struct ClockDev {
  int64_t x0, c, d;
};

// t + c + floor((t - x0) * d / 2^48): the signed 128-bit product is formed
// from __mul64hi and the low 64-bit product; the floor division by 2^48 is
// the arithmetic shift of that 128-bit value.
__device__ inline int64_t align_time(int64_t t, ClockDev k) {
  const int64_t u = t - k.x0;
  const int64_t hi = __mul64hi(u, k.d);
  const uint64_t lo = (uint64_t)u * (uint64_t)k.d;
  const int64_t q = (int64_t)(((uint64_t)hi << 16) | (lo >> 48));
  return t + k.c + q;
}

__device__ inline bool out_of_range(int64_t t) {
  const int64_t lim = (int64_t)1 << 62;
  return t >= lim || t <= -lim;
}

}  // namespace chopper
