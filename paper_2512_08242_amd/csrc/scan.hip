// Device-wide exclusive prefix sums (reduce-then-scan).
//
// Pass 1 sums each tile of kScanTile elements, pass 2 scans the tile sums in
// a single block, pass 3 rescans every tile starting from its prefix.  Each
// thread owns kScanIpt consecutive elements, so the block-level scan is paid
// once per kScanIpt elements.
#include "common.h"

namespace chopper {

constexpr int kScanIpt = 8;
constexpr int kScanTile = kBlock * kScanIpt;

int64_t scan_scratch_elems(int64_t n) { return ceil_div(n, kScanTile) + 1; }

// n_dev (optional): the element count held on the device, at most n
__device__ inline int64_t scan_len(int64_t n, const uint32_t* n_dev) {
  if (!n_dev) return n;
  const int64_t m = (int64_t)*n_dev;
  return m < n ? m : n;
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_scan_reduce(const T* in, int64_t n,
                                                        const uint32_t* n_dev,
                                                        T* tile_sum) {
  n = scan_len(n, n_dev);
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  if (base >= n) {               // whole block: an empty tile
    if (threadIdx.x == 0) tile_sum[blockIdx.x] = 0;
    return;
  }
  T acc = 0;
  for (int j = 0; j < kScanIpt; ++j) {
    int64_t i = base + (int64_t)j * kBlock + threadIdx.x;
    if (i < n) acc += in[i];
  }
  T tot;
  block_exclusive(acc, OpAdd(), (T)0, &tot);
  if (threadIdx.x == 0) tile_sum[blockIdx.x] = tot;
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_scan_spine(T* tile_sum,
                                                       int64_t ntiles,
                                                       T* total) {
  T carry = 0;
  for (int64_t base = 0; base < ntiles; base += kScanTile) {
    T v[kScanIpt];
    T acc = 0;
    for (int j = 0; j < kScanIpt; ++j) {
      int64_t i = base + (int64_t)threadIdx.x * kScanIpt + j;
      v[j] = (i < ntiles) ? tile_sum[i] : (T)0;
      acc += v[j];
    }
    T tot;
    T pre = block_exclusive(acc, OpAdd(), (T)0, &tot) + carry;
    for (int j = 0; j < kScanIpt; ++j) {
      int64_t i = base + (int64_t)threadIdx.x * kScanIpt + j;
      if (i < ntiles) tile_sum[i] = pre;
      pre += v[j];
    }
    carry += tot;
  }
  if (threadIdx.x == 0 && total) *total = carry;
}

template <typename T>
__global__ __launch_bounds__(kBlock) void k_scan_down(const T* in, T* out,
                                                      int64_t n,
                                                      const uint32_t* n_dev,
                                                      const T* tile_pre) {
  n = scan_len(n, n_dev);
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  if (base >= n) return;
  T v[kScanIpt];
  T acc = 0;
  for (int j = 0; j < kScanIpt; ++j) {
    int64_t i = base + (int64_t)threadIdx.x * kScanIpt + j;
    v[j] = (i < n) ? in[i] : (T)0;
    acc += v[j];
  }
  T tot;
  T pre = block_exclusive(acc, OpAdd(), (T)0, &tot) + tile_pre[blockIdx.x];
  for (int j = 0; j < kScanIpt; ++j) {
    int64_t i = base + (int64_t)threadIdx.x * kScanIpt + j;
    if (i < n) out[i] = pre;
    pre += v[j];
  }
}

// Rescan of a tile whose prefix is the sum of the tile sums before it,
// added up by the block itself (used when there are at most kDirectTiles
// tiles); the block holding the last element also writes the total.
constexpr int64_t kDirectTiles = 1024;
template <typename T>
__global__ __launch_bounds__(kBlock) void k_scan_down_direct(
    const T* in, T* out, int64_t n, const uint32_t* n_dev, const T* tile_sum,
    T* total) {
  n = scan_len(n, n_dev);
  const int64_t base = (int64_t)blockIdx.x * kScanTile;
  if (base >= n) {
    if (blockIdx.x == 0 && threadIdx.x == 0 && total) *total = 0;
    return;
  }
  T p = 0;
  for (int64_t i = threadIdx.x; i < (int64_t)blockIdx.x; i += kBlock)
    p += tile_sum[i];
  T prefix;
  block_exclusive(p, OpAdd(), (T)0, &prefix);
  T v[kScanIpt];
  T acc = 0;
  for (int j = 0; j < kScanIpt; ++j) {
    int64_t i = base + (int64_t)threadIdx.x * kScanIpt + j;
    v[j] = (i < n) ? in[i] : (T)0;
    acc += v[j];
  }
  T tot;
  T pre = block_exclusive(acc, OpAdd(), (T)0, &tot) + prefix;
  for (int j = 0; j < kScanIpt; ++j) {
    int64_t i = base + (int64_t)threadIdx.x * kScanIpt + j;
    if (i < n) out[i] = pre;
    pre += v[j];
  }
  if (base + kScanTile >= n && threadIdx.x == 0 && total)
    *total = prefix + tot;
}

template <typename T>
hipError_t exclusive_scan(const T* in, T* out, int64_t n, T* tmp, T* total,
                          hipStream_t s) {
  return exclusive_scan<T>(in, out, n, nullptr, tmp, total, s);
}

template <typename T>
hipError_t exclusive_scan(const T* in, T* out, int64_t n, const uint32_t* n_dev,
                          T* tmp, T* total, hipStream_t s) {
  int64_t ntiles = ceil_div(n, kScanTile);
  hipError_t e;
  if (n <= 0) {
    // total = 0
    e = launch("scan_spine", k_scan_spine<T>, dim3(1), dim3(kBlock), s, tmp,
               (int64_t)0, total);
    return e;
  }
  if (ntiles <= kDirectTiles) {
    // two passes (one for a single tile): each block adds up the tile sums
    // before it
    if (ntiles > 1) {
      e = launch("scan_reduce", k_scan_reduce<T>, dim3((unsigned)ntiles),
                 dim3(kBlock), s, in, n, n_dev, tmp);
      if (e != hipSuccess) return e;
    }
    return launch("scan_down", k_scan_down_direct<T>, dim3((unsigned)ntiles),
                  dim3(kBlock), s, in, out, n, n_dev, (const T*)tmp, total);
  }
  e = launch("scan_reduce", k_scan_reduce<T>, dim3((unsigned)ntiles),
             dim3(kBlock), s, in, n, n_dev, tmp);
  if (e != hipSuccess) return e;
  e = launch("scan_spine", k_scan_spine<T>, dim3(1), dim3(kBlock), s, tmp,
             ntiles, total);
  if (e != hipSuccess) return e;
  return launch("scan_down", k_scan_down<T>, dim3((unsigned)ntiles),
                dim3(kBlock), s, in, out, n, n_dev, (const T*)tmp);
}

template hipError_t exclusive_scan<int64_t>(const int64_t*, int64_t*, int64_t,
                                            const uint32_t*, int64_t*,
                                            int64_t*, hipStream_t);
template hipError_t exclusive_scan<uint32_t>(const uint32_t*, uint32_t*,
                                             int64_t, uint32_t*, uint32_t*,
                                             hipStream_t);
template hipError_t exclusive_scan<int64_t>(const int64_t*, int64_t*, int64_t,
                                            int64_t*, int64_t*, hipStream_t);
template hipError_t exclusive_scan<uint64_t>(const uint64_t*, uint64_t*,
                                             int64_t, uint64_t*, uint64_t*,
                                             hipStream_t);

}  // namespace chopper
