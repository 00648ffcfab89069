// Shared device primitives and host plumbing of libchopper (gfx950).
//
// Wave64 scans are built on __shfl_up (DPP / ds_bpermute underneath); block
// scans combine the per-wave totals through LDS.  All integer work, so every
// reduction is order-independent and exact.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include "../../include/chopper.h"

namespace chopper {

constexpr int kWave = 64;
constexpr int kBlock = 256;               // threads per block, 4 waves
constexpr int kWavesPerBlock = kBlock / kWave;
constexpr uint32_t kNone = 0xFFFFFFFFu;
constexpr int64_t kI64Max = INT64_MAX;
constexpr int64_t kI64Min = INT64_MIN;

__host__ __device__ inline int kind_of(uint32_t cls) {
  return (cls == 5u || cls == 6u) ? 1 : 0;
}

__host__ __device__ inline int64_t ceil_div(int64_t a, int64_t b) {
  return (a + b - 1) / b;
}

// ---------------------------------------------------------------------------
// Wave and block scans
// ---------------------------------------------------------------------------
struct OpAdd {
  template <typename T>
  __device__ T operator()(T a, T b) const { return a + b; }
};
struct OpMin {
  template <typename T>
  __device__ T operator()(T a, T b) const { return a < b ? a : b; }
};
struct OpMax {
  template <typename T>
  __device__ T operator()(T a, T b) const { return a > b ? a : b; }
};

template <typename T>
__device__ inline T shfl_up(T v, int d) {
  return __shfl_up(v, d, kWave);
}

// Inclusive scan across the 64 lanes of a wave.
template <typename T, typename Op>
__device__ inline T wave_inclusive(T v, Op op) {
  const int lane = threadIdx.x & (kWave - 1);
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    T u = shfl_up(v, d);
    if (lane >= d) v = op(u, v);
  }
  return v;
}

// Block-wide exclusive scan (kBlock threads).  `identity` is the value of the
// empty prefix; returns the exclusive value and writes the block total.
template <typename T, typename Op>
__device__ inline T block_exclusive(T v, Op op, T identity, T* total) {
  __shared__ T wave_tot[kWavesPerBlock];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  T inc = wave_inclusive(v, op);
  if (lane == kWave - 1) wave_tot[w] = inc;
  __syncthreads();
  T pre = identity;
  T tot = identity;
#pragma unroll
  for (int i = 0; i < kWavesPerBlock; ++i) {
    if (i < w) pre = op(pre, wave_tot[i]);
    tot = op(tot, wave_tot[i]);
  }
  T prev = shfl_up(inc, 1);                // inclusive value of lane - 1
  T exc = (lane == 0) ? pre : op(pre, prev);
  __syncthreads();
  if (total) *total = tot;
  return exc;
}

// Pair scanned lexicographically by (seg, val) with max: the running maximum
// restricted to the last segment seen, since segment ids never decrease along
// a scan.
struct SegMax {
  uint32_t seg;
  int64_t val;
};
struct OpSegMax {
  __device__ SegMax operator()(SegMax a, SegMax b) const {
    if (a.seg != b.seg) return a.seg > b.seg ? a : b;
    return a.val >= b.val ? a : b;
  }
};
template <>
__device__ inline SegMax shfl_up<SegMax>(SegMax v, int d) {
  SegMax r;
  r.seg = __shfl_up(v.seg, d, kWave);
  r.val = __shfl_up(v.val, d, kWave);
  return r;
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
#define CHOPPER_HIP(x)                      \
  do {                                      \
    hipError_t e_ = (x);                    \
    if (e_ != hipSuccess) return CHOPPER_EHIP; \
  } while (0)

// Carves 256-byte-aligned sub-buffers out of the caller's scratch.  With a
// null base it only measures.
struct Scratch {
  char* base;
  size_t used = 0;
  explicit Scratch(void* b) : base(static_cast<char*>(b)) {}
  template <typename T>
  T* take(int64_t count) {
    size_t bytes = (size_t)(count > 0 ? count : 1) * sizeof(T);
    size_t off = (used + 255) & ~(size_t)255;
    used = off + bytes;
    return base ? reinterpret_cast<T*>(base + off) : nullptr;
  }
};

// Scratch protocol shared by all entry points: returns 1 when the call was a
// size query (already answered), 0 when the caller's buffer is large enough,
// or a negative code.
inline int scratch_check(void* scratch, size_t* scratch_bytes, size_t need) {
  if (!scratch_bytes) return CHOPPER_EINVAL;
  if (!scratch) { *scratch_bytes = need; return 1; }
  if (*scratch_bytes < need) return CHOPPER_ESCRATCH;
  if (((uintptr_t)scratch & 255) != 0) return CHOPPER_EINVAL;
  return 0;
}

// Kernel timing hook (chopper_time_kernel).
struct TimerHook {
  const char* name = nullptr;
  hipEvent_t start = nullptr, stop = nullptr;
};
TimerHook& timer_hook();

template <typename Kern, typename... Args>
inline hipError_t launch(const char* name, Kern kern, dim3 grid, dim3 block,
                         hipStream_t s, Args... args) {
  if (grid.x == 0 || grid.y == 0 || grid.z == 0) return hipSuccess;
  TimerHook& h = timer_hook();
  bool timed = h.name && strcmp(h.name, name) == 0;
  if (timed) (void)hipEventRecord(h.start, s);
  hipLaunchKernelGGL(kern, grid, block, 0, s, args...);
  hipError_t e = hipGetLastError();
  if (timed) (void)hipEventRecord(h.stop, s);
  return e;
}

// Copies `bytes` of device memory at `dev` to `host` once the work queued
// on `s` before it is done, and returns when they are there (polling, not
// the runtime's blocking wait).
hipError_t read_back(const void* dev, void* host, size_t bytes, hipStream_t s);

// The same in two halves: read_back_start queues the copy (at most
// kReadBackMax bytes) into pinned memory that the library keeps and records
// an event after it; work queued on `s` afterwards runs while the host
// waits in read_back_finish, which polls that event only and then copies
// the value to `host`.  Every start is followed by one finish on the same
// host thread.  Without a free pinned slot the copy is done at once by
// read_back_start (the stream drained), and the finish only hands it over.
// A read-back left unfinished (an early error return) waits for its copy
// and frees its slot when it goes out of scope.
constexpr size_t kReadBackMax = 256;
struct ReadBack {
  void* slot = nullptr;
  size_t bytes = 0;
  hipError_t err = hipSuccess;
  alignas(8) unsigned char now[kReadBackMax];
  ReadBack() = default;
  ReadBack(const ReadBack&) = delete;
  ReadBack& operator=(const ReadBack&) = delete;
  ~ReadBack();
};
hipError_t read_back_start(const void* dev, size_t bytes, hipStream_t s,
                           ReadBack* rb);
hipError_t read_back_finish(ReadBack* rb, void* host);

// the same as launch() with `shm` bytes of dynamic LDS
template <typename Kern, typename... Args>
inline hipError_t launch_shm(const char* name, Kern kern, dim3 grid,
                             dim3 block, size_t shm, hipStream_t s,
                             Args... args) {
  if (grid.x == 0 || grid.y == 0 || grid.z == 0) return hipSuccess;
  TimerHook& h = timer_hook();
  bool timed = h.name && strcmp(h.name, name) == 0;
  if (timed) (void)hipEventRecord(h.start, s);
  hipLaunchKernelGGL(kern, grid, block, shm, s, args...);
  hipError_t e = hipGetLastError();
  if (timed) (void)hipEventRecord(h.stop, s);
  return e;
}

inline dim3 grid_for(int64_t items, int per_block) {
  int64_t b = ceil_div(items, per_block);
  return dim3((unsigned)(b > 0 ? b : 0));
}

// ---------------------------------------------------------------------------
// Device-wide exclusive scans (three passes: tile totals, scan of totals in
// one block, rescan of each tile with its prefix).
// ---------------------------------------------------------------------------
int64_t scan_scratch_elems(int64_t n);   // number of T slots needed
template <typename T>
hipError_t exclusive_scan(const T* in, T* out, int64_t n, T* tmp, T* total,
                          hipStream_t s);
// the same over the first min(n, *n_dev) elements (n_dev on the device)
template <typename T>
hipError_t exclusive_scan(const T* in, T* out, int64_t n, const uint32_t* n_dev,
                          T* tmp, T* total, hipStream_t s);

// Sorts (key u64) stably and writes the permutation of 0..n-1.
// Implemented in sort.hip.
struct SortPlan;

}  // namespace chopper
