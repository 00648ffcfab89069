// Host read-back of small device values (flags and counts that size later
// launches), in two halves so that the caller can queue more work on the
// stream before it waits: a one-wave kernel on the stream stores the words
// into a slot of pinned host memory (mapped for the device; a runtime copy
// there would go through the copy engine, which later kernels of the stream
// wait for), an event is recorded after it, and the wait polls that event.
// The slots (a few per device, each with its event) are created on first
// use and kept for the life of the process; when none is free, or pinned
// memory cannot be had, the read-back is done at once into the caller's
// memory, waiting for the whole stream.
#include <chrono>
#include <cstring>
#include <mutex>

#include "common.h"

namespace chopper {

namespace {

// a stream that has not drained after this long is reported as an error
constexpr double kReadBackLimitSeconds = 120.0;
constexpr int kRbDevices = 64;
constexpr int kRbSlots = 4;
static_assert(kReadBackMax / 4 <= kWave, "one word per lane");

struct RbSlot {
  void* pin = nullptr;
  uint32_t* dpin = nullptr;   // its device address
  hipEvent_t ev = nullptr;
  bool busy = false;
  bool failed = false;   // creation failed: never used
};

std::mutex g_rb_mu;
RbSlot g_rb[kRbDevices][kRbSlots];

// Polls until `done` stops returning hipErrorNotReady, within the limit.
template <typename F>
hipError_t poll(F done) {
  hipError_t e;
  const auto t0 = std::chrono::steady_clock::now();
  while ((e = done()) == hipErrorNotReady) {
    const std::chrono::duration<double> dt =
        std::chrono::steady_clock::now() - t0;
    if (dt.count() > kReadBackLimitSeconds) return hipErrorLaunchTimeOut;
  }
  return e;
}

// the synchronous read-back: the copy, then the whole stream drained
hipError_t read_now(const void* dev, void* host, size_t bytes, hipStream_t s) {
  hipError_t e = hipMemcpyAsync(host, dev, bytes, hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return e;
  return poll([&] { return hipStreamQuery(s); });
}

// a free slot of the current device (created on first use), or null
RbSlot* take_slot() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kRbDevices)
    return nullptr;
  std::lock_guard<std::mutex> lk(g_rb_mu);
  for (int i = 0; i < kRbSlots; ++i) {
    RbSlot& q = g_rb[dev][i];
    if (q.busy || q.failed) continue;
    if (!q.pin) {
      if (hipHostMalloc(&q.pin, kReadBackMax, hipHostMallocDefault) !=
          hipSuccess) {
        q.pin = nullptr;
        q.failed = true;
        continue;
      }
      void* dp = nullptr;
      if (hipHostGetDevicePointer(&dp, q.pin, 0) != hipSuccess ||
          hipEventCreateWithFlags(&q.ev, hipEventDisableTiming) !=
              hipSuccess) {
        (void)hipHostFree(q.pin);
        q.pin = nullptr;
        q.ev = nullptr;
        q.failed = true;
        continue;
      }
      q.dpin = static_cast<uint32_t*>(dp);
    }
    q.busy = true;
    return &q;
  }
  return nullptr;
}

void give_slot(RbSlot* q) {
  std::lock_guard<std::mutex> lk(g_rb_mu);
  q->busy = false;
}

// the words of a read-back, one per lane, into the pinned slot
__global__ __launch_bounds__(kWave) void k_put_host(const uint32_t* src,
                                                    uint32_t* dst, int nw) {
  const int i = (int)threadIdx.x;
  if (i < nw) dst[i] = src[i];
  // visible to the host before the kernel (and the event after it) ends
  __threadfence_system();
}

}  // namespace

hipError_t read_back_start(const void* dev, size_t bytes, hipStream_t s,
                           ReadBack* rb) {
  rb->slot = nullptr;
  rb->bytes = bytes;
  rb->err = hipSuccess;
  if (bytes == 0) return hipSuccess;
  if (bytes > kReadBackMax) return hipErrorInvalidValue;
  // whole aligned words only (every caller's case); others read now
  RbSlot* q = (bytes % 4 == 0 && ((uintptr_t)dev & 3) == 0) ? take_slot()
                                                              : nullptr;
  if (!q) {
    // no slot: read now into the inline buffer
    rb->err = read_now(dev, rb->now, bytes, s);
    return rb->err;
  }
  hipError_t e = launch("read_back", k_put_host, dim3(1), dim3(kWave), s,
                        static_cast<const uint32_t*>(dev), q->dpin,
                        (int)(bytes / 4));
  if (e == hipSuccess) e = hipEventRecord(q->ev, s);
  if (e != hipSuccess) {
    give_slot(q);
    return e;
  }
  rb->slot = q;
  return hipSuccess;
}

hipError_t read_back_finish(ReadBack* rb, void* host) {
  if (rb->bytes == 0) return hipSuccess;
  RbSlot* q = static_cast<RbSlot*>(rb->slot);
  if (!q) {
    if (rb->err == hipSuccess) std::memcpy(host, rb->now, rb->bytes);
    return rb->err;
  }
  const hipError_t e = poll([&] { return hipEventQuery(q->ev); });
  if (e == hipSuccess) std::memcpy(host, q->pin, rb->bytes);
  rb->slot = nullptr;
  give_slot(q);
  return e;
}

ReadBack::~ReadBack() {
  if (!slot) return;
  RbSlot* q = static_cast<RbSlot*>(slot);
  // the copy into the slot may still be queued: wait for it before the
  // slot can be taken again
  (void)poll([&] { return hipEventQuery(q->ev); });
  give_slot(q);
}

hipError_t read_back(const void* dev, void* host, size_t bytes,
                     hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  if (bytes > kReadBackMax) return read_now(dev, host, bytes, s);
  ReadBack rb;
  hipError_t e = read_back_start(dev, bytes, s, &rb);
  if (e != hipSuccess) return e;
  return read_back_finish(&rb, host);
}

}  // namespace chopper
