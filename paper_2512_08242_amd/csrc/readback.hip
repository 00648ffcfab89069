// Host read-back of small device values through pinned memory.
#include "common.h"

namespace chopper {

namespace {

constexpr size_t kReadBackCap = 4096;

// one block: words [0, n) of src into host memory, then a system-scope
// fence so that the host sees them once the kernel has finished
__global__ __launch_bounds__(1024) void k_read_back(const uint32_t* src,
                                                    uint32_t* dst, int n) {
  for (int i = (int)threadIdx.x; i < n; i += (int)blockDim.x) dst[i] = src[i];
  __threadfence_system();
}

struct PinnedBuf {
  void* host = nullptr;
  void* dev = nullptr;
};

}  // namespace

hipError_t read_back(const void* dev, void* host, size_t bytes,
                     hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  if (bytes > kReadBackCap || bytes % 4 != 0) return hipErrorInvalidValue;
  thread_local PinnedBuf buf;
  if (!buf.host) {
    hipError_t e = hipHostMalloc(&buf.host, kReadBackCap,
                                 hipHostMallocPortable | hipHostMallocMapped);
    if (e != hipSuccess) {
      buf.host = nullptr;
      return e;
    }
    e = hipHostGetDevicePointer(&buf.dev, buf.host, 0);
    if (e != hipSuccess) return e;
  }
  hipError_t e = launch("read_back", k_read_back, dim3(1), dim3(1024), s,
                        (const uint32_t*)dev, (uint32_t*)buf.dev,
                        (int)(bytes / 4));
  if (e != hipSuccess) return e;
  // poll instead of the runtime's blocking wait, whose wake-up takes tens
  // of microseconds
  while ((e = hipStreamQuery(s)) == hipErrorNotReady) {
  }
  if (e != hipSuccess) return e;
  memcpy(host, buf.host, bytes);
  return hipSuccess;
}

}  // namespace chopper
