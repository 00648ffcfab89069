// Host read-back of small device values (flags and counts that size later
// launches).  The copy goes straight into the caller's host memory; the
// library owns no host or device buffer for it.
#include <chrono>

#include "common.h"

namespace chopper {

namespace {

// a stream that has not drained after this long is reported as an error
constexpr double kReadBackLimitSeconds = 120.0;

}  // namespace

hipError_t read_back(const void* dev, void* host, size_t bytes,
                     hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  hipError_t e = hipMemcpyAsync(host, dev, bytes, hipMemcpyDeviceToHost, s);
  if (e != hipSuccess) return e;
  // poll instead of the runtime's blocking wait, whose wake-up takes tens
  // of microseconds; bounded, so that a stream that never drains returns
  const auto t0 = std::chrono::steady_clock::now();
  while ((e = hipStreamQuery(s)) == hipErrorNotReady) {
    const std::chrono::duration<double> dt =
        std::chrono::steady_clock::now() - t0;
    if (dt.count() > kReadBackLimitSeconds) return hipErrorLaunchTimeOut;
  }
  return e;
}

}  // namespace chopper
