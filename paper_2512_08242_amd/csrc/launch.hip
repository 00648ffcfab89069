// chopper_launch_split: launch overhead split into preparation and call
// overhead (Section V-D eqs. 1-3) from the kernels' dispatch times.
//
// The bubble before a compute kernel is the sum of the two parts, so with
// the bubble already known (chopper_overlap) the split is elementwise: when
// the bubble g is positive the previous compute kernel of the stream ended at
// s' - g, preparation is the dispatch time past that end (at most g) and the
// call overhead the rest.  One wave tile of records per wave, loads striped
// across the lanes and all issued before any use; the clock table sits in
// LDS.
#include <mutex>
#include <vector>

#include "clock.h"
#include "wave.h"

// Scratch of chopper_launch_split_noalloc: the clock table of up to 256 GPUs
// (6 KiB).  Every device the library runs on holds its own copy until the
// process ends.  Host code never passes this name to a kernel or a copy (on
// the host it is only a stand-in for the symbol); it uses the device address
// that static_scratch() looks up once per device.
static __device__ __align__(256) chopper::ClockDev scratch[256];

namespace chopper {

bool validate_records(const chopper_records* r);

namespace {

constexpr int kMaxGpus = 256;
static_assert(sizeof(::scratch) == kMaxGpus * sizeof(ClockDev),
              "the static clock table holds kMaxGpus entries");

__global__ __launch_bounds__(kBlock) void k_launch_split(
    int64_t n, int G, const uint8_t* gpu, const ClockDev* clk,
    const int64_t* launch, const int64_t* start, const int64_t* gap,
    int64_t* prep, int64_t* call, uint32_t* status) {
  __shared__ ClockDev s_clk[kMaxGpus];
  for (int g = (int)threadIdx.x; g < G; g += kBlock) s_clk[g] = clk[g];
  __syncthreads();
  const int lane = lane_id(), wv = (int)(threadIdx.x / kWave);
  const int64_t base =
      ((int64_t)blockIdx.x * kWavesPerBlock + wv) * (int64_t)kWaveTile;
  if (base >= n) return;
  // striped items (j * 64 + lane): every load of the tile in flight at once
  uint32_t g[kTileIpt];
  int64_t tl[kTileIpt], s[kTileIpt], gp[kTileIpt];
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const int64_t k = base + (int64_t)j * kWave + lane;
    const bool v = k < n;
    g[j] = v ? gpu[k] : 0u;
    tl[j] = v ? launch[k] : 0;
    s[j] = v ? start[k] : 0;
    gp[j] = v ? gap[k] : 0;
  }
  uint32_t bad = 0;
#pragma unroll
  for (int j = 0; j < kTileIpt; ++j) {
    const int64_t k = base + (int64_t)j * kWave + lane;
    if (k >= n) continue;
    int64_t p = 0;
    if (g[j] >= (uint32_t)G) {
      bad |= CHOPPER_ST_BAD_GPU;
    } else {
      const int64_t t2 = align_time(tl[j], s_clk[g[j]]);
      if (out_of_range(tl[j]) || out_of_range(t2)) bad |= CHOPPER_ST_RANGE;
      if (gp[j] > 0) {
        const int64_t past = t2 - (s[j] - gp[j]);
        p = past <= 0 ? 0 : (past < gp[j] ? past : gp[j]);
      }
    }
    prep[k] = p;
    call[k] = gp[j] > 0 ? gp[j] - p : 0;
  }
  uint32_t v = bad;
  for (int d = kWave / 2; d > 0; d >>= 1) v |= __shfl_xor(v, d, kWave);
  if (lane == 0 && v) atomicOr(status, v);
}

constexpr int kMaxDevices = 64;

// Device address of `scratch` on the current device, looked up on the first
// call made on that device.  The caller's stream must belong to the current
// device (hipErrorInvalidDevice otherwise).
hipError_t static_scratch(hipStream_t s, ClockDev** out) {
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  if (s != nullptr) {
    hipDevice_t sdev = -1;
    e = hipStreamGetDevice(s, &sdev);
    if (e != hipSuccess) return e;
    if ((int)sdev != dev) return hipErrorInvalidDevice;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(::scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *out = static_cast<ClockDev*>(addr[dev]);
  return hipSuccess;
}

}  // namespace

extern "C" int chopper_launch_split(const chopper_records* rec,
                                    const chopper_clock* clocks,
                                    const int64_t* launch_ns,
                                    const int64_t* start_al,
                                    const int64_t* gap, int64_t* prep_out,
                                    int64_t* call_out, void* scratch,
                                    size_t* scratch_bytes, uint32_t* status,
                                    void* stream) {
  if (!validate_records(rec) || !clocks || !scratch_bytes)
    return CHOPPER_EINVAL;
  const int64_t n = rec->n;
  const int G = rec->n_gpus;
  if (n > 0 && (!rec->gpu || !launch_ns || !start_al || !gap || !prep_out ||
                !call_out))
    return CHOPPER_EINVAL;
  Scratch probe(nullptr);
  probe.take<ClockDev>(G);
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  if (n == 0) return CHOPPER_OK;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  ClockDev* clk = sc.take<ClockDev>(G);
  std::vector<ClockDev> cd(G);
  for (int g = 0; g < G; ++g)
    cd[g] = ClockDev{clocks[g].x0, clocks[g].c, clocks[g].d_q48};
  // (a copy from pageable memory is staged before the call returns)
  CHOPPER_HIP(hipMemcpyAsync(clk, cd.data(), sizeof(ClockDev) * G,
                             hipMemcpyHostToDevice, s));
  CHOPPER_HIP(launch("launch_split", k_launch_split,
                     dim3((unsigned)ceil_div(n, (int64_t)kWaveTile *
                                                    kWavesPerBlock)),
                     dim3(kBlock), s, n, G, rec->gpu, (const ClockDev*)clk,
                     launch_ns, start_al, gap, prep_out, call_out, status));
  return CHOPPER_OK;
}


// Allocation-free variant: the clock table lives in the library's static
// device array instead of the caller's scratch.  No hipMalloc, hipFree or
// other allocating call; the host side builds the table on its stack.
extern "C" int chopper_launch_split_noalloc(const chopper_records* rec,
                                            const chopper_clock* clocks,
                                            const int64_t* launch_ns,
                                            const int64_t* start_al,
                                            const int64_t* gap,
                                            int64_t* prep_out,
                                            int64_t* call_out,
                                            uint32_t* status, void* stream) {
  if (!validate_records(rec) || !clocks || !status) return CHOPPER_EINVAL;
  const int64_t n = rec->n;
  const int G = rec->n_gpus;
  if (n > 0 && (!rec->gpu || !launch_ns || !start_al || !gap || !prep_out ||
                !call_out))
    return CHOPPER_EINVAL;
  // the static table holds the clocks of at most kMaxGpus GPUs
  if (G < 1 || G > kMaxGpus) return CHOPPER_ESCRATCH;
  if (n == 0) return CHOPPER_OK;
  hipStream_t s = (hipStream_t)stream;
  ClockDev* clk = nullptr;
  CHOPPER_HIP(static_scratch(s, &clk));
  ClockDev cd[kMaxGpus];
  for (int g = 0; g < G; ++g)
    cd[g] = ClockDev{clocks[g].x0, clocks[g].c, clocks[g].d_q48};
  // every entry the kernel reads (0 .. G-1) is written here, so nothing left
  // by an earlier call is read; a copy from pageable memory is staged before
  // the call returns
  CHOPPER_HIP(hipMemcpyAsync(clk, cd, sizeof(ClockDev) * G,
                             hipMemcpyHostToDevice, s));
  CHOPPER_HIP(launch("launch_split", k_launch_split,
                     dim3((unsigned)ceil_div(n, (int64_t)kWaveTile *
                                                    kWavesPerBlock)),
                     dim3(kBlock), s, n, G, rec->gpu, (const ClockDev*)clk,
                     launch_ns, start_al, gap, prep_out, call_out, status));
  return CHOPPER_OK;
}

}  // namespace chopper
