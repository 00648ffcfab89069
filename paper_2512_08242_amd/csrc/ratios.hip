// Derived metrics of aggregated rows (paper Section III-C: metrics derived
// from several counters and the kernel duration, e.g. bandwidth; eq. 10:
// peak-clock duration = cycles / peak frequency), plus the ABI's small
// utilities.  Built without fast-math and with contraction off: every value
// is IEEE double arithmetic in the documented order.
#include "common.h"

namespace chopper {

TimerHook& timer_hook() {
  static TimerHook h;
  return h;
}

static const char* const kKernelNames[] = {
    "align_transform_records", "align_transform_markers", "align_fill",
    "align_dense_classes", "sort_class_hist", "sort_class_partition",
    "sort_class_verify", "sort_class_offsets", "sort_digit_hist",
    "sort_digit_scatter", "sort_make_keys", "sort_time_minmax",
    "attr_marker_gather", "attr_marker_links", "attr_records",
    "ov_runs_fixup", "ov_runs_spine", "ov_runs_count", "ov_runs_write",
    "ov_runs_inc_spine", "ov_runs_comm_overlap", "ov_records", "ov_markers",
    "ov_gpus", "ov_gap",
    "agg_fill_owner", "agg_elect", "agg_count", "agg_offsets", "agg_assign",
    "agg_reduce_records", "agg_reduce_rows", "agg_apply_overflow",
    "agg_zero_rows", "agg_zero", "scan_reduce", "scan_spine", "scan_down",
    "ratios_rows", "ratios_windows", "sort_fill", "sort_init_minmax",
    "sort_class_count", "status_set", "ov_fill",
    "agg_workload_first", "sort_major_sorted", "agg_heads_records",
    "agg_heads_rows", "agg_fast_reduce_records", "agg_fast_reduce_rows",
    "agg_workload_from_gpu", "bi_params", "bi_clear", "bi_fill",
    "bi_fixup", "ov_comm_records", "agg_nat_init", "agg_nat_pre",
    "agg_nat_tiles", "agg_heads_nat", "agg_gpu_rows",
    "agg_exact_keys", "join_resort", "attr_windows", "agg_items",
    "view_flags", "view_units", "view_fill", "view_records", "view_rows",
    "view_iter_max", "view_medians", "launch_split", "join_fill",
    "join_labels", "join_heads", "join_runs", "join_order", "join_pass_prep",
    "join_dense", "join_match", "join_gather", "stats_clear", "stats_keys",
    "stats_offsets", "stats_scatter", "stats_pass", "stats_select",
    "stats_final"};

__global__ __launch_bounds__(kBlock) void k_ratios(
    const int64_t* level_offset, int depth, int64_t cap, const uint64_t* n,
    const int64_t* dur, const int64_t* ovl, const uint64_t* ctr, int nc,
    double fpeak, double* out) {
  int64_t total = level_offset[depth + 2];
  if (total > cap) total = cap;
  const int64_t r = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (r >= total) return;
  const double d = (double)dur[r];
  out[r] = (double)ovl[r] / d;
  if (nc >= 16) {
    const uint64_t cyc = ctr[0 * cap + r];
    const uint64_t mfma = ctr[1 * cap + r];
    const uint64_t rw = ctr[4 * cap + r] + ctr[5 * cap + r];
    const uint64_t sclk = ctr[13 * cap + r];
    const double dpeak = (double)cyc * 1000.0 / fpeak;
    out[1 * cap + r] = (double)rw / d;
    out[2 * cap + r] = (double)sclk / (double)n[r];
    out[3 * cap + r] = (double)mfma / (double)cyc;
    out[4 * cap + r] = dpeak;
    out[5 * cap + r] = d / dpeak;
  } else {
    const double nan = __builtin_nan("");
    for (int z = 1; z < 6; ++z) out[z * cap + r] = nan;
  }
}

__global__ __launch_bounds__(kBlock) void k_window_fractions(int64_t nw,
                                                             const int64_t* w,
                                                             double* out) {
  const int64_t j = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (j >= nw) return;
  const int64_t len = w[4 * j] + w[4 * j + 1] + w[4 * j + 2] + w[4 * j + 3];
  for (int z = 0; z < 4; ++z) out[4 * j + z] = (double)w[4 * j + z] / (double)len;
}

}  // namespace chopper

using namespace chopper;

extern "C" int chopper_ratios(const chopper_rows* rows, int32_t depth,
                              int32_t n_counters, double freq_peak_mhz,
                              double* out, void* stream) {
  if (!rows || !out || !rows->level_offset || depth < 0 || depth > 8 ||
      n_counters < 0 || n_counters > 16 || rows->cap < 0)
    return CHOPPER_EINVAL;
  if (rows->cap == 0) return CHOPPER_OK;
  if (!rows->n || !rows->dur || !rows->ovl || (n_counters > 0 && !rows->ctr))
    return CHOPPER_EINVAL;
  CHOPPER_HIP(launch("ratios_rows", k_ratios, grid_for(rows->cap, kBlock),
                     dim3(kBlock), (hipStream_t)stream,
                     (const int64_t*)rows->level_offset, (int)depth, rows->cap,
                     (const uint64_t*)rows->n, (const int64_t*)rows->dur,
                     (const int64_t*)rows->ovl, (const uint64_t*)rows->ctr,
                     (int)n_counters, freq_peak_mhz, out));
  return CHOPPER_OK;
}

extern "C" int chopper_window_fractions(int64_t n, const int64_t* win,
                                        double* out, void* stream) {
  if (n < 0 || (n > 0 && (!win || !out))) return CHOPPER_EINVAL;
  if (n == 0) return CHOPPER_OK;
  CHOPPER_HIP(launch("ratios_windows", k_window_fractions, grid_for(n, kBlock),
                     dim3(kBlock), (hipStream_t)stream, n, win, out));
  return CHOPPER_OK;
}

extern "C" const char* chopper_strerror(int code) {
  switch (code) {
    case CHOPPER_OK: return "ok";
    case CHOPPER_EINVAL: return "invalid argument";
    case CHOPPER_ESCRATCH: return "scratch buffer too small";
    case CHOPPER_EOVERFLOW: return "clock fit outside its exact range";
    case CHOPPER_EHIP: return "HIP runtime error";
    default: return "unknown error";
  }
}

extern "C" int chopper_version(void) { return 100; }

extern "C" const char* chopper_kernel_name(int i) {
  const int n = (int)(sizeof(kKernelNames) / sizeof(kKernelNames[0]));
  return (i >= 0 && i < n) ? kKernelNames[i] : nullptr;
}

extern "C" int chopper_time_kernel(const char* name, void* start_event,
                                   void* stop_event) {
  TimerHook& h = timer_hook();
  if (!name) {
    h.name = nullptr;
    return CHOPPER_OK;
  }
  if (!start_event || !stop_event) return CHOPPER_EINVAL;
  for (int i = 0; chopper_kernel_name(i); ++i) {
    if (strcmp(chopper_kernel_name(i), name) == 0) {
      h.name = chopper_kernel_name(i);
      h.start = (hipEvent_t)start_event;
      h.stop = (hipEvent_t)stop_event;
      return CHOPPER_OK;
    }
  }
  return CHOPPER_EINVAL;
}
