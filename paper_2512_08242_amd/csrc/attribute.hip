// chopper_attribute: every kernel record is assigned, level by level, to the
// annotation marker containing its aligned start (paper Section I
// granularities; III-A annotations for kernels, operations, layers and
// iterations).
//
// Markers are sorted by (gpu, level, empty, start') into contiguous
// per-(gpu, level) segments of non-empty markers.  Each non-empty marker
// also records the range of next-level markers that start inside it; the
// search for level l+1 then runs only over that range (plus the single
// marker just before it, which is the only other candidate), so a record
// pays log2 of the child count per level instead of log2 of the segment.
// The narrowed answer equals the full-segment answer for any sorted marker
// set, nested or not.
#include "sort.h"

namespace chopper {

bool validate_records(const chopper_records* r);
bool validate_markers(const chopper_markers* m);

// first index in [lo, hi) with a[i] > x
__device__ inline int64_t upper_bound_i64(const int64_t* a, int64_t lo,
                                          int64_t hi, int64_t x) {
  while (lo < hi) {
    int64_t mid = lo + ((hi - lo) >> 1);
    if (a[mid] <= x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// first index in [lo, hi) with a[i] >= x
__device__ inline int64_t lower_bound_i64(const int64_t* a, int64_t lo,
                                          int64_t hi, int64_t x) {
  while (lo < hi) {
    int64_t mid = lo + ((hi - lo) >> 1);
    if (a[mid] < x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// sorted marker columns
__global__ __launch_bounds__(kBlock) void k_marker_gather(
    int64_t nm, const uint32_t* mord, const int64_t* ms, const int64_t* me,
    int64_t* sms, int64_t* sme, uint32_t* sid) {
  int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (p >= nm) return;
  uint32_t j = mord[p];
  sms[p] = ms[j];
  sme[p] = me[j];
  sid[p] = j;
}

// overlap check between neighbours of a (gpu, level) segment, and the
// child range of every non-empty marker at the next level
__global__ __launch_bounds__(kBlock) void k_marker_links(
    int G, int D, const uint32_t* coff, const int64_t* sms, const int64_t* sme,
    uint32_t* clo, uint32_t* chi, uint32_t* status) {
  // one block column per (gpu, level) segment
  const int seg = blockIdx.y;          // g * D + l
  const int g = seg / D, l = seg % D;
  const uint32_t cls = (uint32_t)seg * 2u;
  const int64_t b = coff[cls], e = coff[cls + 1];
  int64_t cb = 0, ce = 0;
  if (l + 1 < D) {
    cb = coff[cls + 2];
    ce = coff[cls + 3];
  }
  (void)g;
  bool ov = false;
  for (int64_t p = b + (int64_t)blockIdx.x * kBlock + threadIdx.x; p < e;
       p += (int64_t)gridDim.x * kBlock) {
    if (p + 1 < e && sme[p] > sms[p + 1]) ov = true;
    if (l + 1 < D) {
      clo[p] = (uint32_t)lower_bound_i64(sms, cb, ce, sms[p]);
      chi[p] = (uint32_t)lower_bound_i64(sms, cb, ce, sme[p]);
    }
  }
  if (__ballot(ov) != 0 && (threadIdx.x & (kWave - 1)) == 0)
    atomicOr(status, (uint32_t)CHOPPER_ST_MARKER_OVERLAP);
}

__global__ __launch_bounds__(kBlock) void k_attribute_records(
    int64_t n, int G, int D, const uint8_t* gpu, const int64_t* start,
    const uint32_t* coff, const int64_t* sms, const int64_t* sme,
    const uint32_t* sid, const uint32_t* clo, const uint32_t* chi,
    uint32_t* idx) {
  const int64_t k = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (k >= n) return;
  const int g = gpu[k];
  if (g >= G) {
    for (int l = 0; l < D; ++l) idx[(int64_t)l * n + k] = kNone;
    return;
  }
  const int64_t s = start[k];
  int64_t parent = -1;
  for (int l = 0; l < D; ++l) {
    const uint32_t cls = (uint32_t)(g * D + l) * 2u;
    const int64_t sb = coff[cls], se = coff[cls + 1];
    int64_t lo = sb, hi = se;
    if (parent >= 0) {
      lo = clo[parent];
      hi = chi[parent];
    }
    int64_t j = upper_bound_i64(sms, lo, hi, s) - 1;
    if (j < lo) j = (lo > sb) ? lo - 1 : -1;
    uint32_t out = kNone;
    parent = -1;
    if (j >= 0 && s < sme[j]) {
      out = sid[j];
      parent = j;
    }
    idx[(int64_t)l * n + k] = out;
  }
}

struct AttrLayout {
  uint32_t* mord;
  uint32_t* coff;
  int64_t* sms;
  int64_t* sme;
  uint32_t* sid;
  uint32_t* clo;
  uint32_t* chi;
  ClassSortLayout sort;
};

static AttrLayout attr_layout(Scratch& sc, int64_t nm, int G, int D) {
  AttrLayout L;
  const int C = G * D * 2 + 1;
  L.mord = sc.take<uint32_t>(nm);
  L.coff = sc.take<uint32_t>(C + 1);
  L.sms = sc.take<int64_t>(nm);
  L.sme = sc.take<int64_t>(nm);
  L.sid = sc.take<uint32_t>(nm);
  L.clo = sc.take<uint32_t>(nm);
  L.chi = sc.take<uint32_t>(nm);
  L.sort = class_sort_layout(sc, nm, C);
  return L;
}

}  // namespace chopper

using namespace chopper;

extern "C" int chopper_attribute(const chopper_records* rec,
                                 const int64_t* start_al,
                                 const chopper_markers* mk,
                                 const int64_t* mstart_al,
                                 const int64_t* mend_al, uint32_t* idx_out,
                                 void* scratch, size_t* scratch_bytes,
                                 uint32_t* status, void* stream) {
  if (!validate_records(rec) || !mk || !validate_markers(mk) || !scratch_bytes)
    return CHOPPER_EINVAL;
  const int64_t n = rec->n, nm = mk->n;
  const int G = rec->n_gpus, D = mk->depth;
  if (n > 0 && (!start_al || !idx_out)) return CHOPPER_EINVAL;
  if (nm > 0 && (!mstart_al || !mend_al)) return CHOPPER_EINVAL;
  Scratch probe(nullptr);
  attr_layout(probe, nm, G, D);
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  AttrLayout L = attr_layout(sc, nm, G, D);
  KeyMarker km{mk->gpu, mk->level, mstart_al, mend_al, G, D};
  bool range_err = false;
  rc = class_sort(km, L.sort, L.mord, L.coff, &range_err, s, -1);
  if (rc != CHOPPER_OK) return rc;
  if (range_err)
    CHOPPER_HIP(launch("status_set", k_status_set, dim3(1), dim3(1), s,
                       (uint32_t)CHOPPER_ST_RANGE, status));
  if (nm > 0) {
    CHOPPER_HIP(launch("attr_marker_gather", k_marker_gather,
                       grid_for(nm, kBlock), dim3(kBlock), s, nm,
                       (const uint32_t*)L.mord, mstart_al, mend_al, L.sms,
                       L.sme, L.sid));
    const int64_t per_seg = ceil_div(nm, (int64_t)G * D);
    unsigned gx = (unsigned)ceil_div(per_seg, kBlock);
    if (gx < 1) gx = 1;
    if (gx > 1024) gx = 1024;
    CHOPPER_HIP(launch("attr_marker_links", k_marker_links,
                       dim3(gx, (unsigned)(G * D)), dim3(kBlock), s, G, D,
                       (const uint32_t*)L.coff, (const int64_t*)L.sms,
                       (const int64_t*)L.sme, L.clo, L.chi, status));
  }
  if (n == 0) return CHOPPER_OK;
  CHOPPER_HIP(launch("attr_records", k_attribute_records, grid_for(n, kBlock),
                     dim3(kBlock), s, n, G, D, rec->gpu, start_al,
                     (const uint32_t*)L.coff, (const int64_t*)L.sms,
                     (const int64_t*)L.sme, (const uint32_t*)L.sid,
                     (const uint32_t*)L.clo, (const uint32_t*)L.chi, idx_out));
  return CHOPPER_OK;
}
