// chopper_attribute: every kernel record is assigned, level by level, to the
// annotation marker containing its aligned start (paper Section I
// granularities; III-A annotations for kernels, operations, layers and
// iterations).
//
// Markers are sorted by (gpu, level, empty, start') into contiguous
// per-(gpu, level) segments of non-empty markers, and a bucket index over
// each segment's starts narrows every search to a few markers.  The answer
// at a level is the last marker of the record's (gpu, level) segment whose
// start is <= the record's start, if the record starts before its end; the
// levels are independent, so a record searches all of them in lockstep.
#include "sort.h"
#include "bindex.h"

namespace chopper {

bool validate_records(const chopper_records* r);
bool validate_markers(const chopper_markers* m);

// sorted marker columns and the (gpu, level) segment of every non-empty
// marker (kNone for empty or invalid ones)
__global__ __launch_bounds__(kBlock) void k_marker_gather(
    int64_t nm, KeyMarker km, const uint32_t* mord, const int64_t* ms,
    const int64_t* me, int64_t* sms, int64_t* sme, uint32_t* sid,
    uint32_t* sseg) {
  int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (p >= nm) return;
  uint32_t j = mord[p];
  sms[p] = ms[j];
  sme[p] = me[j];
  sid[p] = j;
  const uint32_t c = km.cls(j);
  sseg[p] = ((c & 1u) || c >= (uint32_t)(km.G * km.D * 2)) ? kNone : c >> 1;
}

// overlap check between neighbours of a (gpu, level) segment
__global__ __launch_bounds__(kBlock) void k_marker_links(
    int G, int D, const uint32_t* coff, const int64_t* sms, const int64_t* sme,
    uint32_t* status) {
  // one block column per (gpu, level) segment
  const int seg = blockIdx.y;          // g * D + l
  const uint32_t cls = (uint32_t)seg * 2u;
  const int64_t b = coff[cls], e = coff[cls + 1];
  (void)G;
  (void)D;
  bool ov = false;
  for (int64_t p = b + (int64_t)blockIdx.x * kBlock + threadIdx.x; p < e;
       p += (int64_t)gridDim.x * kBlock) {
    if (p + 1 < e && sme[p] > sms[p + 1]) ov = true;
  }
  if (__ballot(ov) != 0 && (threadIdx.x & (kWave - 1)) == 0)
    atomicOr(status, (uint32_t)CHOPPER_ST_MARKER_OVERLAP);
}

// segment parameters held in LDS when there are at most this many
constexpr int kLdsSegs = 512;

template <int MaxD, bool kLds>
__global__ __launch_bounds__(kBlock) void k_attribute_records(
    int64_t n, int G, int D, const uint8_t* gpu, const int64_t* start,
    BIndex X, const int64_t* sme, const uint32_t* sid, uint32_t* idx) {
  __shared__ BSeg s_seg[kLds ? kLdsSegs : 1];
  if (kLds) {
    for (int i = threadIdx.x; i < G * D; i += kBlock) s_seg[i] = X.seg[i];
    __syncthreads();
  }
  const int64_t k = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (k >= n) return;
  const int g = gpu[k];
  if (g >= G) {
    for (int l = 0; l < D; ++l) idx[(int64_t)l * n + k] = kNone;
    return;
  }
  const int64_t s = start[k];
  BSeg P[MaxD];
  int64_t lo[MaxD], hi[MaxD], t[MaxD];
#pragma unroll
  for (int l = 0; l < MaxD; ++l) {
    t[l] = s;
    lo[l] = hi[l] = 0;
    if (l < D) {
      P[l] = kLds ? s_seg[g * D + l] : X.seg[g * D + l];
      bi_range(X, P[l], s, &lo[l], &hi[l]);
    }
  }
  bsearch_k<MaxD>(X.key, lo, hi, t);
#pragma unroll
  for (int l = 0; l < MaxD; ++l) {
    if (l >= D) break;
    const int64_t j = lo[l] - 1;
    uint32_t out = kNone;
    if (j >= (int64_t)P[l].sb && s < sme[j]) out = sid[j];
    idx[(int64_t)l * n + k] = out;
  }
}

struct AttrLayout {
  uint32_t* mord;
  uint32_t* coff;
  int64_t* sms;
  int64_t* sme;
  uint32_t* sid;
  uint32_t* sseg;
  BSeg* bsegs;
  uint32_t* btable;
  int64_t btable_cap;
  uint32_t* btmp;
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
  L.sseg = sc.take<uint32_t>(nm);
  L.bsegs = sc.take<BSeg>((int64_t)G * D);
  L.btable_cap = bindex_table_cap(nm, (int64_t)G * D);
  L.btable = sc.take<uint32_t>(L.btable_cap);
  L.btmp = sc.take<uint32_t>((int64_t)G * D + 1);
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
                       grid_for(nm, kBlock), dim3(kBlock), s, nm, km,
                       (const uint32_t*)L.mord, mstart_al, mend_al, L.sms,
                       L.sme, L.sid, L.sseg));
    const int64_t per_seg = ceil_div(nm, (int64_t)G * D);
    unsigned gx = (unsigned)ceil_div(per_seg, kBlock);
    if (gx < 1) gx = 1;
    if (gx > 1024) gx = 1024;
    CHOPPER_HIP(launch("attr_marker_links", k_marker_links,
                       dim3(gx, (unsigned)(G * D)), dim3(kBlock), s, G, D,
                       (const uint32_t*)L.coff, (const int64_t*)L.sms,
                       (const int64_t*)L.sme, status));
  }
  if (n == 0 || D == 0) return CHOPPER_OK;
  // bucket index of the non-empty marker starts of every (gpu, level)
  CHOPPER_HIP(bindex_build(L.sms, L.sseg, nm, nullptr, L.coff, L.coff + 1, 2,
                           G * D, L.bsegs, L.btable, L.btable_cap, L.btmp, s));
  const BIndex X{L.sms, L.bsegs, L.btable};
  auto run = [&](auto kern) -> int {
    CHOPPER_HIP(launch("attr_records", kern, grid_for(n, kBlock),
                       dim3(kBlock), s, n, G, D, rec->gpu, start_al, X,
                       (const int64_t*)L.sme, (const uint32_t*)L.sid,
                       idx_out));
    return CHOPPER_OK;
  };
  const bool lds = G * D <= kLdsSegs;
  if (D <= 4)
    return lds ? run(k_attribute_records<4, true>)
               : run(k_attribute_records<4, false>);
  return lds ? run(k_attribute_records<8, true>)
             : run(k_attribute_records<8, false>);
  return CHOPPER_OK;
}
