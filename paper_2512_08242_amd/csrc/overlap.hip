// chopper_overlap: compute/communication overlap (paper Section V-C) and
// launch bubbles (Section V-D eqs. 1-3; caption of Fig. end_to_end).
//
// An instant is compute-active iff some compute kernel covers it (c(t) > 0 in
// the +-1 event count), so the sweep reduces to the union of each GPU's
// compute intervals and the union of its communication intervals.  Walking
// the records in (gpu, kind, start') order, an interval opens a new union
// run iff its start lies beyond the running maximum of all earlier ends of
// the same (gpu, kind) -- a segmented max-scan.  Prefix sums of run lengths
// then give F(t) = active time before t for either kind by one binary
// search, and the time where both are active is accumulated per
// communication run, so every window (kernel, marker, GPU) costs a few
// binary searches and no per-window sweep.
#include "sort.h"

namespace chopper {

bool validate_records(const chopper_records* r);
bool validate_markers(const chopper_markers* m);

constexpr int kOvIpt = 8;
constexpr int kOvTile = kBlock * kOvIpt;
constexpr int kSegs = 512;            // gpu * 2 + kind

struct Runs {
  const int64_t* rs;      // run start
  const int64_t* re;      // run end
  const int64_t* pl;      // exclusive prefix of run lengths
  const int64_t* pov;     // exclusive prefix of overlapped time (comm runs)
  const int64_t* fcrs;    // compute-active time before each comm run start
  const uint32_t* rbeg;   // [kSegs] first run of a segment
  const uint32_t* rend;   // [kSegs] one past its last run
};

// active time of segment seg strictly before t
__device__ inline int64_t F_active(const Runs& R, uint32_t seg, int64_t t) {
  int64_t b = R.rbeg[seg], e = R.rend[seg];
  int64_t lo = b, hi = e;
  while (lo < hi) {
    int64_t mid = lo + ((hi - lo) >> 1);
    if (R.rs[mid] <= t) lo = mid + 1;
    else hi = mid;
  }
  int64_t j = lo - 1;
  if (j < b) return 0;
  int64_t end = R.re[j] < t ? R.re[j] : t;
  return R.pl[j] - R.pl[b] + (end - R.rs[j]);
}

// time before t where both kinds are active on gpu g
__device__ inline int64_t F_both(const Runs& R, uint32_t g, int64_t t) {
  const uint32_t seg = g * 2u + 1u;
  int64_t b = R.rbeg[seg], e = R.rend[seg];
  int64_t lo = b, hi = e;
  while (lo < hi) {
    int64_t mid = lo + ((hi - lo) >> 1);
    if (R.rs[mid] <= t) lo = mid + 1;
    else hi = mid;
  }
  int64_t j = lo - 1;
  if (j < b) return 0;
  int64_t end = R.re[j] < t ? R.re[j] : t;
  return R.pov[j] - R.pov[b] + F_active(R, g * 2u, end) - R.fcrs[j];
}

struct KItem {
  uint32_t seg;
  int64_t s, e;
};

__device__ inline KItem korder_item(const uint32_t* korder, const uint8_t* gpu,
                                    const uint8_t* cls, const int64_t* start,
                                    const int64_t* end, int64_t p) {
  uint32_t r = korder[p];
  KItem it;
  it.seg = (uint32_t)gpu[r] * 2u + (uint32_t)kind_of(cls[r]);
  it.s = start[r];
  int64_t e = end[r];
  it.e = e > it.s ? e : it.s;
  return it;
}

// ---------------- union runs -----------------------------------------------
__global__ __launch_bounds__(kBlock) void k_runs_tile_max(
    int64_t n, const uint32_t* korder, const uint8_t* gpu, const uint8_t* cls,
    const int64_t* start, const int64_t* end, SegMax* tile_agg) {
  const int64_t base = (int64_t)blockIdx.x * kOvTile;
  SegMax acc{0u, kI64Min};
  OpSegMax op;
  for (int j = 0; j < kOvIpt; ++j) {
    int64_t p = base + (int64_t)threadIdx.x * kOvIpt + j;
    if (p < n) {
      KItem it = korder_item(korder, gpu, cls, start, end, p);
      acc = op(acc, SegMax{it.seg, it.e});
    }
  }
  SegMax tot;
  block_exclusive(acc, op, SegMax{0u, kI64Min}, &tot);
  if (threadIdx.x == 0) tile_agg[blockIdx.x] = tot;
}

// exclusive scan of the tile maxima in one block; also the grand total
__global__ __launch_bounds__(kBlock) void k_runs_spine(SegMax* tile_agg,
                                                       int64_t ntiles,
                                                       SegMax* grand) {
  OpSegMax op;
  SegMax carry{0u, kI64Min};
  for (int64_t base = 0; base < ntiles; base += kBlock) {
    int64_t i = base + threadIdx.x;
    SegMax v = i < ntiles ? tile_agg[i] : SegMax{0u, kI64Min};
    SegMax tot;
    SegMax ex = block_exclusive(v, op, SegMax{0u, kI64Min}, &tot);
    if (i < ntiles) tile_agg[i] = op(carry, ex);
    carry = op(carry, tot);
  }
  if (threadIdx.x == 0) *grand = carry;
}

// Per-item exclusive running maximum; returns head flags for the tile's items.
__device__ inline void runs_tile_scan(int64_t n, const uint32_t* korder,
                                      const uint8_t* gpu, const uint8_t* cls,
                                      const int64_t* start, const int64_t* end,
                                      const SegMax* tile_pre, KItem (&it)[kOvIpt],
                                      SegMax (&ex)[kOvIpt],
                                      bool (&head)[kOvIpt], bool (&valid)[kOvIpt]) {
  const int64_t base = (int64_t)blockIdx.x * kOvTile;
  OpSegMax op;
  SegMax acc{0u, kI64Min};
  SegMax loc[kOvIpt];
  for (int j = 0; j < kOvIpt; ++j) {
    int64_t p = base + (int64_t)threadIdx.x * kOvIpt + j;
    valid[j] = p < n;
    if (valid[j]) it[j] = korder_item(korder, gpu, cls, start, end, p);
    else it[j] = KItem{0u, 0, 0};
    loc[j] = acc;
    if (valid[j]) acc = op(acc, SegMax{it[j].seg, it[j].e});
  }
  SegMax tot;
  SegMax pre = block_exclusive(acc, op, SegMax{0u, kI64Min}, &tot);
  pre = op(tile_pre[blockIdx.x], pre);
  for (int j = 0; j < kOvIpt; ++j) {
    ex[j] = op(pre, loc[j]);
    const int64_t p = base + (int64_t)threadIdx.x * kOvIpt + j;
    head[j] = valid[j] &&
              (p == 0 || ex[j].seg != it[j].seg || it[j].s > ex[j].val);
  }
}

__global__ __launch_bounds__(kBlock) void k_runs_count(
    int64_t n, const uint32_t* korder, const uint8_t* gpu, const uint8_t* cls,
    const int64_t* start, const int64_t* end, const SegMax* tile_pre,
    uint32_t* tile_heads) {
  KItem it[kOvIpt];
  SegMax ex[kOvIpt];
  bool head[kOvIpt], valid[kOvIpt];
  runs_tile_scan(n, korder, gpu, cls, start, end, tile_pre, it, ex, head,
                 valid);
  uint32_t c = 0;
  for (int j = 0; j < kOvIpt; ++j) c += head[j] ? 1u : 0u;
  uint32_t tot;
  block_exclusive(c, OpAdd(), 0u, &tot);
  if (threadIdx.x == 0) tile_heads[blockIdx.x] = tot;
}

__global__ __launch_bounds__(kBlock) void k_runs_write(
    int64_t n, const uint32_t* korder, const uint8_t* gpu, const uint8_t* cls,
    const int64_t* start, const int64_t* end, const SegMax* tile_pre,
    const uint32_t* tile_run0, const uint32_t* nruns, const SegMax* grand,
    int64_t* rs, int64_t* re, uint32_t* rseg, uint32_t* rbeg, uint32_t* rend) {
  KItem it[kOvIpt];
  SegMax ex[kOvIpt];
  bool head[kOvIpt], valid[kOvIpt];
  runs_tile_scan(n, korder, gpu, cls, start, end, tile_pre, it, ex, head,
                 valid);
  uint32_t c = 0;
  for (int j = 0; j < kOvIpt; ++j) c += head[j] ? 1u : 0u;
  uint32_t tot;
  uint32_t r = block_exclusive(c, OpAdd(), 0u, &tot) + tile_run0[blockIdx.x];
  const int64_t base = (int64_t)blockIdx.x * kOvTile;
  for (int j = 0; j < kOvIpt; ++j) {
    const int64_t p = base + (int64_t)threadIdx.x * kOvIpt + j;
    if (head[j]) {
      rs[r] = it[j].s;
      rseg[r] = it[j].seg;
      const bool new_seg = (p == 0) || ex[j].seg != it[j].seg;
      if (p > 0) re[r - 1] = ex[j].val;   // the previous run ends here
      if (new_seg) {
        rbeg[it[j].seg] = r;
        if (p > 0) rend[ex[j].seg] = r;
      }
      ++r;
    }
    if (valid[j] && p == n - 1) {
      const uint32_t R = *nruns;
      re[R - 1] = grand->val;
      rend[it[j].seg] = R;
    }
  }
}

__global__ __launch_bounds__(kBlock) void k_runs_len(const uint32_t* nruns,
                                                     const int64_t* rs,
                                                     const int64_t* re,
                                                     int64_t* len, int64_t cap) {
  int64_t r = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (r >= cap) return;
  len[r] = r < (int64_t)*nruns ? re[r] - rs[r] : 0;
}

// overlapped time inside each comm run: compute-active time within it
__global__ __launch_bounds__(kBlock) void k_runs_comm_overlap(
    const uint32_t* nruns, Runs R, const uint32_t* rseg, int64_t* ovc,
    int64_t* fcrs, int64_t cap) {
  int64_t r = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (r >= cap) return;
  int64_t v = 0, f = 0;
  if (r < (int64_t)*nruns) {
    uint32_t seg = rseg[r];
    if (seg & 1u) {
      uint32_t cseg = seg - 1u;
      f = F_active(R, cseg, R.rs[r]);
      v = F_active(R, cseg, R.re[r]) - f;
    }
  }
  ovc[r] = v;
  fcrs[r] = f;
}

// ---------------- queries ----------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_overlap_records(
    int64_t n, int G, const uint8_t* gpu, const uint8_t* cls,
    const int64_t* start, const int64_t* end, Runs R, int64_t* ovl) {
  const int64_t k = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (k >= n) return;
  const uint32_t g = gpu[k];
  const int64_t s = start[k], e = end[k];
  int64_t o = 0;
  if (e > s && (int)g < G) {
    // a compute kernel's overlapped time is the comm-active time inside it
    // and vice versa
    const uint32_t other = g * 2u + (kind_of(cls[k]) ? 0u : 1u);
    o = F_active(R, other, e) - F_active(R, other, s);
  }
  ovl[k] = o;
}

__device__ inline void window(const Runs& R, uint32_t g, int64_t a, int64_t b,
                              int64_t* out) {
  if (b <= a) {
    out[0] = out[1] = out[2] = out[3] = 0;
    return;
  }
  const int64_t c = F_active(R, g * 2u, b) - F_active(R, g * 2u, a);
  const int64_t m = F_active(R, g * 2u + 1u, b) - F_active(R, g * 2u + 1u, a);
  const int64_t o = F_both(R, g, b) - F_both(R, g, a);
  out[0] = c - o;
  out[1] = m - o;
  out[2] = o;
  out[3] = (b - a) - c - m + o;
}

__global__ __launch_bounds__(kBlock) void k_overlap_markers(
    int64_t nm, int G, const uint8_t* mgpu, const int64_t* ms,
    const int64_t* me, Runs R, int64_t* mwin) {
  const int64_t j = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (j >= nm) return;
  int64_t w[4] = {0, 0, 0, 0};
  const uint32_t g = mgpu[j];
  if ((int)g < G) window(R, g, ms[j], me[j], w);
  for (int z = 0; z < 4; ++z) mwin[4 * j + z] = w[z];
}

// GPU window: the first run of a (gpu, kind) segment starts at its smallest
// start', the last run ends at its largest end'
__global__ void k_overlap_gpus(int G, Runs R, int64_t* gwin) {
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= G) return;
  int64_t a = kI64Max, b = kI64Min;
  for (uint32_t seg = g * 2u; seg < g * 2u + 2u; ++seg) {
    const uint32_t rb = R.rbeg[seg], re = R.rend[seg];
    if (re > rb) {
      a = R.rs[rb] < a ? R.rs[rb] : a;
      b = R.re[re - 1] > b ? R.re[re - 1] : b;
    }
  }
  if (a == kI64Max) a = b = 0;
  int64_t w[4];
  window(R, (uint32_t)g, a, b, w);
  gwin[6 * g + 0] = a;
  gwin[6 * g + 1] = b;
  for (int z = 0; z < 4; ++z) gwin[6 * g + 2 + z] = w[z];
}

// ---------------- bubbles ----------------------------------------------------
// In (gpu, stream, start') order the previous compute record of a compute
// record is found by walking back over communication records of the same
// (gpu, stream).  Each communication record is walked over by at most one
// compute record (the next one), so the total work is linear.
__global__ __launch_bounds__(kBlock) void k_gap(
    int64_t n, const uint32_t* order, const uint8_t* gpu, const uint8_t* stream,
    const uint8_t* cls, const int64_t* start, const int64_t* end,
    int64_t* gap) {
  const int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (p >= n) return;
  const uint32_t r = order[p];
  int64_t gv = 0;
  if (!kind_of(cls[r])) {
    const uint8_t g = gpu[r], st = stream[r];
    for (int64_t q = p - 1; q >= 0; --q) {
      const uint32_t rq = order[q];
      if (gpu[rq] != g || stream[rq] != st) break;
      if (!kind_of(cls[rq])) {
        const int64_t b = start[r] - end[rq];
        gv = b > 0 ? b : 0;
        break;
      }
    }
  }
  gap[r] = gv;
}

// ---------------------------------------------------------------------------
struct OverlapLayout {
  int64_t ntiles;
  SegMax* tile_agg;
  SegMax* grand;
  uint32_t* tile_heads;
  uint32_t* tile_run0;
  uint32_t* nruns;
  uint32_t* scan_u32;
  int64_t* rs;
  int64_t* re;
  uint32_t* rseg;
  uint32_t* rbeg;     // kSegs, then rend kSegs
  uint32_t* rend;
  int64_t* len;
  int64_t* pl;
  int64_t* ovc;
  int64_t* pov;
  int64_t* fcrs;
  int64_t* scan_i64;
  int64_t* tot_i64;
};

static OverlapLayout overlap_layout(Scratch& sc, int64_t n, int G) {
  OverlapLayout L;
  L.ntiles = ceil_div(n, kOvTile);
  L.tile_agg = sc.take<SegMax>(L.ntiles);
  L.grand = sc.take<SegMax>(1);
  L.tile_heads = sc.take<uint32_t>(L.ntiles);
  L.tile_run0 = sc.take<uint32_t>(L.ntiles);
  L.nruns = sc.take<uint32_t>(1);
  L.scan_u32 = sc.take<uint32_t>(scan_scratch_elems(L.ntiles));
  L.rs = sc.take<int64_t>(n);
  L.re = sc.take<int64_t>(n);
  L.rseg = sc.take<uint32_t>(n);
  L.rbeg = sc.take<uint32_t>(2 * kSegs);
  L.rend = L.rbeg ? L.rbeg + kSegs : nullptr;
  L.len = sc.take<int64_t>(n);
  L.pl = sc.take<int64_t>(n);
  L.ovc = sc.take<int64_t>(n);
  L.pov = sc.take<int64_t>(n);
  L.fcrs = sc.take<int64_t>(n);
  L.scan_i64 = sc.take<int64_t>(scan_scratch_elems(n));
  L.tot_i64 = sc.take<int64_t>(2);
  return L;
}

}  // namespace chopper

using namespace chopper;

extern "C" int chopper_overlap(const chopper_records* rec,
                               const int64_t* start_al, const int64_t* end_al,
                               const uint32_t* order, const uint32_t* korder,
                               const chopper_markers* mk,
                               const int64_t* mstart_al, const int64_t* mend_al,
                               int64_t* ovl_out, int64_t* gap_out,
                               int64_t* mwin_out, int64_t* gwin_out,
                               void* scratch, size_t* scratch_bytes,
                               uint32_t* status, void* stream) {
  if (!validate_records(rec) || !validate_markers(mk) || !scratch_bytes)
    return CHOPPER_EINVAL;
  const int64_t n = rec->n;
  const int64_t nm = mk ? mk->n : 0;
  const int G = rec->n_gpus;
  if (n > 0 && (!start_al || !end_al || !order || !korder || !ovl_out ||
                !gap_out))
    return CHOPPER_EINVAL;
  if (nm > 0 && (!mstart_al || !mend_al || !mwin_out)) return CHOPPER_EINVAL;
  if (!gwin_out) return CHOPPER_EINVAL;
  Scratch probe(nullptr);
  overlap_layout(probe, n, G);
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  OverlapLayout L = overlap_layout(sc, n, G);
  const unsigned T = (unsigned)L.ntiles;

  CHOPPER_HIP(launch("ov_fill", k_fill_u32, grid_for(2 * kSegs, kBlock),
                     dim3(kBlock), s, L.rbeg, (int64_t)(2 * kSegs), 0u));
  if (n > 0) {
    // union runs of every (gpu, kind)
    CHOPPER_HIP(launch("ov_runs_tile_max", k_runs_tile_max, dim3(T),
                       dim3(kBlock), s, n, korder, rec->gpu, rec->cls,
                       start_al, end_al, L.tile_agg));
    CHOPPER_HIP(launch("ov_runs_spine", k_runs_spine, dim3(1), dim3(kBlock), s,
                       L.tile_agg, L.ntiles, L.grand));
    CHOPPER_HIP(launch("ov_runs_count", k_runs_count, dim3(T), dim3(kBlock), s,
                       n, korder, rec->gpu, rec->cls, start_al, end_al,
                       (const SegMax*)L.tile_agg, L.tile_heads));
    CHOPPER_HIP(exclusive_scan<uint32_t>(L.tile_heads, L.tile_run0, L.ntiles,
                                         L.scan_u32, L.nruns, s));
    CHOPPER_HIP(launch("ov_runs_write", k_runs_write, dim3(T), dim3(kBlock), s,
                       n, korder, rec->gpu, rec->cls, start_al, end_al,
                       (const SegMax*)L.tile_agg, (const uint32_t*)L.tile_run0,
                       (const uint32_t*)L.nruns, (const SegMax*)L.grand, L.rs,
                       L.re, L.rseg, L.rbeg, L.rend));
    CHOPPER_HIP(launch("ov_runs_len", k_runs_len, grid_for(n, kBlock),
                       dim3(kBlock), s, (const uint32_t*)L.nruns,
                       (const int64_t*)L.rs, (const int64_t*)L.re, L.len, n));
    CHOPPER_HIP(exclusive_scan<int64_t>(L.len, L.pl, n, L.scan_i64, L.tot_i64,
                                        s));
  }
  Runs R{L.rs, L.re, L.pl, L.pov, L.fcrs, L.rbeg, L.rend};
  if (n > 0) {
    CHOPPER_HIP(launch("ov_runs_comm_overlap", k_runs_comm_overlap,
                       grid_for(n, kBlock), dim3(kBlock), s,
                       (const uint32_t*)L.nruns, R, (const uint32_t*)L.rseg,
                       L.ovc, L.fcrs, n));
    CHOPPER_HIP(exclusive_scan<int64_t>(L.ovc, L.pov, n, L.scan_i64,
                                        L.tot_i64 + 1, s));
    CHOPPER_HIP(launch("ov_records", k_overlap_records, grid_for(n, kBlock),
                       dim3(kBlock), s, n, G, rec->gpu, rec->cls, start_al,
                       end_al, R, ovl_out));
  }
  if (nm > 0)
    CHOPPER_HIP(launch("ov_markers", k_overlap_markers, grid_for(nm, kBlock),
                       dim3(kBlock), s, nm, G, mk->gpu, mstart_al, mend_al, R,
                       mwin_out));
  CHOPPER_HIP(launch("ov_gpus", k_overlap_gpus, grid_for(G, kBlock),
                     dim3(kBlock), s, G, R, gwin_out));
  if (n > 0) {
    CHOPPER_HIP(launch("ov_gap", k_gap, grid_for(n, kBlock), dim3(kBlock), s,
                       n, order, rec->gpu, rec->stream, rec->cls, start_al,
                       end_al, gap_out));
  }
  return CHOPPER_OK;
}
