// chopper_join_counters: counters of serialized hardware-profiling passes
// attached to the runtime trace's kernels (Section III-A: only two or three
// counters per pass, kernels serialized, no valid timestamps; Section III-B:
// alignment attaches the counters to operations, layers and iterations).
//
// A record and a pass entry match on (gpu, stream, iteration label,
// ordinal) and class.  Both sides are brought into (gpu, stream) order --
// the records by `order`, a pass by a stable class partition of its own
// order -- and cut into runs of equal (gpu, stream, label): with every
// label's records consecutive along its (gpu, stream) and labels increasing
// (checked, JOIN_ORDER otherwise), a label is one run and the ordinal is the
// position inside it.  Record runs find their pass run by a binary search
// over the pass's run table; each record then reads entry run start +
// ordinal.
#include <algorithm>
#include <vector>

#include "sort.h"
#include "wave.h"

namespace chopper {

bool validate_records(const chopper_records* r);
bool validate_markers(const chopper_markers* m);
hipError_t read_back(const void* dev, void* host, size_t bytes, hipStream_t s);

namespace {

constexpr int kMaxPasses = 8;
constexpr int kDenseT = 1024;

__global__ void k_join_fill_u64(uint64_t* p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

__global__ void k_join_zero(uint32_t* p) { *p = 0; }

__global__ void k_join_fill_u8(uint8_t* p, int64_t n, uint32_t* pres) {
  const int64_t i0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int64_t i = i0; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = 0;
  if (pres)
    for (int64_t i = i0; i < 65536 / 4; i += (int64_t)gridDim.x * blockDim.x)
      pres[i] = 0;
}

// iteration label of every record (NONE: no iteration marker)
__global__ void k_join_rec_labels(int64_t n, const uint32_t* idx_iter,
                                  int64_t nm, const uint32_t* m_label,
                                  uint32_t* lab) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const uint32_t m = idx_iter[i];
  lab[i] = (int64_t)m < nm ? m_label[m] : kNone;
}

// the (gpu, stream) pairs of the records
__global__ void k_join_presence(int64_t n, const uint8_t* gpu,
                                const uint8_t* stream, uint8_t* pres) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) pres[(uint32_t)gpu[i] * 256u + stream[i]] = 1;
}

// Dense class ids of the records' (gpu, stream) pairs in (gpu, stream)
// order; every other pair gets the id after the last (pass entries of such
// pairs can match nothing); count[0] = number of records' pairs.
__global__ __launch_bounds__(kDenseT) void k_join_dense(const uint8_t* pres,
                                                        uint16_t* cmap,
                                                        uint32_t* count) {
  __shared__ uint32_t s_w[kDenseT / kWave + 1];
  const int t = threadIdx.x, lane = lane_id(), w = t / kWave;
  uint4 f[4];
  const uint4* src = reinterpret_cast<const uint4*>(pres) + t * 4;
#pragma unroll
  for (int q = 0; q < 4; ++q) f[q] = src[q];
  const uint8_t* fb = reinterpret_cast<const uint8_t*>(f);
  uint32_t c = 0;
#pragma unroll
  for (int b = 0; b < 64; ++b) c += fb[b] ? 1u : 0u;
  const uint32_t incl = wave_incl(c, OpAdd(), 0u);
  if (lane == kWave - 1) s_w[w] = incl;
  __syncthreads();
  uint32_t id = incl - c, tot = 0;
  for (int q = 0; q < kDenseT / kWave; ++q) {
    if (q < w) id += s_w[q];
    tot += s_w[q];
  }
  uint16_t ids[64];
#pragma unroll
  for (int b = 0; b < 64; ++b) {
    ids[b] = (uint16_t)(fb[b] ? id : tot);
    id += fb[b] ? 1u : 0u;
  }
  uint4* dst = reinterpret_cast<uint4*>(cmap) + t * 8;
  const uint4* iv = reinterpret_cast<const uint4*>(ids);
#pragma unroll
  for (int q = 0; q < 8; ++q) dst[q] = iv[q];
  if (t == 0) *count = tot;
}

// Items of a (gpu, stream)-ordered sequence: key = (gpu, stream, label).
struct Seq {
  const uint32_t* idx;     // sequence position -> item
  const uint8_t* gpu;
  const uint8_t* stream;
  const uint32_t* lab;
  const uint16_t* cmap;    // (gpu, stream) -> dense class
  int64_t n;
  __device__ uint32_t cls(uint32_t i) const {
    return cmap[(uint32_t)gpu[i] * 256u + stream[i]];
  }
};

// key of a sequence item: label | class << 32 | pass class << 48
__device__ inline uint64_t item_key(const Seq& S, const uint8_t* pcls,
                                    uint32_t i) {
  return (uint64_t)S.lab[i] | (uint64_t)S.cls(i) << 32 |
         (pcls ? (uint64_t)pcls[i] << 48 : 0ull);
}

// run heads: an item with an iteration whose predecessor differs in
// (gpu, stream, label) -- items without an iteration belong to no run, and
// one of them between two items of a label starts a second run of it.  The
// key of every position is kept for the later passes, which then read it
// in sequence order.
// The heads of a block of kBlock positions are also counted (tcnt), so that
// the run numbers come from a scan of the block counts.
__global__ __launch_bounds__(kBlock) void k_join_heads(Seq S,
                                                       const uint8_t* pcls,
                                                       uint32_t* head,
                                                       uint64_t* key,
                                                       uint32_t* tcnt) {
  __shared__ uint32_t s_c[kWavesPerBlock];
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool ok = p < S.n;
  const uint64_t kb = ok ? item_key(S, pcls, S.idx[p]) : 0ull;
  // the predecessor's key from the lane below; lane 0 loads it
  uint64_t ka = wave_shr1_any((uint64_t)0, kb);
  if (lane_id() == 0 && ok && p > 0) ka = item_key(S, pcls, S.idx[p - 1]);
  const uint64_t kMask = 0x0000FFFFFFFFFFFFull;    // class and label
  uint32_t h = 0;
  if (ok && (uint32_t)kb != kNone) h = (p == 0 || ((ka ^ kb) & kMask) != 0);
  if (ok) {
    head[p] = h;
    key[p] = kb;
  }
  const uint32_t c = (uint32_t)__popcll(__ballot(h != 0));
  if (lane_id() == 0) s_c[threadIdx.x / kWave] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t sum = 0;
    for (int w = 0; w < kWavesPerBlock; ++w) sum += s_c[w];
    tcnt[blockIdx.x] = sum;
  }
}

// run table: start position, (gpu, stream) and label of every run, the run
// number of a head being the heads before it (block prefix tpre + the
// heads below it in its block); excl (optional) gets that count at every
// position
__global__ __launch_bounds__(kBlock) void k_join_runs(
    int64_t n, const uint32_t* head, const uint32_t* tpre,
    const uint64_t* key, uint32_t* rstart, uint32_t* rcls, uint32_t* rlab,
    uint32_t* excl) {
  __shared__ uint32_t s_c[kWavesPerBlock];
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const uint32_t h = p < n ? head[p] : 0u;
  const uint64_t m = __ballot(h != 0);
  const int w = threadIdx.x / kWave;
  if (lane_id() == 0) s_c[w] = (uint32_t)__popcll(m);
  __syncthreads();
  uint32_t r = tpre[blockIdx.x] + lanes_below(m);
  for (int q = 0; q < w; ++q) r += s_c[q];
  if (p >= n) return;
  if (excl) excl[p] = r;
  if (!h) return;
  const uint64_t k = key[p];
  rstart[r] = (uint32_t)p;
  rcls[r] = (uint32_t)(k >> 32) & 0xFFFFu;
  rlab[r] = (uint32_t)k;
}

// run and ordinal of every record, stored at the record (NONE: no
// iteration)
__global__ void k_join_rec_pos(int64_t n, const uint32_t* order,
                               const uint32_t* head, const uint32_t* excl,
                               const uint64_t* key, const uint32_t* rstart,
                               uint32_t* rrun, uint32_t* rord) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= n) return;
  const uint32_t r = order[p];
  if ((uint32_t)key[p] == kNone) {
    rrun[r] = kNone;
    rord[r] = 0;
    return;
  }
  const uint32_t run = excl[p] + head[p] - 1;
  rrun[r] = run;
  rord[r] = (uint32_t)p - rstart[run];
}

// JOIN_ORDER: a run whose label is not above that of the previous run of
// its (gpu, stream); otherwise the run table is sorted by (gpu, stream,
// label) and every label has one run
__global__ void k_join_order(const uint32_t* nruns, const uint32_t* rcls,
                             const uint32_t* rlab, uint32_t* status) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r == 0 || r >= (int64_t)*nruns) return;
  if (rcls[r - 1] == rcls[r] && rlab[r - 1] >= rlab[r])
    atomicOr(status, CHOPPER_ST_JOIN_ORDER);
}

// pass run of every record run: binary search by (gpu, stream, label)
__global__ void k_join_match(const uint32_t* nr, const uint32_t* rcls,
                             const uint32_t* rlab, const uint32_t* nq,
                             const uint32_t* qcls, const uint32_t* qlab,
                             uint32_t* match) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= (int64_t)*nr) return;
  const uint64_t key = (uint64_t)rcls[r] << 32 | rlab[r];
  int64_t lo = 0, hi = (int64_t)*nq;     // first run with key >= ours
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    const uint64_t k = (uint64_t)qcls[mid] << 32 | qlab[mid];
    if (k < key) lo = mid + 1;
    else hi = mid;
  }
  const bool hit = lo < (int64_t)*nq &&
                   ((uint64_t)qcls[lo] << 32 | qlab[lo]) == key;
  match[r] = hit ? (uint32_t)lo : kNone;
}

struct PassCols {
  int32_t n_cols;
  int32_t bit;
  int32_t dst[16];
};

// every record, in input order: its entry in the pass (run start +
// ordinal), the key and class check, and the pass's columns (0 where
// nothing matches)
__global__ __launch_bounds__(kBlock) void k_join_gather(
    int64_t n, const uint32_t* rrun, const uint32_t* rord, const uint8_t* cls,
    const uint32_t* rcls, const uint32_t* rlab, const uint32_t* match,
    const uint32_t* qstart, const uint32_t* nq, int64_t m,
    const uint32_t* qorder, const uint64_t* qkey, const uint64_t* values,
    PassCols C, uint64_t* counters, uint8_t* matched, uint32_t* status) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool miss = false;
  if (r < n) {
    const uint32_t run = rrun[r];
    int64_t q = -1;
    if (run != kNone) {
      const uint32_t qr = match[run];
      if (qr != kNone) {
        const int64_t pos = (int64_t)qstart[qr] + rord[r];
        const int64_t q1 =
            (int64_t)qr + 1 < (int64_t)*nq ? (int64_t)qstart[qr + 1] : m;
        // the entry at the ordinal is the record's only if it still has the
        // run's key (entries without an iteration may follow the run)
        if (pos < q1) {
          const uint64_t k = qkey[pos];
          if ((uint32_t)k == rlab[run] &&
              ((uint32_t)(k >> 32) & 0xFFFFu) == rcls[run] &&
              (uint32_t)(k >> 48) == cls[r])
            q = qorder[pos];
        }
      }
      miss = q < 0;
    }
    for (int c = 0; c < C.n_cols; ++c)
      counters[(int64_t)C.dst[c] * n + r] =
          q >= 0 ? values[(int64_t)c * m + q] : 0ull;
    if (q >= 0) matched[r] |= (uint8_t)(1u << C.bit);
  }
  if (__ballot(miss) != 0 && lane_id() == 0)
    atomicOr(status, CHOPPER_ST_JOIN_MISS);
}

}  // namespace

extern "C" int chopper_join_counters(
    const chopper_records* rec, const int64_t* start_al, const uint32_t* order,
    const uint32_t* idx, int32_t depth, int32_t iter_level,
    const chopper_markers* mk, const chopper_counter_pass* passes,
    int32_t n_passes, uint64_t* counters_out, uint8_t* matched_out,
    void* scratch, size_t* scratch_bytes, uint32_t* status, void* stream) {
  if (!validate_records(rec) || !validate_markers(mk) || !mk ||
      !scratch_bytes || n_passes < 0 || n_passes > kMaxPasses ||
      (n_passes > 0 && !passes) || depth < 1 || iter_level < 0 ||
      iter_level >= depth || depth > mk->depth)
    return CHOPPER_EINVAL;
  const int64_t n = rec->n, nm = mk->n;
  if (n > 0 && (!start_al || !order || !idx || !counters_out || !matched_out))
    return CHOPPER_EINVAL;
  if (nm > 0 && !mk->label) return CHOPPER_EINVAL;
  int64_t mmax = 0;
  uint32_t used = 0;
  for (int p = 0; p < n_passes; ++p) {
    const chopper_counter_pass& P = passes[p];
    if (P.n < 0 || P.n >= (int64_t)0xFFFFFFFF || P.n_cols < 1 ||
        P.n_cols > 16)
      return CHOPPER_EINVAL;
    if (P.n > 0 && (!P.gpu || !P.stream || !P.cls || !P.label || !P.values))
      return CHOPPER_EINVAL;
    for (int c = 0; c < P.n_cols; ++c) {
      if (P.dst[c] < 0 || P.dst[c] >= 16 || ((used >> P.dst[c]) & 1u))
        return CHOPPER_EINVAL;
      used |= 1u << P.dst[c];
    }
    mmax = P.n > mmax ? P.n : mmax;
  }
  // scratch: record labels and runs; per pass (reused): times, class map,
  // class sort, order, heads and runs
  auto layout = [&](Scratch& sc, std::vector<void*>& v) {
    v.clear();
    v.push_back(sc.take<uint32_t>(n));             // 0 rec labels
    v.push_back(sc.take<uint32_t>(n));             // 1 heads
    v.push_back(sc.take<uint32_t>(n));             // 2 excl
    v.push_back(sc.take<uint32_t>(n + 1));         // 3 rstart
    v.push_back(sc.take<uint32_t>(n + 1));         // 4 rcls
    v.push_back(sc.take<uint32_t>(n + 1));         // 5 rlab
    v.push_back(sc.take<uint32_t>(n + 1));         // 6 match
    v.push_back(sc.take<uint32_t>(4));             // 7 totals (R, Q, C)
    v.push_back(sc.take<uint32_t>(
        scan_scratch_elems(n > mmax ? n : mmax)));  // 8 scan tmp
    v.push_back(sc.take<uint64_t>(n > mmax ? n : mmax));  // 9 keys
    v.push_back(sc.take<uint8_t>(65536));          // 10 presence
    v.push_back(sc.take<uint16_t>(65536));         // 11 class map
    v.push_back(sc.take<uint32_t>(mmax));          // 12 qorder
    v.push_back(sc.take<uint32_t>(256 + 1));       // 13 class offsets
    v.push_back(sc.take<uint32_t>(mmax));          // 14 q heads
    v.push_back(sc.take<uint32_t>(
        2 * (ceil_div(n > mmax ? n : mmax, kBlock) + 1)));  // 15 block heads
    v.push_back(sc.take<uint32_t>(mmax + 1));      // 16 qstart
    v.push_back(sc.take<uint32_t>(mmax + 1));      // 17 qcls
    v.push_back(sc.take<uint32_t>(mmax + 1));      // 18 qlab
    v.push_back(sc.take<uint32_t>(n));             // 19 run of each record
    v.push_back(sc.take<uint32_t>(n));             // 20 its ordinal
  };
  std::vector<void*> v;
  Scratch probe(nullptr);
  layout(probe, v);
  ClassSortLayout probe_sort = class_sort_layout(probe, mmax, 256);
  (void)probe_sort;
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  if (n == 0) return CHOPPER_OK;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  layout(sc, v);
  ClassSortLayout SL = class_sort_layout(sc, mmax, 256);
  uint32_t* rlabv = (uint32_t*)v[0];
  uint32_t *head = (uint32_t*)v[1], *excl = (uint32_t*)v[2];
  uint32_t *rstart = (uint32_t*)v[3], *rcls = (uint32_t*)v[4],
           *rlab = (uint32_t*)v[5], *match = (uint32_t*)v[6];
  uint32_t* tot = (uint32_t*)v[7];
  uint32_t* tmp = (uint32_t*)v[8];
  uint64_t* key = (uint64_t*)v[9];
  uint32_t *rrun = (uint32_t*)v[19], *rord = (uint32_t*)v[20];
  uint8_t* pres = (uint8_t*)v[10];
  uint16_t* cmap = (uint16_t*)v[11];
  uint32_t *qorder = (uint32_t*)v[12], *coff = (uint32_t*)v[13];
  uint32_t* qhead = (uint32_t*)v[14];
  uint32_t* tcnt = (uint32_t*)v[15];
  uint32_t* tpre = tcnt + ceil_div(n > mmax ? n : mmax, kBlock) + 1;
  uint32_t *qstart = (uint32_t*)v[16], *qcls = (uint32_t*)v[17],
           *qlab = (uint32_t*)v[18];
  const dim3 gn = grid_for(n, kBlock);

  // columns no pass fills are zero; no record matched yet
  for (int c = 0; c < 16; ++c)
    if (!((used >> c) & 1u))
      CHOPPER_HIP(launch("join_fill", k_join_fill_u64,
                         dim3((unsigned)std::min<int64_t>(
                             ceil_div(n, (int64_t)kBlock), 4096)),
                         dim3(kBlock), s, counters_out + (int64_t)c * n, n));
  CHOPPER_HIP(launch("join_fill", k_join_fill_u8, gn, dim3(kBlock), s,
                     matched_out, n, (uint32_t*)nullptr));
  // dense classes of the records' (gpu, stream) pairs (one read-back)
  CHOPPER_HIP(launch("join_fill", k_join_fill_u8, dim3(64), dim3(kBlock), s,
                     (uint8_t*)nullptr, (int64_t)0, (uint32_t*)pres));
  CHOPPER_HIP(launch("join_pass_prep", k_join_presence, gn, dim3(kBlock), s,
                     n, rec->gpu, rec->stream, pres));
  CHOPPER_HIP(launch("join_dense", k_join_dense, dim3(1), dim3(kDenseT), s,
                     (const uint8_t*)pres, cmap, tot + 2));
  uint32_t nclass = 0;
  CHOPPER_HIP(read_back(tot + 2, &nclass, sizeof(uint32_t), s));
  // (pass entries of other pairs take one more class)
  if (nclass + 1 > 256) return CHOPPER_EINVAL;
  // the records' runs along `order`
  CHOPPER_HIP(launch("join_labels", k_join_rec_labels, gn, dim3(kBlock), s,
                     n, idx + (int64_t)iter_level * n, nm, mk->label, rlabv));
  const Seq R{order, rec->gpu, rec->stream, rlabv, cmap, n};
  CHOPPER_HIP(launch("join_heads", k_join_heads, gn, dim3(kBlock), s, R,
                     (const uint8_t*)nullptr, head, key, tcnt));
  CHOPPER_HIP(exclusive_scan<uint32_t>(tcnt, tpre, (int64_t)gn.x, tmp, tot,
                                       s));
  CHOPPER_HIP(launch("join_runs", k_join_runs, gn, dim3(kBlock), s, n,
                     (const uint32_t*)head, (const uint32_t*)tpre,
                     (const uint64_t*)key, rstart, rcls, rlab, excl));
  CHOPPER_HIP(launch("join_order", k_join_order, gn, dim3(kBlock), s,
                     (const uint32_t*)tot, (const uint32_t*)rcls,
                     (const uint32_t*)rlab, status));
  CHOPPER_HIP(launch("join_runs", k_join_rec_pos, gn, dim3(kBlock), s, n,
                     order, (const uint32_t*)head, (const uint32_t*)excl,
                     (const uint64_t*)key, (const uint32_t*)rstart, rrun,
                     rord));
  for (int p = 0; p < n_passes; ++p) {
    const chopper_counter_pass& P = passes[p];
    const int64_t m = P.n;
    PassCols C{P.n_cols, p, {0}};
    for (int c = 0; c < P.n_cols; ++c) C.dst[c] = P.dst[c];
    if (m > 0) {
      // stable partition of the pass by class, in its own order (the
      // pass's order is its time: the partition needs no time key)
      ClassSortLayout L = SL;
      L.n = m;
      L.ntiles = sort_tiles(m);
      bool range_err = false;
      KeyRecStream kq{P.gpu, P.stream, nullptr, cmap, (int)nclass + 1};
      rc = class_sort(kq, L, qorder, coff, &range_err, s, 1);
      if (rc != CHOPPER_OK) return rc;
      const Seq Q{qorder, P.gpu, P.stream, P.label, cmap, m};
      const dim3 gm = grid_for(m, kBlock);
      CHOPPER_HIP(launch("join_heads", k_join_heads, gm, dim3(kBlock), s, Q,
                         P.cls, qhead, key, tcnt));
      CHOPPER_HIP(exclusive_scan<uint32_t>(tcnt, tpre, (int64_t)gm.x, tmp,
                                           tot + 1, s));
      CHOPPER_HIP(launch("join_runs", k_join_runs, gm, dim3(kBlock), s, m,
                         (const uint32_t*)qhead, (const uint32_t*)tpre,
                         (const uint64_t*)key, qstart, qcls, qlab,
                         (uint32_t*)nullptr));
      CHOPPER_HIP(launch("join_order", k_join_order, gm, dim3(kBlock), s,
                         (const uint32_t*)(tot + 1), (const uint32_t*)qcls,
                         (const uint32_t*)qlab, status));
    } else {
      CHOPPER_HIP(launch("join_fill", k_join_zero, dim3(1), dim3(1), s,
                         tot + 1));
    }
    CHOPPER_HIP(launch("join_match", k_join_match, gn, dim3(kBlock), s,
                       (const uint32_t*)tot, (const uint32_t*)rcls,
                       (const uint32_t*)rlab, (const uint32_t*)(tot + 1),
                       (const uint32_t*)qcls, (const uint32_t*)qlab, match));
    CHOPPER_HIP(launch("join_gather", k_join_gather, gn, dim3(kBlock), s, n,
                       (const uint32_t*)rrun, (const uint32_t*)rord, rec->cls,
                       (const uint32_t*)rcls, (const uint32_t*)rlab,
                       (const uint32_t*)match, (const uint32_t*)qstart,
                       (const uint32_t*)(tot + 1), m,
                       (const uint32_t*)qorder, (const uint64_t*)key,
                       P.values, C, counters_out, matched_out, status));
  }
  return CHOPPER_OK;
}

}  // namespace chopper
