// chopper_join_counters: counters of serialized hardware-profiling passes
// attached to the runtime trace's kernels (Section III-A: only two or three
// counters per pass, kernels serialized, no valid timestamps; Section III-B:
// alignment attaches the counters to operations, layers and iterations).
//
// A record and a pass entry match on (gpu, stream, iteration label,
// ordinal) and class.  Both sides are brought into (gpu, stream) order --
// the records by `order`, a pass by a stable class partition of its own
// order -- and cut into runs of equal (gpu, stream, label).  When along
// every (gpu, stream) each label is one run and labels increase (what
// iteration markers in time order give), the ordinal is the position
// inside the run.  A side whose run table breaks that (checked on the
// device, one flag word read back for all sides) is first sorted stably by
// (gpu, stream, label), which keeps each label's time order, and cut into
// runs again.  Record runs find their pass run by a binary search over the
// pass's run table; each record then reads entry run start + ordinal.
// Records far from their sorted order are gathered in sorted order through
// a row-major stage instead (one more pass, no scattered column reads).
// JOIN_ORDER (a warning) marks labels that decrease along a (gpu, stream).
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
// (four per lane: more label gathers in flight)
__global__ __launch_bounds__(kBlock) void k_join_rec_labels(
    int64_t n, const uint32_t* idx_iter, int64_t nm, const uint32_t* m_label,
    uint32_t* lab) {
  const int64_t i0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i0 >= n) return;
  uint32_t m[4], l[4];
  const bool full = i0 + 4 <= n && ((uintptr_t)idx_iter & 15) == 0;
  if (full) {
    const uint4 v = *reinterpret_cast<const uint4*>(idx_iter + i0);
    m[0] = v.x; m[1] = v.y; m[2] = v.z; m[3] = v.w;
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) m[j] = i0 + j < n ? idx_iter[i0 + j] : kNone;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) l[j] = (int64_t)m[j] < nm ? m_label[m[j]] : kNone;
  if (full) {
    *reinterpret_cast<uint4*>(lab + i0) = make_uint4(l[0], l[1], l[2], l[3]);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (i0 + j < n) lab[i0 + j] = l[j];
  }
}

// the (gpu, stream) pairs of the records
// Four records per lane (word loads of the byte columns); a pair is written
// only where it differs from the record before: records come in long runs
// of one pair, and equal writes would queue on one byte.
__global__ __launch_bounds__(kBlock) void k_join_presence(
    int64_t n, const uint8_t* gpu, const uint8_t* stream, uint8_t* pres) {
  const int64_t i0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  uint32_t pr[4];
  const bool full = i0 + 4 <= n && ((uintptr_t)gpu & 3) == 0 &&
                    ((uintptr_t)stream & 3) == 0;
  if (full) {
    const uint32_t g4 = *reinterpret_cast<const uint32_t*>(gpu + i0);
    const uint32_t s4 = *reinterpret_cast<const uint32_t*>(stream + i0);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      pr[j] = ((g4 >> (8 * j)) & 255u) * 256u + ((s4 >> (8 * j)) & 255u);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      pr[j] = i0 + j < n ? (uint32_t)gpu[i0 + j] * 256u + stream[i0 + j]
                         : kNone;
  }
  uint32_t prev = wave_shr1_u32(kNone, pr[3]);
  if (lane_id() == 0) prev = kNone;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (pr[j] != kNone && pr[j] != prev) pres[pr[j]] = 1;
    prev = pr[j];
  }
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

// key of a sequence item: label | class << 32
__device__ inline uint64_t item_key(const Seq& S, uint32_t i) {
  return (uint64_t)S.lab[i] | (uint64_t)S.cls(i) << 32;
}

// run heads: an item with an iteration whose predecessor differs in
// (gpu, stream, label) -- items without an iteration belong to no run, and
// one of them between two items of a label starts a second run of it.  The
// key of every position is kept for the later passes, which then read it
// in sequence order.  Each wave takes 256 consecutive positions, four per
// lane (more gathers in flight per wave), and writes the head count of its
// 256 positions (tcnt is per kBlock positions, as k_join_runs reads it).
constexpr int kHeadsIpt = 4;
__global__ __launch_bounds__(kBlock) void k_join_heads(Seq S,
                                                       uint32_t* head,
                                                       uint64_t* key,
                                                       uint32_t* tcnt) {
  const int lane = lane_id();
  const int64_t W = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave;
  const int64_t base = W * (kWave * kHeadsIpt);
  if (base >= S.n) return;                                 // whole wave
  const int64_t p0 = base + (int64_t)lane * kHeadsIpt;
  uint32_t e[kHeadsIpt];
  bool ok[kHeadsIpt];
  // (vector loads only from a 16-byte aligned order)
  if (p0 + kHeadsIpt <= S.n && ((uintptr_t)S.idx & 15) == 0) {
    const uint4 v = *reinterpret_cast<const uint4*>(S.idx + p0);
    e[0] = v.x; e[1] = v.y; e[2] = v.z; e[3] = v.w;
#pragma unroll
    for (int j = 0; j < kHeadsIpt; ++j) ok[j] = true;
  } else {
#pragma unroll
    for (int j = 0; j < kHeadsIpt; ++j) {
      ok[j] = p0 + j < S.n;
      e[j] = ok[j] ? S.idx[p0 + j] : 0u;
    }
  }
  uint64_t k[kHeadsIpt];
#pragma unroll
  for (int j = 0; j < kHeadsIpt; ++j) k[j] = ok[j] ? item_key(S, e[j]) : 0ull;
  // the predecessor of the lane's first position: the lane below's last
  // key; lane 0 reads it
  uint64_t ka = wave_shr1_any((uint64_t)0, k[kHeadsIpt - 1]);
  if (lane == 0 && p0 > 0) ka = item_key(S, S.idx[p0 - 1]);
  uint32_t h[kHeadsIpt];
  uint32_t cnt = 0;
#pragma unroll
  for (int j = 0; j < kHeadsIpt; ++j) {
    const uint64_t prev = j == 0 ? ka : k[j - 1];
    h[j] = (ok[j] && (uint32_t)k[j] != kNone && (p0 + j == 0 || prev != k[j]))
               ? 1u
               : 0u;
    cnt += (uint32_t)__popcll(__ballot(h[j] != 0));
  }
  if (p0 + kHeadsIpt <= S.n) {
    *reinterpret_cast<uint4*>(head + p0) = make_uint4(h[0], h[1], h[2], h[3]);
    ulonglong2* kp = reinterpret_cast<ulonglong2*>(key + p0);
    kp[0] = make_ulonglong2(k[0], k[1]);
    kp[1] = make_ulonglong2(k[2], k[3]);
  } else {
#pragma unroll
    for (int j = 0; j < kHeadsIpt; ++j)
      if (ok[j]) {
        head[p0 + j] = h[j];
        key[p0 + j] = k[j];
      }
  }
  if (lane == 0) tcnt[W] = cnt;
}

// The same for a pass in class order: the class of a position comes from
// the class offsets of the partition (coff[0 .. C]), so only the label and
// the kernel class are read through the permutation.  Each wave takes 256
// consecutive positions, four per lane (more gathers in flight per wave),
// and writes the head count of its 256 positions (tcnt is per kBlock
// positions, as k_join_runs reads it).
__global__ __launch_bounds__(kBlock) void k_join_heads_pass(
    int64_t m, const uint32_t* qorder, const uint32_t* label,
    const uint8_t* kcls, const uint32_t* coff, int C, uint32_t* head,
    uint64_t* key, uint32_t* tcnt) {
  __shared__ uint32_t s_off[256 + 1];
  for (int c = threadIdx.x; c <= C; c += kBlock) s_off[c] = coff[c];
  __syncthreads();
  const int lane = lane_id();
  const int64_t W = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave;
  const int64_t base = W * (kWave * kHeadsIpt);
  if (base >= m) return;                                   // whole wave
  // class of position q: the last c < C with s_off[c] <= q
  auto cls_at = [&](int64_t q) {
    int lo = 0, hi = C;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if ((int64_t)s_off[mid] <= q) lo = mid;
      else hi = mid;
    }
    return (uint32_t)lo;
  };
  const int64_t p0 = base + (int64_t)lane * kHeadsIpt;
  uint32_t e[kHeadsIpt];
  bool ok[kHeadsIpt];
  if (p0 + kHeadsIpt <= m) {
    const uint4 v = *reinterpret_cast<const uint4*>(qorder + p0);
    e[0] = v.x; e[1] = v.y; e[2] = v.z; e[3] = v.w;
#pragma unroll
    for (int j = 0; j < kHeadsIpt; ++j) ok[j] = true;
  } else {
#pragma unroll
    for (int j = 0; j < kHeadsIpt; ++j) {
      ok[j] = p0 + j < m;
      e[j] = ok[j] ? qorder[p0 + j] : 0u;
    }
  }
  uint64_t k[kHeadsIpt];
  uint32_t c = ok[0] ? cls_at(p0) : 0u;
#pragma unroll
  for (int j = 0; j < kHeadsIpt; ++j) {
    if (!ok[j]) {
      k[j] = 0ull;
      continue;
    }
    while ((int)c + 1 < C && (int64_t)s_off[c + 1] <= p0 + j) ++c;
    k[j] = (uint64_t)label[e[j]] | (uint64_t)c << 32 |
           (uint64_t)kcls[e[j]] << 48;
  }
  // the predecessor of the lane's first position: the lane below's last
  // key; lane 0 reads it
  uint64_t ka = wave_shr1_any((uint64_t)0, k[kHeadsIpt - 1]);
  if (lane == 0 && p0 > 0) {
    const uint32_t ep = qorder[p0 - 1];
    ka = (uint64_t)label[ep] | (uint64_t)cls_at(p0 - 1) << 32;
  }
  const uint64_t kMask = 0x0000FFFFFFFFFFFFull;    // class and label
  uint32_t h[kHeadsIpt];
  uint32_t cnt = 0;
#pragma unroll
  for (int j = 0; j < kHeadsIpt; ++j) {
    const uint64_t prev = j == 0 ? ka : k[j - 1];
    h[j] = (ok[j] && (uint32_t)k[j] != kNone &&
            (p0 + j == 0 || ((prev ^ k[j]) & kMask) != 0))
               ? 1u
               : 0u;
    cnt += (uint32_t)__popcll(__ballot(h[j] != 0));
  }
  if (p0 + kHeadsIpt <= m) {
    *reinterpret_cast<uint4*>(head + p0) = make_uint4(h[0], h[1], h[2], h[3]);
    ulonglong2* kp = reinterpret_cast<ulonglong2*>(key + p0);
    kp[0] = make_ulonglong2(k[0], k[1]);
    kp[1] = make_ulonglong2(k[2], k[3]);
  } else {
#pragma unroll
    for (int j = 0; j < kHeadsIpt; ++j)
      if (ok[j]) {
        head[p0 + j] = h[j];
        key[p0 + j] = k[j];
      }
  }
  if (lane == 0) tcnt[W] = cnt;
}

// run table: start position, (gpu, stream) and label of every run, the run
// number of a head being the heads before it (prefix tpre of its 256
// positions + the heads before it among them); excl (optional) gets that
// count at every position.  Each wave takes 256 consecutive positions, four
// per lane, as the heads passes do.
__global__ __launch_bounds__(kBlock) void k_join_runs(
    int64_t n, const uint32_t* head, const uint32_t* tpre,
    const uint64_t* key, uint32_t* rstart, uint32_t* rcls, uint32_t* rlab,
    uint32_t* excl) {
  const int lane = lane_id();
  const int64_t W = (int64_t)blockIdx.x * kWavesPerBlock + threadIdx.x / kWave;
  const int64_t base = W * (kWave * kHeadsIpt);
  if (base >= n) return;                                   // whole wave
  const int64_t p0 = base + (int64_t)lane * kHeadsIpt;
  const bool full = p0 + kHeadsIpt <= n;
  uint32_t h[kHeadsIpt];
  if (full) {
    const uint4 v = *reinterpret_cast<const uint4*>(head + p0);
    h[0] = v.x; h[1] = v.y; h[2] = v.z; h[3] = v.w;
  } else {
#pragma unroll
    for (int j = 0; j < kHeadsIpt; ++j) h[j] = p0 + j < n ? head[p0 + j] : 0u;
  }
  const uint32_t c = h[0] + h[1] + h[2] + h[3];
  uint32_t r = tpre[W] + wave_incl(c, OpAdd(), 0u) - c;
  uint32_t ex[kHeadsIpt];
#pragma unroll
  for (int j = 0; j < kHeadsIpt; ++j) {
    ex[j] = r;
    if (h[j]) {
      const int64_t p = p0 + j;
      const uint64_t k = key[p];
      rstart[r] = (uint32_t)p;
      rcls[r] = (uint32_t)(k >> 32) & 0xFFFFu;
      rlab[r] = (uint32_t)k;
    }
    r += h[j];
  }
  if (!excl) return;
  if (full) {
    *reinterpret_cast<uint4*>(excl + p0) = make_uint4(ex[0], ex[1], ex[2], ex[3]);
  } else {
#pragma unroll
    for (int j = 0; j < kHeadsIpt; ++j)
      if (p0 + j < n) excl[p0 + j] = ex[j];
  }
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

// Run-table check: bit `bit` of *flag when a run's label is not above that
// of the previous run of its (gpu, stream) -- a label in two runs, or labels
// out of order: the side must be sorted by label first; JOIN_ORDER when a
// label is below that of the previous run (labels decrease).  Otherwise the
// table is sorted by (gpu, stream, label) and every label has one run.
// (run tables are short: a fixed grid strides over them)
__global__ void k_join_order(const uint32_t* nruns, const uint32_t* rcls,
                             const uint32_t* rlab, uint32_t* status,
                             uint32_t* flag, uint32_t bit) {
  const int64_t nr = (int64_t)*nruns;
  bool split = false, dec = false;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < nr;
       r += (int64_t)gridDim.x * blockDim.x)
    if (r > 0 && rcls[r - 1] == rcls[r]) {
      split |= rlab[r - 1] >= rlab[r];
      dec |= rlab[r - 1] > rlab[r];
    }
  const uint64_t any_split = __ballot(split), any_dec = __ballot(dec);
  if (lane_id() == 0) {
    if (any_split != 0) atomicOr(flag, bit);
    if (any_dec != 0) atomicOr(status, CHOPPER_ST_JOIN_ORDER);
  }
}

// out[q] = seq[perm[q]]: a sequence reordered by a permutation of its
// positions
__global__ void k_join_compose(int64_t n, const uint32_t* seq,
                               const uint32_t* perm, uint32_t* out) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q < n) out[q] = seq[perm[q]];
}

// pass run of every record run: binary search by (gpu, stream, label); the
// record run gets the class-order positions [start, next run's start) of
// that pass run, or an empty range
__global__ void k_join_match(const uint32_t* nr, const uint32_t* rcls,
                             const uint32_t* rlab, const uint32_t* nq,
                             const uint32_t* qcls, const uint32_t* qlab,
                             const uint32_t* qstart, int64_t m,
                             uint2* match) {
  const int64_t n_r = (int64_t)*nr, n_q = (int64_t)*nq;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < n_r;
       r += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t key = (uint64_t)rcls[r] << 32 | rlab[r];
    int64_t lo = 0, hi = n_q;     // first run with key >= ours
    while (lo < hi) {
      const int64_t mid = (lo + hi) >> 1;
      const uint64_t k = (uint64_t)qcls[mid] << 32 | qlab[mid];
      if (k < key) lo = mid + 1;
      else hi = mid;
    }
    const bool hit =
        lo < n_q && ((uint64_t)qcls[lo] << 32 | qlab[lo]) == key;
    match[r] = hit ? make_uint2(qstart[lo], lo + 1 < n_q
                                                ? qstart[lo + 1]
                                                : (uint32_t)m)
                   : make_uint2(0u, 0u);
  }
}

// one pass as the gather sees it
struct PassView {
  const uint2* match;       // record run -> class-order positions of its
                            // pass run [x, y) (empty: no such run)
  const uint32_t* qorder;   // class-order position -> entry
  const uint64_t* qkey;     // class-order position -> entry key
  const uint64_t* values;   // [n_cols][m]
  int64_t m;
  int32_t n_cols;
  int32_t dst[16];
};

struct JoinPasses {
  int32_t np;
  PassView p[kMaxPasses];
};

// the entry of every pass for a record of run `run` (kNone: the record has
// no iteration) at ordinal `ord`, with run key (kc, kl) and kernel class kk:
// q[p] = entry index, or -1 when none matches.  All entries are found
// before any value is read, so that the passes' dependent loads overlap.
__device__ inline void join_entries(const JoinPasses& J, uint32_t run,
                                    uint32_t ord, uint32_t kc, uint32_t kl,
                                    uint32_t kk, int64_t (&q)[kMaxPasses]) {
#pragma unroll
  for (int p = 0; p < kMaxPasses; ++p) {
    q[p] = -1;
    if (p >= J.np || run == kNone) continue;
    const PassView& P = J.p[p];
    const uint2 qr = P.match[run];
    const int64_t pos = (int64_t)qr.x + ord;
    // the entry at the ordinal is the record's only if it still has the
    // run's key (entries without an iteration may follow the run)
    if (pos < (int64_t)qr.y) {
      const uint64_t k = P.qkey[pos];
      if ((uint32_t)k == kl && ((uint32_t)(k >> 32) & 0xFFFFu) == kc &&
          (uint32_t)(k >> 48) == kk)
        q[p] = P.qorder[pos];
    }
  }
}

// every record, in input order, against every pass: its entry (run start +
// ordinal), the key and class check, and the pass's columns (0 where
// nothing matches); the matched bits are written once
__global__ __launch_bounds__(kBlock) void k_join_gather(
    int64_t n, const uint32_t* rrun, const uint32_t* rord, const uint8_t* cls,
    const uint32_t* rcls, const uint32_t* rlab, JoinPasses J,
    uint64_t* counters, uint8_t* matched, uint32_t* status) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  bool miss = false;
  if (r < n) {
    const uint32_t run = rrun[r];
    uint32_t ord = 0, kc = 0, kl = 0, kk = 0;
    if (run != kNone) {
      ord = rord[r];
      kc = rcls[run];
      kl = rlab[run];
      kk = cls[r];
    }
    int64_t q[kMaxPasses];
    join_entries(J, run, ord, kc, kl, kk, q);
    uint32_t bits = 0;
#pragma unroll
    for (int p = 0; p < kMaxPasses; ++p) {
      if (p >= J.np) break;
      const PassView& P = J.p[p];
      if (run != kNone && q[p] < 0) miss = true;
      for (int c = 0; c < P.n_cols; ++c)
        counters[(int64_t)P.dst[c] * n + r] =
            q[p] >= 0 ? P.values[(int64_t)c * P.m + q[p]] : 0ull;
      if (q[p] >= 0) bits |= 1u << p;
    }
    matched[r] = (uint8_t)bits;
  }
  if (__ballot(miss) != 0 && lane_id() == 0)
    atomicOr(status, CHOPPER_ST_JOIN_MISS);
}

// Records far from their sorted order (e.g. a shuffled trace): the input
// order gather would read every run table and pass column at random.
// Instead the records are taken in their sorted sequence -- run, ordinal
// and the pass entries then advance together -- and each record's values
// go to a row of a row-major stage; a second pass copies every record's
// row (whole cache lines) to the counter columns in input order.
//
// Sampled locality of a sequence: bit `bit` of *flag when, in some sampled
// block of kBlock consecutive positions, more than a quarter of the steps
// jump by more than kNearJump.
constexpr int64_t kNearJump = 4096;
constexpr int kLocalityBlocks = 512;
__global__ __launch_bounds__(kBlock) void k_join_locality(const uint32_t* seq,
                                                          int64_t n,
                                                          int64_t step,
                                                          uint32_t* flag,
                                                          uint32_t bit) {
  const int64_t i = (int64_t)blockIdx.x * step + threadIdx.x;
  bool far = false;
  if (i + 1 < n) {
    const int64_t d = (int64_t)seq[i + 1] - (int64_t)seq[i];
    far = d > kNearJump || d < -kNearJump;
  }
  const int c = __syncthreads_count(far ? 1 : 0);
  if (threadIdx.x == 0 && c > kBlock / 4) atomicOr(flag, bit);
}

// position of every record in the sorted sequence
__global__ void k_join_rec_inv(int64_t n, const uint32_t* seq, uint32_t* pinv) {
  const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (p < n) pinv[seq[p]] = (uint32_t)p;
}

// the gather in sorted order: position p's run and ordinal come from the
// run table (run = heads up to p, ordinal = p - run start); its W values
// go to stage row p.  The block's rows are consecutive in the stage: they
// are put together in LDS and stored as one contiguous block.
__global__ __launch_bounds__(kBlock) void k_join_gather_sorted(
    int64_t n, const uint32_t* seq, const uint32_t* head, const uint32_t* excl,
    const uint64_t* key, const uint32_t* rstart, const uint8_t* cls,
    const uint32_t* rcls, const uint32_t* rlab, JoinPasses J, int W,
    uint64_t* stage, uint8_t* smatched, uint32_t* status) {
  __shared__ uint64_t s_rows[kBlock * 16];
  const int64_t p0 = (int64_t)blockIdx.x * kBlock;
  const int64_t p = p0 + threadIdx.x;
  bool miss = false;
  if (p < n) {
    uint32_t run = kNone, ord = 0, kc = 0, kl = 0, kk = 0;
    if ((uint32_t)key[p] != kNone) {
      run = excl[p] + head[p] - 1;
      ord = (uint32_t)p - rstart[run];
      kc = rcls[run];
      kl = rlab[run];
      kk = cls[seq[p]];
    }
    int64_t q[kMaxPasses];
    join_entries(J, run, ord, kc, kl, kk, q);
    uint64_t* row = s_rows + threadIdx.x * W;
    uint32_t bits = 0;
    int k = 0;
#pragma unroll
    for (int z = 0; z < kMaxPasses; ++z) {
      if (z >= J.np) break;
      const PassView& P = J.p[z];
      if (run != kNone && q[z] < 0) miss = true;
      for (int c = 0; c < P.n_cols; ++c)
        row[k++] = q[z] >= 0 ? P.values[(int64_t)c * P.m + q[z]] : 0ull;
      if (q[z] >= 0) bits |= 1u << z;
    }
    smatched[p] = (uint8_t)bits;
  }
  __syncthreads();
  const int64_t rows = n - p0 < kBlock ? n - p0 : kBlock;
  const int64_t tot = rows * W;
  uint64_t* dst = stage + p0 * (int64_t)W;
  for (int64_t i = threadIdx.x; i < tot; i += kBlock) dst[i] = s_rows[i];
  if (__ballot(miss) != 0 && lane_id() == 0)
    atomicOr(status, CHOPPER_ST_JOIN_MISS);
}

struct StageCols {
  int32_t W;
  int32_t dst[16];    // counter column of stage column k
};

// stage rows back to the records: record r reads row pinv[r]
__global__ __launch_bounds__(kBlock) void k_join_unstage(
    int64_t n, const uint32_t* pinv, const uint64_t* stage,
    const uint8_t* smatched, StageCols S, uint64_t* counters,
    uint8_t* matched) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= n) return;
  const int64_t p = pinv[r];
  const uint64_t* row = stage + p * (int64_t)S.W;
  uint64_t v[16];
  if ((S.W & 1) == 0) {
    // rows of an even width are 16-byte aligned (the stage is 256-aligned)
#pragma unroll
    for (int k = 0; k < 8; ++k)
      if (2 * k < S.W) {
        const uint4 x = reinterpret_cast<const uint4*>(row)[k];
        v[2 * k] = (uint64_t)x.x | (uint64_t)x.y << 32;
        v[2 * k + 1] = (uint64_t)x.z | (uint64_t)x.w << 32;
      }
  } else {
#pragma unroll
    for (int k = 0; k < 16; ++k)
      if (k < S.W) v[k] = row[k];
  }
#pragma unroll
  for (int k = 0; k < 16; ++k)
    if (k < S.W) counters[(int64_t)S.dst[k] * n + r] = v[k];
  matched[r] = smatched[p];
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
  int W = 0;   // stage width: the columns of all passes
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
    W += P.n_cols;
  }
  // scratch: record labels, runs and keys, the class map, per-pass
  // temporaries (reused) and what the gather reads of every pass
  const int64_t nmax = n > mmax ? n : mmax;
  struct PassBuf {
    uint2* match;
    uint32_t *qstart, *qorder, *qcls, *qlab, *coff;
    uint64_t* key;
  };
  struct Bufs {
    uint32_t *rlabv, *head, *excl, *rstart, *rcls, *rlab, *tot, *tmp;
    uint32_t *qhead, *tcnt, *tpre, *rrun, *rord, *perm, *seq2, *scoff, *flag;
    uint64_t *rkey, *stage;
    uint8_t *pres, *smatched;
    uint16_t* cmap;
    PassBuf pb[kMaxPasses];
  } B;
  auto layout = [&](Scratch& sc) {
    B.rlabv = sc.take<uint32_t>(n);
    B.head = sc.take<uint32_t>(n);
    B.excl = sc.take<uint32_t>(n);
    B.rstart = sc.take<uint32_t>(n + 1);
    B.rcls = sc.take<uint32_t>(n + 1);
    B.rlab = sc.take<uint32_t>(n + 1);
    // runs of the records, class count, runs of every pass
    B.tot = sc.take<uint32_t>(2 + kMaxPasses);
    B.tmp = sc.take<uint32_t>(scan_scratch_elems(nmax));
    B.rkey = sc.take<uint64_t>(n);
    B.pres = sc.take<uint8_t>(65536);
    B.cmap = sc.take<uint16_t>(65536);
    B.qhead = sc.take<uint32_t>(mmax);
    B.tcnt = sc.take<uint32_t>(ceil_div(nmax, kBlock) + 1);
    B.tpre = sc.take<uint32_t>(ceil_div(nmax, kBlock) + 1);
    B.rrun = sc.take<uint32_t>(n);
    B.rord = sc.take<uint32_t>(n);
    // re-sort by label of a side whose labels are not one run each
    B.perm = sc.take<uint32_t>(nmax);
    B.seq2 = sc.take<uint32_t>(nmax);
    B.scoff = sc.take<uint32_t>(256 + 1);
    B.flag = sc.take<uint32_t>(1);
    // sorted-order gather of records far from their sorted order
    B.stage = sc.take<uint64_t>(n * (int64_t)W);
    B.smatched = sc.take<uint8_t>(n);
    for (int p = 0; p < n_passes; ++p) {
      const int64_t m = passes[p].n;
      B.pb[p].match = sc.take<uint2>(n + 1);
      B.pb[p].qstart = sc.take<uint32_t>(m + 1);
      B.pb[p].qorder = sc.take<uint32_t>(m);
      B.pb[p].qcls = sc.take<uint32_t>(m + 1);
      B.pb[p].qlab = sc.take<uint32_t>(m + 1);
      B.pb[p].coff = sc.take<uint32_t>(256 + 1);
      B.pb[p].key = sc.take<uint64_t>(m);
    }
  };
  Scratch probe(nullptr);
  layout(probe);
  ClassSortLayout probe_sort = class_sort_layout(probe, nmax, 256);
  (void)probe_sort;
  int rc = scratch_check(scratch, scratch_bytes, probe.used);
  if (rc != 0) return rc > 0 ? CHOPPER_OK : rc;
  if (!status) return CHOPPER_EINVAL;
  if (n == 0) return CHOPPER_OK;
  hipStream_t s = (hipStream_t)stream;
  Scratch sc(scratch);
  layout(sc);
  ClassSortLayout SL = class_sort_layout(sc, nmax, 256);
  const dim3 gn = grid_for(n, kBlock);

  // columns no pass fills are zero
  for (int c = 0; c < 16; ++c)
    if (!((used >> c) & 1u))
      CHOPPER_HIP(launch("join_fill", k_join_fill_u64,
                         dim3((unsigned)std::min<int64_t>(
                             ceil_div(n, (int64_t)kBlock), 4096)),
                         dim3(kBlock), s, counters_out + (int64_t)c * n, n));
  // dense classes of the records' (gpu, stream) pairs (one read-back)
  CHOPPER_HIP(launch("join_fill", k_join_fill_u8, dim3(64), dim3(kBlock), s,
                     (uint8_t*)nullptr, (int64_t)0, (uint32_t*)B.pres));
  CHOPPER_HIP(launch("join_pass_prep", k_join_presence,
                     grid_for(n, kBlock * 4), dim3(kBlock), s,
                     n, rec->gpu, rec->stream, B.pres));
  CHOPPER_HIP(launch("join_dense", k_join_dense, dim3(1), dim3(kDenseT), s,
                     (const uint8_t*)B.pres, B.cmap, B.tot + 1));
  uint32_t nclass = 0;
  CHOPPER_HIP(read_back(B.tot + 1, &nclass, sizeof(uint32_t), s));
  // (pass entries of other pairs take one more class)
  if (nclass + 1 > 256) return CHOPPER_EINVAL;
  // the records' runs along `order`, then each record's run and ordinal
  CHOPPER_HIP(launch("join_labels", k_join_rec_labels,
                     grid_for(n, kBlock * 4), dim3(kBlock), s,
                     n, idx + (int64_t)iter_level * n, nm, mk->label,
                     B.rlabv));
  CHOPPER_HIP(launch("join_fill", k_join_zero, dim3(1), dim3(1), s, B.flag));
  // records far from their sorted order (bit 31, read back with the
  // re-sort bits)
  {
    const int64_t nb = std::min<int64_t>(ceil_div(n, (int64_t)kBlock),
                                         kLocalityBlocks);
    CHOPPER_HIP(launch("join_locality", k_join_locality, dim3((unsigned)nb),
                       dim3(kBlock), s, order, n, n / nb, B.flag,
                       1u << 31));
  }
  const dim3 gr(std::min<unsigned>(gn.x, 1024u));
  const dim3 gw((unsigned)ceil_div((int64_t)gn.x, (int64_t)kWavesPerBlock));
  // run table of the records along `seq`; the check only on the first cut
  auto record_runs = [&](const uint32_t* seq, bool check) -> int {
    const Seq R{seq, rec->gpu, rec->stream, B.rlabv, B.cmap, n};
    CHOPPER_HIP(launch("join_heads", k_join_heads, gw, dim3(kBlock), s, R,
                       B.head, B.rkey, B.tcnt));
    CHOPPER_HIP(exclusive_scan<uint32_t>(B.tcnt, B.tpre, (int64_t)gn.x,
                                         B.tmp, B.tot, s));
    CHOPPER_HIP(launch("join_runs", k_join_runs, gw, dim3(kBlock), s, n,
                       (const uint32_t*)B.head, (const uint32_t*)B.tpre,
                       (const uint64_t*)B.rkey, B.rstart, B.rcls, B.rlab,
                       B.excl));
    if (check)
      CHOPPER_HIP(launch("join_order", k_join_order, gr, dim3(kBlock), s,
                         (const uint32_t*)B.tot, (const uint32_t*)B.rcls,
                         (const uint32_t*)B.rlab, status, B.flag, 1u));
    return CHOPPER_OK;
  };
  // run table of pass p along its class order
  auto pass_runs = [&](int p, bool check) -> int {
    const chopper_counter_pass& P = passes[p];
    const PassBuf& Q_ = B.pb[p];
    const int64_t m = P.n;
    uint32_t* nq = B.tot + 2 + p;
    const dim3 gm = grid_for(m, kBlock);
    const dim3 gmw((unsigned)ceil_div((int64_t)gm.x, (int64_t)kWavesPerBlock));
    CHOPPER_HIP(launch("join_heads", k_join_heads_pass, gmw, dim3(kBlock), s,
                       m, (const uint32_t*)Q_.qorder, P.label, P.cls,
                       (const uint32_t*)Q_.coff, (int)nclass + 1, B.qhead,
                       Q_.key, B.tcnt));
    CHOPPER_HIP(exclusive_scan<uint32_t>(B.tcnt, B.tpre, (int64_t)gm.x,
                                         B.tmp, nq, s));
    CHOPPER_HIP(launch("join_runs", k_join_runs, gmw, dim3(kBlock), s, m,
                       (const uint32_t*)B.qhead, (const uint32_t*)B.tpre,
                       (const uint64_t*)Q_.key, Q_.qstart, Q_.qcls, Q_.qlab,
                       (uint32_t*)nullptr));
    if (check)
      CHOPPER_HIP(launch("join_order", k_join_order,
                         dim3(std::min<unsigned>(gm.x, 1024u)), dim3(kBlock),
                         s, (const uint32_t*)nq, (const uint32_t*)Q_.qcls,
                         (const uint32_t*)Q_.qlab, status, B.flag,
                         2u << p));
    return CHOPPER_OK;
  };
  // stable sort of the positions of `seq` (n items) by (class, label) into
  // B.seq2
  auto sort_by_label = [&](const uint32_t* seq, int64_t cnt,
                           const uint8_t* g, const uint8_t* st,
                           const uint32_t* lab) -> int {
    ClassSortLayout L = SL;
    L.n = cnt;
    L.ntiles = sort_tiles(cnt);
    bool range_err = false;
    const KeySeqLabel acc{seq, g, st, lab, B.cmap, (int)nclass + 1};
    int r = class_sort(acc, L, B.perm, B.scoff, &range_err, s, 0);
    if (r != CHOPPER_OK) return r;
    if (range_err) return CHOPPER_EINVAL;   // 32-bit labels always fit
    CHOPPER_HIP(launch("join_resort", k_join_compose, grid_for(cnt, kBlock),
                       dim3(kBlock), s, cnt, seq, (const uint32_t*)B.perm,
                       B.seq2));
    return CHOPPER_OK;
  };
  rc = record_runs(order, true);
  if (rc != CHOPPER_OK) return rc;
  // every pass: class order, keys and run table
  for (int p = 0; p < n_passes; ++p) {
    const chopper_counter_pass& P = passes[p];
    const PassBuf& Q_ = B.pb[p];
    if (P.n > 0) {
      // stable partition of the pass by class, in its own order (the
      // pass's order is its time: the partition needs no time key)
      ClassSortLayout L = SL;
      L.n = P.n;
      L.ntiles = sort_tiles(P.n);
      bool range_err = false;
      KeyRecStream kq{P.gpu, P.stream, nullptr, B.cmap, (int)nclass + 1};
      rc = class_sort(kq, L, Q_.qorder, Q_.coff, &range_err, s, 1);
      if (rc != CHOPPER_OK) return rc;
      rc = pass_runs(p, true);
      if (rc != CHOPPER_OK) return rc;
    } else {
      CHOPPER_HIP(launch("join_fill", k_join_zero, dim3(1), dim3(1), s,
                         B.tot + 2 + p));
    }
  }
  // sides whose labels are not one run each: sorted by label, cut again
  uint32_t resort = 0;
  CHOPPER_HIP(read_back(B.flag, &resort, sizeof(uint32_t), s));
  const uint32_t* rseq = order;
  if (resort & 1u) {
    rc = sort_by_label(order, n, rec->gpu, rec->stream, B.rlabv);
    if (rc != CHOPPER_OK) return rc;
    rseq = B.seq2;
    rc = record_runs(rseq, false);
    if (rc != CHOPPER_OK) return rc;
  }
  const bool scattered = (resort >> 31) & 1u;
  if (!scattered) {
    CHOPPER_HIP(launch("join_runs", k_join_rec_pos, gn, dim3(kBlock), s, n,
                       rseq, (const uint32_t*)B.head, (const uint32_t*)B.excl,
                       (const uint64_t*)B.rkey, (const uint32_t*)B.rstart,
                       B.rrun, B.rord));
  } else {
    // sorted-order gather: every record's sorted position (in rrun), and
    // the sequence kept in rord when it is the re-sorted one (seq2 is
    // reused by the passes' re-sorts below)
    CHOPPER_HIP(launch("join_runs", k_join_rec_inv, gn, dim3(kBlock), s, n,
                       rseq, B.rrun));
    if (rseq == B.seq2) {
      CHOPPER_HIP(hipMemcpyAsync(B.rord, B.seq2, sizeof(uint32_t) * n,
                                 hipMemcpyDeviceToDevice, s));
      rseq = B.rord;
    }
  }
  // (in input-order mode the records' re-sorted sequence is no longer
  // needed: seq2 is reused)
  JoinPasses J;
  J.np = n_passes;
  for (int p = 0; p < n_passes; ++p) {
    const chopper_counter_pass& P = passes[p];
    const PassBuf& Q_ = B.pb[p];
    const int64_t m = P.n;
    if (m > 0 && ((resort >> (p + 1)) & 1u)) {
      rc = sort_by_label(Q_.qorder, m, P.gpu, P.stream, P.label);
      if (rc != CHOPPER_OK) return rc;
      CHOPPER_HIP(hipMemcpyAsync(Q_.qorder, B.seq2, sizeof(uint32_t) * m,
                                 hipMemcpyDeviceToDevice, s));
      rc = pass_runs(p, false);
      if (rc != CHOPPER_OK) return rc;
    }
    CHOPPER_HIP(launch("join_match", k_join_match, gr, dim3(kBlock), s,
                       (const uint32_t*)B.tot, (const uint32_t*)B.rcls,
                       (const uint32_t*)B.rlab, (const uint32_t*)(B.tot + 2 + p),
                       (const uint32_t*)Q_.qcls, (const uint32_t*)Q_.qlab,
                       (const uint32_t*)Q_.qstart, m, Q_.match));
    PassView& V = J.p[p];
    V.match = Q_.match;
    V.qorder = Q_.qorder;
    V.qkey = Q_.key;
    V.values = P.values;
    V.m = m;
    V.n_cols = P.n_cols;
    for (int c = 0; c < 16; ++c) V.dst[c] = c < P.n_cols ? P.dst[c] : 0;
  }
  if (!scattered) {
    CHOPPER_HIP(launch("join_gather", k_join_gather, gn, dim3(kBlock), s, n,
                       (const uint32_t*)B.rrun, (const uint32_t*)B.rord,
                       rec->cls, (const uint32_t*)B.rcls,
                       (const uint32_t*)B.rlab, J, counters_out, matched_out,
                       status));
    return CHOPPER_OK;
  }
  CHOPPER_HIP(launch("join_gather", k_join_gather_sorted, gn, dim3(kBlock), s,
                     n, rseq, (const uint32_t*)B.head,
                     (const uint32_t*)B.excl, (const uint64_t*)B.rkey,
                     (const uint32_t*)B.rstart, rec->cls,
                     (const uint32_t*)B.rcls, (const uint32_t*)B.rlab, J, W,
                     B.stage, B.smatched, status));
  StageCols SC;
  SC.W = W;
  {
    int k = 0;
    for (int p = 0; p < n_passes; ++p)
      for (int c = 0; c < passes[p].n_cols; ++c) SC.dst[k++] = passes[p].dst[c];
    for (; k < 16; ++k) SC.dst[k] = 0;
  }
  CHOPPER_HIP(launch("join_gather", k_join_unstage, gn, dim3(kBlock), s, n,
                     (const uint32_t*)B.rrun, (const uint64_t*)B.stage,
                     (const uint8_t*)B.smatched, SC, counters_out,
                     matched_out));
  return CHOPPER_OK;
}

}  // namespace chopper
