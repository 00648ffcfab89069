// Bucket index over a segmented sorted key array.
//
// Every segment [sb, se) of non-decreasing int64 keys gets a table of
// power-of-two time buckets: entry b is the first position whose key is at
// least lo + (b << shift), entry nb is se.  The number of buckets is about
// a quarter of the keys, so a search for the last key <= t reads the
// segment's parameters, two adjacent table entries and then binary-searches
// the few keys of one bucket; a skewed key distribution only makes some
// buckets wider, never worse than a plain binary search of the segment.
#pragma once

#include "common.h"

namespace chopper {

struct BSeg {
  int64_t lo;        // first key of the segment
  uint32_t sb, se;   // positions of the segment's keys
  uint32_t shift;    // log2 of the bucket width
  uint32_t nb;       // buckets; 0: no table, search the whole segment
  uint32_t toff;     // first table entry of the segment
  uint32_t pad;
};

// table entries that no key wrote (inside a gap longer than the fill run)
constexpr uint32_t kUnset = 0xFFFFFFFFu;
// about one bucket per kKeysPerBucket keys; a key writes at most kFillRun
// entries, so no thread stalls on a long gap
constexpr int kKeysPerBucket = 4;
constexpr int kFillRun = 256;

struct BIndex {
  const int64_t* key;
  const BSeg* seg;
  const uint32_t* table;
};

// first position in [lo, hi) with key > t
__device__ inline int64_t bi_bsearch(const int64_t* key, int64_t lo,
                                     int64_t hi, int64_t t) {
  while (lo < hi) {
    const int64_t mid = lo + ((hi - lo) >> 1);
    if (key[mid] <= t) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// K searches in lockstep, so that their loads overlap: on return lo[k] is
// the first position in [lo[k], hi[k]) with key > t[k].
template <int K>
__device__ inline void bsearch_k(const int64_t* key, int64_t (&lo)[K],
                                 int64_t (&hi)[K], const int64_t (&t)[K]) {
  for (;;) {
    bool act = false;
    int64_t mid[K], v[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      mid[k] = lo[k] + ((hi[k] - lo[k]) >> 1);
      if (lo[k] < hi[k]) {
        act = true;
        v[k] = key[mid[k]];
      }
    }
    if (!act) break;
#pragma unroll
    for (int k = 0; k < K; ++k) {
      if (lo[k] < hi[k]) {
        if (v[k] <= t[k]) lo[k] = mid[k] + 1;
        else hi[k] = mid[k];
      }
    }
  }
}

// Bucket width (log2) and count of a segment of cnt keys from lo to last:
// the smallest power of two with at most ceil(cnt / kKeysPerBucket)
// buckets over the span.  Any cnt gives a valid index; it only sets the
// bucket width.
__device__ inline void bi_geometry(int64_t lo, int64_t last, int64_t cnt,
                                   uint32_t* shift, uint32_t* nb) {
  const int64_t d = (int64_t)((uint64_t)last - (uint64_t)lo);
  const uint64_t span = d > 0 ? (uint64_t)d : 0;
  const uint64_t target =
      (uint64_t)((cnt + kKeysPerBucket - 1) / kKeysPerBucket);
  uint32_t k = 0;
  while (k < 63 && (span >> k) + 1 > target) ++k;
  *shift = k;
  *nb = (uint32_t)((span >> k) + 1);
}

// Bucket of a key, clamped to the table (keys are sorted, so the clamp only
// guards against inputs that are not).
__device__ inline int64_t bi_bucket(const BSeg& P, int64_t kv) {
  const uint64_t d = (uint64_t)kv - (uint64_t)P.lo;
  if ((int64_t)d < 0) return 0;
  const uint64_t b = d >> P.shift;
  return b < (uint64_t)P.nb ? (int64_t)b : (int64_t)P.nb - 1;
}

// Entries bp + 1 .. bi of segment P's table take v, at most kFillRun of
// them (the rest of a longer gap stays unset).  A key at position i whose
// predecessor in the segment is in bucket bp (-1 for the segment's first
// key) and which is itself in bucket bi writes i this way, and the
// segment's last key also writes se into the entries after its bucket up to
// nb: then entry b is the first position with key >= lo + (b << shift).
__device__ inline void bi_fill_range(uint32_t* table, const BSeg& P,
                                     int64_t bp, int64_t bi, uint32_t v) {
  uint32_t* tb = table + P.toff;
  const int64_t hi = bi < bp + kFillRun ? bi : bp + kFillRun;
  for (int64_t b = bp + 1; b <= hi; ++b) tb[b] = v;
}

// Search range of t in segment P: the answer (first position with key > t)
// lies in [*lo, *hi].
__device__ inline void bi_range(const BIndex& X, const BSeg& P, int64_t t,
                                int64_t* lo, int64_t* hi) {
  if (P.se <= P.sb || t < P.lo) {
    *lo = *hi = P.sb;
    return;
  }
  if (P.nb == 0) {
    *lo = P.sb;
    *hi = P.se;
    return;
  }
  const uint64_t b = ((uint64_t)t - (uint64_t)P.lo) >> P.shift;
  if (b >= P.nb) {
    *lo = *hi = P.se;
    return;
  }
  // an entry inside a long gap is unset: the range then widens to the
  // segment's end on that side, which only costs a longer search
  const uint32_t a = X.table[P.toff + b], c = X.table[P.toff + b + 1];
  *lo = a != kUnset ? (int64_t)a : (int64_t)P.sb;
  *hi = c != kUnset ? (int64_t)c : (int64_t)P.se;
}

// first position of segment s with key > t (the segment's start if none)
__device__ inline int64_t bi_upper(const BIndex& X, uint32_t s, int64_t t) {
  const BSeg P = X.seg[s];
  int64_t lo, hi;
  bi_range(X, P, t, &lo, &hi);
  return bi_bsearch(X.key, lo, hi, t);
}

// Scratch: segment parameters and the table for nkeys keys in nseg segments.
int64_t bindex_table_cap(int64_t nkeys, int64_t nseg);

// Builds the index.  Segment s spans [sbeg[s * stride], send[s * stride]);
// keyseg[i] is the segment of key i or kNone; *nkeys_dev (device) bounds the
// keys actually present when non-null.  `tmp` holds nseg + 1 uint32.  With
// `cleared` the caller has already set all table_cap entries to kUnset (an
// earlier kernel of the same stream, see bindex_clear).
hipError_t bindex_build(const int64_t* key, const uint32_t* keyseg,
                        int64_t nkeys, const uint32_t* nkeys_dev,
                        const uint32_t* sbeg, const uint32_t* send, int stride,
                        int nseg, BSeg* segs, uint32_t* table,
                        int64_t table_cap, uint32_t* tmp, hipStream_t s,
                        bool cleared = false);

// The index without its fill: segment parameters and a cleared table, in
// one launch (block 0 computes the parameters while every block clears).
// The caller then fills the table, every key i of segment P (bucket bi,
// its predecessor's bp) with bi_fill_range(table, P, bp, bi, i), the
// segment's last key also bi_fill_range(table, P, bi, P.nb, P.se).
hipError_t bindex_prepare(const int64_t* key, const uint32_t* sbeg,
                          const uint32_t* send, int stride, int nseg,
                          BSeg* segs, uint32_t* table, int64_t table_cap,
                          uint32_t* tmp, hipStream_t s);

// Part of a grid-stride clear of the table that a kernel of any grid can
// take on: block b of nb clears its share.
__device__ inline void bindex_clear(uint32_t* table, int64_t cap, int64_t b,
                                    int64_t nb) {
  for (int64_t e = b * kBlock + threadIdx.x; e < cap; e += nb * kBlock)
    table[e] = kUnset;
}

}  // namespace chopper
