// Construction of the bucket index (see bindex.h).
//
//   1-2. one block: per segment the first key, the bucket width (smallest
//      power of two with at most ceil(count / 4) buckets over the key span)
//      and the bucket count, and the scan of the table sizes into offsets;
//   3. every key writes the entries of the buckets that start in the gap
//      after the previous key (at most kFillRun of them, so no thread stalls
//      on a long gap), the last key also the entries after it;
//   4. entries left unset (long gaps only) make a search fall back to the
//      segment's bounds on that side (bi_range).
#include "bindex.h"
#include "wave.h"

namespace chopper {

int64_t bindex_table_cap(int64_t nkeys, int64_t nseg) {
  return nkeys / kKeysPerBucket + 2 * nseg + 2;
}

// One block: every segment's parameters (first key, bucket width: the
// smallest power of two with at most ceil(count / 4) buckets over the key
// span, bucket count) and the exclusive scan of the table sizes; segments
// that would not fit the table keep no table and are searched whole.
// With `clear`, every block of the grid first clears its share of the
// whole table (block 0 then computes the parameters).
__global__ __launch_bounds__(1024) void k_bi_params(
    const int64_t* key, const uint32_t* sbeg, const uint32_t* send, int stride,
    int nseg, BSeg* segs, int64_t cap, uint32_t* total, uint32_t* clear) {
  __shared__ uint32_t s_w[1024 / kWave];
  if (clear)
    for (int64_t e = (int64_t)blockIdx.x * 1024 + threadIdx.x; e < cap;
         e += (int64_t)gridDim.x * 1024)
      clear[e] = kUnset;
  if (blockIdx.x != 0) return;   // block-uniform
  const int lane = lane_id(), w = (int)(threadIdx.x / kWave);
  uint64_t carry = 0;
  for (int base = 0; base < nseg; base += 1024) {
    const int sidx = base + (int)threadIdx.x;
    BSeg P;
    P.lo = 0;
    P.sb = P.se = 0;
    P.shift = 0;
    P.nb = 0;
    P.toff = 0;
    P.pad = 0;
    uint32_t ent = 0;
    if (sidx < nseg) {
      P.sb = sbeg[(int64_t)sidx * stride];
      P.se = send[(int64_t)sidx * stride];
      if (P.se > P.sb) {
        const int64_t cnt = (int64_t)P.se - P.sb;
        P.lo = key[P.sb];
        bi_geometry(P.lo, key[P.se - 1], cnt, &P.shift, &P.nb);
        ent = P.nb + 1;
      }
    }
    const uint32_t incl = wave_incl(ent, OpAdd(), 0u);
    if (lane == kWave - 1) s_w[w] = incl;
    __syncthreads();
    uint64_t pre = carry, tot = carry;
    for (int q = 0; q < 1024 / kWave; ++q) {
      if (q < w) pre += s_w[q];
      tot += s_w[q];
    }
    pre += incl - ent;
    if (sidx < nseg) {
      // offsets are stored for every segment, so they never decrease
      P.toff = (uint32_t)(pre < (uint64_t)cap ? pre : cap);
      if (pre + ent > (uint64_t)cap) P.nb = 0;
      segs[sidx] = P;
    }
    carry = tot;
    __syncthreads();
  }
  if (threadIdx.x == 0) *total = (uint32_t)(carry < (uint64_t)cap ? carry : cap);
}

__global__ __launch_bounds__(kBlock) void k_bi_clear(uint32_t* table,
                                                     const uint32_t* total) {
  const int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (e < (int64_t)*total) table[e] = kUnset;
}

// Eight consecutive keys per thread (vector loads when the chunk is whole
// and aligned); the segment parameters come from LDS when they fit.
constexpr int kFillIpt = 8;
constexpr int kFillLdsSegs = 512;
__global__ __launch_bounds__(kBlock) void k_bi_fill(
    const int64_t* key, const uint32_t* keyseg, int64_t nkeys,
    const uint32_t* nkeys_dev, const BSeg* segs, int nseg, uint32_t* table) {
  __shared__ BSeg s_seg[kFillLdsSegs];
  const bool lds = nseg <= kFillLdsSegs;
  if (lds) {
    for (int i = threadIdx.x; i < nseg; i += kBlock) s_seg[i] = segs[i];
    __syncthreads();
  }
  int64_t nk = nkeys;
  if (nkeys_dev && (int64_t)*nkeys_dev < nk) nk = (int64_t)*nkeys_dev;
  const int64_t i0 = ((int64_t)blockIdx.x * kBlock + threadIdx.x) * kFillIpt;
  if (i0 >= nk) return;
  int64_t k[kFillIpt + 1];
  uint32_t sg[kFillIpt];
  const bool whole = i0 + kFillIpt <= nk && ((uintptr_t)key & 15) == 0 &&
                     ((uintptr_t)keyseg & 15) == 0;
  if (whole) {
#pragma unroll
    for (int j = 0; j < kFillIpt; j += 2) {
      const longlong2 v = *(const longlong2*)(key + i0 + j);
      k[j + 1] = v.x;
      k[j + 2] = v.y;
    }
#pragma unroll
    for (int j = 0; j < kFillIpt; j += 4) {
      const uint4 v = *(const uint4*)(keyseg + i0 + j);
      sg[j] = v.x;
      sg[j + 1] = v.y;
      sg[j + 2] = v.z;
      sg[j + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < kFillIpt; ++j) {
      const bool in = i0 + j < nk;
      k[j + 1] = in ? key[i0 + j] : 0;
      sg[j] = in ? keyseg[i0 + j] : kNone;
    }
  }
  k[0] = i0 > 0 ? key[i0 - 1] : 0;
#pragma unroll
  for (int j = 0; j < kFillIpt; ++j) {
    const int64_t i = i0 + j;
    const uint32_t sidx = sg[j];
    if (sidx == kNone || sidx >= (uint32_t)nseg) continue;
    const BSeg P = lds ? s_seg[sidx] : segs[sidx];
    if (P.nb == 0 || i < P.sb || i >= P.se) continue;
    const int64_t bi = bi_bucket(P, k[j + 1]);
    const int64_t bp = i == P.sb ? -1 : bi_bucket(P, k[j]);
    bi_fill_range(table, P, bp, bi, (uint32_t)i);
    if (i == (int64_t)P.se - 1) bi_fill_range(table, P, bi, P.nb, P.se);
  }
}

hipError_t bindex_build(const int64_t* key, const uint32_t* keyseg,
                        int64_t nkeys, const uint32_t* nkeys_dev,
                        const uint32_t* sbeg, const uint32_t* send, int stride,
                        int nseg, BSeg* segs, uint32_t* table,
                        int64_t table_cap, uint32_t* tmp, hipStream_t s,
                        bool cleared) {
  if (nseg <= 0) return hipSuccess;
  uint32_t* total = tmp + nseg;
  hipError_t e;
  e = launch("bi_params", k_bi_params, dim3(1), dim3(1024), s, key, sbeg, send,
             stride, nseg, segs, table_cap, total, (uint32_t*)nullptr);
  if (e != hipSuccess) return e;
  if (!cleared) {
    e = launch("bi_clear", k_bi_clear, grid_for(table_cap, kBlock),
               dim3(kBlock), s, table, (const uint32_t*)total);
    if (e != hipSuccess) return e;
  }
  if (nkeys > 0) {
    e = launch("bi_fill", k_bi_fill, grid_for(nkeys, kBlock * kFillIpt),
               dim3(kBlock), s, key, keyseg, nkeys, nkeys_dev,
               (const BSeg*)segs, nseg, table);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t bindex_prepare(const int64_t* key, const uint32_t* sbeg,
                          const uint32_t* send, int stride, int nseg,
                          BSeg* segs, uint32_t* table, int64_t table_cap,
                          uint32_t* tmp, hipStream_t s) {
  if (nseg <= 0) return hipSuccess;
  int64_t gx = ceil_div(table_cap, (int64_t)1024 * 4);
  gx = gx < 1 ? 1 : (gx > 1024 ? 1024 : gx);
  return launch("bi_params", k_bi_params, dim3((unsigned)gx), dim3(1024), s,
                key, sbeg, send, stride, nseg, segs, table_cap, tmp + nseg,
                table);
}

}  // namespace chopper
