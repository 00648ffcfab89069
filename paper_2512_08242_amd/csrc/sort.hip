// Stable sorts of items by (class, time) for gfx950.
//
// Fast path: a stable counting-sort pass by class (class ids are dense, at
// most 256) followed by a check that every class run of the output is
// non-decreasing in time.  When the input already lists each class in time
// order -- what a profiler emits per GPU and stream -- that single pass is
// the complete stable sort.
//
// General path: LSD radix sort of packed 64-bit keys (class << T | time -
// tmin) with 8-bit digits.  Every pass: per-tile digit histograms in LDS, a
// device-wide exclusive scan of the digit-major histogram table, then a
// stable scatter whose in-tile ranks come from wave64 ballots (eight
// __ballot calls match lanes with equal digits, popcount of the lower lanes
// gives the rank) and per-wave digit counts in LDS.  Each tile is first
// reordered in LDS so that the global writes of one digit bucket are
// contiguous.
#include "sort.h"
#include "wave.h"

namespace chopper {

constexpr int kSortIpt = 8;
constexpr int kSortTile = kBlock * kSortIpt;

int64_t sort_tiles(int64_t n) { return ceil_div(n, kSortTile); }

// ---------------------------------------------------------------------------
// In-tile stable ranking of up to 256 digit values.
// Items are striped: item j of thread t is tile position j * kBlock + t, so
// tile order is (row j, wave, lane).  Every wave-row counts its digits with
// `nbits` ballots (lanes with equal digits find each other; the lowest one
// records the count), one pass turns the counts of the 8 x 4 (row, wave)
// cells into per-digit exclusive prefixes, and an item's rank is its cell's
// prefix plus the number of equal lanes below it.
// On return count[d] = number of valid items with digit d in the tile,
// start[d] = exclusive prefix of count, rank[j] = stable position of the
// item among equal digits.
// ---------------------------------------------------------------------------
// Lanes among those with v that hold the same digit as this lane.  Rows of
// one or two distinct digits -- the usual case for classes of consecutive
// records -- take two or three ballots; other rows match bit by bit.
__device__ inline uint64_t digit_peers(uint32_t d, bool v, int nbits) {
  const uint64_t vm = __ballot(v);
  if (vm == 0) return 0;
  // (the lanes read are uniform: a lane read, not a permute through LDS)
  const uint32_t d0 = (uint32_t)__builtin_amdgcn_readlane(
      (int)d, __ffsll((long long)vm) - 1);
  const uint64_t m0 = __ballot(v && d == d0);
  if (m0 == vm) return vm;
  const uint64_t rest = vm & ~m0;
  const uint32_t d1 = (uint32_t)__builtin_amdgcn_readlane(
      (int)d, __ffsll((long long)rest) - 1);
  const uint64_t m1 = __ballot(v && d == d1);
  if ((m0 | m1) == vm) return d == d0 ? m0 : m1;
  uint64_t peers = vm;
  for (int b = 0; b < nbits; ++b) {
    const bool bit = (d >> b) & 1u;
    const uint64_t bb = __ballot(bit);
    peers &= bit ? bb : ~bb;
  }
  return peers;
}

struct RankShared {
  uint16_t cell[kSortIpt][kWavesPerBlock][256];   // counts, then prefixes
  uint32_t count[256];
  uint32_t start[256];
};

__device__ inline void tile_rank(const uint32_t (&dig)[kSortIpt],
                                 const bool (&valid)[kSortIpt],
                                 uint32_t (&rank)[kSortIpt], RankShared& sh,
                                 int nbits) {
  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int w = t / kWave;
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  {
    uint4* z = reinterpret_cast<uint4*>(&sh.cell[0][0][0]);
    constexpr int kZ = (int)(sizeof(sh.cell) / sizeof(uint4));
    for (int i = t; i < kZ; i += kBlock) z[i] = make_uint4(0u, 0u, 0u, 0u);
  }
  __syncthreads();
  uint32_t rin[kSortIpt];
#pragma unroll
  for (int j = 0; j < kSortIpt; ++j) {
    const uint32_t d = dig[j];
    const bool v = valid[j];
    const uint64_t peers = digit_peers(d, v, nbits);
    rin[j] = __popcll(peers & lt);
    if (v && rin[j] == 0) sh.cell[j][w][d] = (uint16_t)__popcll(peers);
  }
  __syncthreads();
  {
    // digit t: exclusive prefix over the cells in tile order
    uint32_t acc = 0;
#pragma unroll
    for (int j = 0; j < kSortIpt; ++j)
#pragma unroll
      for (int q = 0; q < kWavesPerBlock; ++q) {
        const uint32_t c = sh.cell[j][q][t];
        sh.cell[j][q][t] = (uint16_t)acc;
        acc += c;
      }
    sh.count[t] = acc;
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kSortIpt; ++j)
    if (valid[j]) rank[j] = sh.cell[j][w][dig[j]] + rin[j];
  uint32_t tot;
  sh.start[t] = block_exclusive(sh.count[t], OpAdd(), 0u, &tot);
  __syncthreads();
}

// number of ballots that separate c classes
__host__ __device__ inline int class_bits(int c) {
  int b = 0;
  while (b < 8 && (1 << b) < c) ++b;
  return b;
}

// ---------------------------------------------------------------------------
// Class-partition fast path
// ---------------------------------------------------------------------------
// Class ids of the tile in the striped arrangement the ranking needs (item
// j of thread t at position j * kBlock + t): loaded eight consecutive items
// per lane and turned around through `s_tmp` (kSortTile bytes; class ids
// are below 256).
template <typename Acc>
__device__ inline void striped_classes(const Acc& acc, int64_t base,
                                       int64_t n, uint8_t* s_tmp,
                                       uint32_t (&dig)[kSortIpt],
                                       bool (&valid)[kSortIpt]) {
  uint32_t d[kSortIpt];
  bool v[kSortIpt];
  cls_block(acc, base + (int64_t)threadIdx.x * kSortIpt, n, d, v);
#pragma unroll
  for (int j = 0; j < kSortIpt; ++j)
    s_tmp[threadIdx.x * kSortIpt + j] = (uint8_t)d[j];
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kSortIpt; ++j) {
    const int q = j * kBlock + (int)threadIdx.x;
    valid[j] = base + q < n;
    dig[j] = valid[j] ? (uint32_t)s_tmp[q] : 0u;
  }
  __syncthreads();
}

// With `unsorted`, also a cheap sufficient test of sortedness on the same
// items, while they are at hand: is the input ordered by (major, time)?
template <typename Acc>
__global__ __launch_bounds__(kBlock) void k_class_hist(Acc acc, int64_t n,
                                                       int64_t ntiles,
                                                       uint32_t* tilehist,
                                                       uint32_t* unsorted) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int nbits = class_bits(acc.nclass());
  const int lane = threadIdx.x & (kWave - 1);
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  // (counts need no order: eight consecutive items per lane, vector loads)
  uint32_t d[kSortIpt];
  bool v[kSortIpt];
  cls_block(acc, base + (int64_t)threadIdx.x * kSortIpt, n, d, v);
  // one LDS add per distinct class of every wave-row
#pragma unroll
  for (int j = 0; j < kSortIpt; ++j) {
    const uint64_t peers = digit_peers(d[j], v[j], nbits);
    if (v[j] && __popcll(peers & lt) == 0)
      atomicAdd(&h[d[j]], (uint32_t)__popcll(peers));
  }
  if (unsorted) {
    // eight consecutive items and the next one per lane
    const int64_t i0 = base + (int64_t)threadIdx.x * kSortIpt;
    bool bad = false;
    if (i0 < n) {
      uint32_t m[9];
      int64_t t[9];
      bool w[9];
      major_time_block(acc, i0, n, m, t, w);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (w[j + 1])
          bad = bad || m[j] > m[j + 1] || (m[j] == m[j + 1] && t[j + 1] < t[j]);
    }
    wave_flag_or(unsorted, bad, 1u);
  }
  __syncthreads();
  if ((int)threadIdx.x < acc.nclass())
    tilehist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = h[threadIdx.x];
}

// Block 0 also writes the class start offsets: coff[c] = first position of
// class c (the scanned table's first tile), coff[C] = n.
template <typename Acc, typename Cols>
__global__ __launch_bounds__(kBlock) void k_class_partition(
    Acc acc, int64_t n, int64_t ntiles, const uint32_t* tileoff,
    uint32_t* out, uint32_t* coff, Cols cols) {
  if (blockIdx.x == 0) {
    const int C = acc.nclass();
    for (int c = threadIdx.x; c <= C; c += kBlock)
      coff[c] = c < C ? tileoff[(int64_t)c * ntiles] : (uint32_t)n;
  }
  __shared__ RankShared sh;
  __shared__ uint32_t s_val[kSortTile];
  __shared__ uint8_t s_dig[kSortTile];
  __shared__ uint32_t s_gbase[256];
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  uint32_t dig[kSortIpt], rank[kSortIpt];
  bool valid[kSortIpt];
  striped_classes(acc, base, n, s_dig, dig, valid);
  tile_rank(dig, valid, rank, sh, class_bits(acc.nclass()));
  if ((int)threadIdx.x < acc.nclass())
    s_gbase[threadIdx.x] =
        tileoff[(int64_t)threadIdx.x * ntiles + blockIdx.x];
  for (int j = 0; j < kSortIpt; ++j) {
    if (!valid[j]) continue;
    uint32_t lp = sh.start[dig[j]] + rank[j];
    s_val[lp] = (uint32_t)(base + (int64_t)j * kBlock + threadIdx.x);
    s_dig[lp] = (uint8_t)dig[j];
  }
  __syncthreads();
  const int64_t tile_n = (n - base) < kSortTile ? (n - base) : kSortTile;
  for (int j = 0; j < kSortIpt; ++j) {
    int q = j * kBlock + threadIdx.x;
    if (q >= tile_n) continue;
    uint32_t d = s_dig[q];
    const int64_t pos = (int64_t)s_gbase[d] + (q - sh.start[d]);
    out[pos] = s_val[q];
    cols.put(pos, s_val[q], d);
  }
}

// (both checks stop reading once some wave has found the answer)
template <typename Acc>
__global__ __launch_bounds__(kBlock) void k_class_verify(Acc acc, int64_t n,
                                                         const uint32_t* perm,
                                                         uint32_t* unsorted) {
  if (__builtin_amdgcn_readfirstlane((int)flag_read(unsorted)) != 0) return;
  int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  bool bad = false;
  if (p + 1 < n) {
    uint32_t a = perm[p], b = perm[p + 1];
    bad = acc.cls(a) == acc.cls(b) && acc.time(b) < acc.time(a);
  }
  wave_flag_or(unsorted, bad, 1u);
}

// ---------------------------------------------------------------------------
// General path: packed keys + LSD radix passes
// ---------------------------------------------------------------------------
template <typename Acc>
__global__ __launch_bounds__(kBlock) void k_time_minmax(Acc acc, int64_t n,
                                                        int64_t* mm) {
  int64_t lo = kI64Max, hi = kI64Min;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kBlock) {
    int64_t t = acc.time(i);
    lo = t < lo ? t : lo;
    hi = t > hi ? t : hi;
  }
  for (int d = kWave / 2; d > 0; d >>= 1) {
    int64_t a = __shfl_xor(lo, d, kWave), b = __shfl_xor(hi, d, kWave);
    lo = a < lo ? a : lo;
    hi = b > hi ? b : hi;
  }
  if ((threadIdx.x & (kWave - 1)) == 0) {
    atomicMin((long long*)&mm[0], (long long)lo);
    atomicMax((long long*)&mm[1], (long long)hi);
  }
}

__global__ void k_init_minmax(int64_t* mm) {
  mm[0] = kI64Max;
  mm[1] = kI64Min;
}

template <typename Acc>
__global__ __launch_bounds__(kBlock) void k_make_keys(Acc acc, int64_t n,
                                                      const int64_t* mm,
                                                      int tbits, uint64_t* key,
                                                      uint32_t* val) {
  int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i >= n) return;
  uint64_t t = (uint64_t)(acc.time(i) - mm[0]);
  uint64_t c = acc.cls(i);
  key[i] = (tbits >= 64 ? 0ull : (c << tbits)) | t;
  val[i] = (uint32_t)i;
}

__global__ __launch_bounds__(kBlock) void k_digit_hist(const uint64_t* key,
                                                       int64_t n, int shift,
                                                       int64_t ntiles,
                                                       uint32_t* tilehist) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  for (int j = 0; j < kSortIpt; ++j) {
    int64_t i = base + (int64_t)j * kBlock + threadIdx.x;
    if (i < n) atomicAdd(&h[(uint32_t)(key[i] >> shift) & 255u], 1u);
  }
  __syncthreads();
  tilehist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = h[threadIdx.x];
}

__global__ __launch_bounds__(kBlock) void k_digit_scatter(
    const uint64_t* key_in, const uint32_t* val_in, int64_t n, int shift,
    int64_t ntiles, const uint32_t* tileoff, uint64_t* key_out,
    uint32_t* val_out) {
  __shared__ RankShared sh;
  __shared__ uint64_t s_key[kSortTile];
  __shared__ uint32_t s_val[kSortTile];
  __shared__ uint32_t s_gbase[256];
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  uint32_t dig[kSortIpt], rank[kSortIpt];
  bool valid[kSortIpt];
  uint64_t k[kSortIpt];
  uint32_t v[kSortIpt];
  for (int j = 0; j < kSortIpt; ++j) {
    int64_t i = base + (int64_t)j * kBlock + threadIdx.x;
    valid[j] = i < n;
    k[j] = valid[j] ? key_in[i] : 0ull;
    v[j] = valid[j] ? val_in[i] : 0u;
    dig[j] = (uint32_t)(k[j] >> shift) & 255u;
  }
  tile_rank(dig, valid, rank, sh, 8);
  s_gbase[threadIdx.x] = tileoff[(int64_t)threadIdx.x * ntiles + blockIdx.x];
  for (int j = 0; j < kSortIpt; ++j) {
    if (!valid[j]) continue;
    uint32_t lp = sh.start[dig[j]] + rank[j];
    s_key[lp] = k[j];
    s_val[lp] = v[j];
  }
  __syncthreads();
  const int64_t tile_n = (n - base) < kSortTile ? (n - base) : kSortTile;
  for (int j = 0; j < kSortIpt; ++j) {
    int q = j * kBlock + threadIdx.x;
    if (q >= tile_n) continue;
    uint64_t kk = s_key[q];
    uint32_t d = (uint32_t)(kk >> shift) & 255u;
    int64_t pos = (int64_t)s_gbase[d] + (q - sh.start[d]);
    if (key_out) key_out[pos] = kk;
    val_out[pos] = s_val[q];
  }
}

// class histogram for more than 256 classes (general path only)
template <typename Acc>
__global__ __launch_bounds__(kBlock) void k_class_count_global(
    Acc acc, int64_t n, uint32_t* counts) {
  int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (i < n) atomicAdd(&counts[acc.cls(i)], 1u);
}

__global__ void k_fill_u32(uint32_t* p, int64_t n, uint32_t v) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = v;
}

__global__ void k_status_set(uint32_t bits, uint32_t* status) {
  atomicOr(status, bits);
}

// ---------------------------------------------------------------------------
// Host driver
// ---------------------------------------------------------------------------
static int bitlen_u64(uint64_t x) {
  int b = 0;
  while (x) { ++b; x >>= 1; }
  return b;
}

ClassSortLayout class_sort_layout(Scratch& sc, int64_t n, int C) {
  ClassSortLayout L;
  L.n = n;
  L.C = C;   // maximum number of classes the tables are sized for
  L.ntiles = sort_tiles(n);
  int64_t hist_elems = (int64_t)(C > 256 ? 256 : C) * L.ntiles;
  int64_t radix_elems = 256 * L.ntiles;
  int64_t tab = hist_elems > radix_elems ? hist_elems : radix_elems;
  if (C > 256 && C > tab) tab = C;
  L.tilehist = sc.take<uint32_t>(tab);
  L.tileoff = sc.take<uint32_t>(tab);
  L.scantmp = sc.take<uint32_t>(scan_scratch_elems(tab));
  L.total = sc.take<uint32_t>(4);
  L.flag = sc.take<uint32_t>(4);
  L.mm = sc.take<int64_t>(2);
  L.key0 = sc.take<uint64_t>(n);
  L.key1 = sc.take<uint64_t>(n);
  L.val0 = sc.take<uint32_t>(n);
  L.val1 = sc.take<uint32_t>(n);
  return L;
}

template <typename Acc, typename Cols>
int class_sort(const Acc& acc, const ClassSortLayout& L, uint32_t* out,
               uint32_t* coff, bool* range_error, hipStream_t s,
               int known_sorted, const Cols& cols, bool* cols_done) {
  if (cols_done) *cols_done = false;
  const int64_t n = L.n;
  const int C = acc.nclass();
  const int64_t T = L.ntiles;
  if (C > L.C) return CHOPPER_EINVAL;
  *range_error = false;
  if (n == 0) {
    CHOPPER_HIP(launch("sort_fill", k_fill_u32, dim3(1), dim3(kBlock), s,
                       coff, (int64_t)(C + 1), 0u));
    return CHOPPER_OK;
  }
  bool sorted = false;
  if (C <= 256) {
    // cheap sufficient test on the input, ordered by (major, time), made
    // by the histogram pass; its read-back is waited for after the
    // partition is queued, which runs either way
    ReadBack rb;
    if (known_sorted < 0)
      CHOPPER_HIP(launch("sort_fill", k_fill_u32, dim3(1), dim3(kBlock), s,
                         L.flag, (int64_t)1, 0u));
    CHOPPER_HIP(launch("sort_class_hist", k_class_hist<Acc>, dim3((unsigned)T),
                       dim3(kBlock), s, acc, n, T, L.tilehist,
                       known_sorted < 0 ? L.flag : (uint32_t*)nullptr));
    if (known_sorted < 0)
      CHOPPER_HIP(read_back_start(L.flag, sizeof(uint32_t), s, &rb));
    CHOPPER_HIP(exclusive_scan<uint32_t>(L.tilehist, L.tileoff, (int64_t)C * T,
                                         L.scantmp, L.total, s));
    CHOPPER_HIP(launch("sort_class_partition", k_class_partition<Acc, Cols>,
                       dim3((unsigned)T), dim3(kBlock), s, acc, n, T,
                       (const uint32_t*)L.tileoff, out, coff, cols));
    if (known_sorted < 0) {
      uint32_t unsorted = 1;
      CHOPPER_HIP(read_back_finish(&rb, &unsorted));
      if (unsorted == 0) known_sorted = 1;
    }
    if (known_sorted == 1) {
      sorted = true;
    } else {
      // the partition may still be the sorted order (e.g. input already in
      // class order): verify the class runs of the output
      CHOPPER_HIP(launch("sort_fill", k_fill_u32, dim3(1), dim3(kBlock), s,
                         L.flag, (int64_t)1, 0u));
      CHOPPER_HIP(launch("sort_class_verify", k_class_verify<Acc>,
                         grid_for(n, kBlock), dim3(kBlock), s, acc, n,
                         (const uint32_t*)out, L.flag));
      uint32_t unsorted = 1;
      CHOPPER_HIP(read_back(L.flag, &unsorted, sizeof(uint32_t), s));
      sorted = (unsorted == 0);
    }
  } else {
    CHOPPER_HIP(launch("sort_fill", k_fill_u32, grid_for(C, kBlock),
                       dim3(kBlock), s, L.tilehist, (int64_t)C, 0u));
    CHOPPER_HIP(launch("sort_class_count", k_class_count_global<Acc>,
                       grid_for(n, kBlock), dim3(kBlock), s, acc, n,
                       L.tilehist));
    CHOPPER_HIP(exclusive_scan<uint32_t>(L.tilehist, coff, (int64_t)C,
                                         L.scantmp, coff + C, s));
  }
  if (sorted) {
    if (cols_done) *cols_done = true;
    return CHOPPER_OK;
  }

  // general path
  CHOPPER_HIP(launch("sort_init_minmax", k_init_minmax, dim3(1), dim3(1), s,
                     L.mm));
  CHOPPER_HIP(launch("sort_time_minmax", k_time_minmax<Acc>,
                     dim3((unsigned)(T < 1024 ? T : 1024)), dim3(kBlock), s,
                     acc, n, L.mm));
  int64_t mm[2];
  CHOPPER_HIP(read_back(L.mm, mm, sizeof(mm), s));
  const int tbits = bitlen_u64((uint64_t)(mm[1] - mm[0]));
  const int cbits = bitlen_u64((uint64_t)(C > 1 ? C - 1 : 0));
  if (tbits + cbits > 64) {
    *range_error = true;
    return CHOPPER_OK;
  }
  CHOPPER_HIP(launch("sort_make_keys", k_make_keys<Acc>, grid_for(n, kBlock),
                     dim3(kBlock), s, acc, n, (const int64_t*)L.mm, tbits,
                     L.key0, L.val0));
  return radix_sort_pairs(L, tbits + cbits, out, nullptr, s);
}

int radix_sort_pairs(const ClassSortLayout& L, int bits, uint32_t* out,
                     uint64_t* keys_out, hipStream_t s) {
  const int64_t n = L.n;
  const int64_t T = L.ntiles;
  if (n == 0) return CHOPPER_OK;
  const int passes = bits <= 0 ? 0 : (bits + 7) / 8;
  uint64_t* kin = L.key0;
  uint64_t* kout = L.key1;
  uint32_t* vin = L.val0;
  uint32_t* vout = L.val1;
  for (int p = 0; p < passes; ++p) {
    const int shift = 8 * p;
    const bool last = (p == passes - 1);
    CHOPPER_HIP(launch("sort_digit_hist", k_digit_hist, dim3((unsigned)T),
                       dim3(kBlock), s, (const uint64_t*)kin, n, shift, T,
                       L.tilehist));
    CHOPPER_HIP(exclusive_scan<uint32_t>(L.tilehist, L.tileoff, 256 * T,
                                         L.scantmp, L.total, s));
    CHOPPER_HIP(launch("sort_digit_scatter", k_digit_scatter,
                       dim3((unsigned)T), dim3(kBlock), s,
                       (const uint64_t*)kin, (const uint32_t*)vin, n, shift, T,
                       (const uint32_t*)L.tileoff, last ? keys_out : kout,
                       last ? out : vout));
    uint64_t* tk = kin; kin = kout; kout = tk;
    uint32_t* tv = vin; vin = vout; vout = tv;
  }
  if (passes == 0) {
    CHOPPER_HIP(hipMemcpyAsync(out, L.val0, sizeof(uint32_t) * n,
                               hipMemcpyDeviceToDevice, s));
    if (keys_out)
      CHOPPER_HIP(hipMemcpyAsync(keys_out, L.key0, sizeof(uint64_t) * n,
                                 hipMemcpyDeviceToDevice, s));
  }
  return CHOPPER_OK;
}

// ---------------------------------------------------------------------------
// Two class partitions of the same items, for input already ordered by
// (major, time): one histogram pass fills both tables (A's classes, then
// B's), one scan covers both, one pass writes both permutations.
// ---------------------------------------------------------------------------
template <typename AccA, typename AccB>
__global__ __launch_bounds__(kBlock) void k_class_hist2(
    AccA a, AccB b, int64_t n, int64_t ntiles, const WaveClasses* wcls,
    uint32_t* tilehist) {
  __shared__ uint32_t h[2][256];
  h[0][threadIdx.x] = 0;
  h[1][threadIdx.x] = 0;
  __syncthreads();
  static_assert(kSortTile == kWavesPerBlock * kWaveTile,
                "a sort tile is four wave tiles");
  if (wcls) {
    // the tile's wave tiles, when each holds at most two classes per key
    // (the same decision in every thread)
    const int64_t w0 = (int64_t)blockIdx.x * kWavesPerBlock;
    const int64_t nw = ceil_div(n, (int64_t)kWaveTile);
    bool few = true;
    for (int q = 0; q < kWavesPerBlock; ++q)
      if (w0 + q < nw)
        few = few && wcls[w0 + q].a1 != kManyClasses &&
              wcls[w0 + q].b1 != kManyClasses;
    if (few) {
      // thread q * 4 + k: wave q, key k / 2, class k % 2
      const int q = (int)threadIdx.x >> 2, k = (int)threadIdx.x & 3;
      if (q < kWavesPerBlock && w0 + q < nw) {
        const WaveClasses& c = wcls[w0 + q];
        const uint32_t raw = k == 0 ? c.a0 : k == 1 ? c.a1 : k == 2 ? c.b0 : c.b1;
        const uint32_t cnt =
            k == 0 ? c.na0 : k == 1 ? c.na1 : k == 2 ? c.nb0 : c.nb1;
        if (cnt > 0)
          atomicAdd(&h[k >> 1][k < 2 ? a.cls_of_raw(raw) : b.cls_of_raw(raw)],
                    cnt);
      }
      __syncthreads();
      const int CA = a.nclass();
      if ((int)threadIdx.x < CA)
        tilehist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = h[0][threadIdx.x];
      if ((int)threadIdx.x < b.nclass())
        tilehist[(int64_t)(CA + threadIdx.x) * ntiles + blockIdx.x] =
            h[1][threadIdx.x];
      return;
    }
  }
  const int lane = threadIdx.x & (kWave - 1);
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  const int nb[2] = {class_bits(a.nclass()), class_bits(b.nclass())};
  // every class id of the tile first (eight consecutive items per lane,
  // vector loads; counts need no order), then the counts
  uint32_t d[2][kSortIpt];
  bool v[kSortIpt];
  cls_block(a, base + (int64_t)threadIdx.x * kSortIpt, n, d[0], v);
  cls_block(b, base + (int64_t)threadIdx.x * kSortIpt, n, d[1], v);
#pragma unroll
  for (int j = 0; j < kSortIpt; ++j) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const uint64_t peers = digit_peers(d[q][j], v[j], nb[q]);
      if (v[j] && __popcll(peers & lt) == 0)
        atomicAdd(&h[q][d[q][j]], (uint32_t)__popcll(peers));
    }
  }
  __syncthreads();
  const int CA = a.nclass();
  if ((int)threadIdx.x < CA)
    tilehist[(int64_t)threadIdx.x * ntiles + blockIdx.x] = h[0][threadIdx.x];
  if ((int)threadIdx.x < b.nclass())
    tilehist[(int64_t)(CA + threadIdx.x) * ntiles + blockIdx.x] =
        h[1][threadIdx.x];
}

// Tiles of at most two classes per key -- nearly every tile of records in
// (gpu, start') order: one GPU's compute and communication streams -- are
// partitioned by a pass of their own: the tile's classes c0 (its first
// item's) and c1 come from its waves' class records; every thread takes
// eight consecutive items and compares their raw codes with c1; one block
// scan of the class-c1 counts of both keys (packed in one word) ranks every
// item; both permutations are laid out in LDS in output order, so that the
// stores are coalesced.  It flags the other tiles, and the general pass
// below (the LDS ranking) does only those.
template <typename AccA, typename AccB>
__global__ __launch_bounds__(kBlock) void k_class_partition2_two(
    AccA a, AccB b, int64_t n, int64_t ntiles, const uint32_t* tileoff,
    const WaveClasses* wcls, uint32_t* outA, uint32_t* outB,
    uint8_t* general) {
  __shared__ uint32_t s_out[2][kSortTile];
  __shared__ uint32_t s_w[kWavesPerBlock];
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  const int tile_n =
      (int)((n - base) < kSortTile ? (n - base) : (int64_t)kSortTile);
  // the tile's classes per key (the same in every thread): wave 0's first
  // class is the tile's first item's
  const int64_t w0 = (int64_t)blockIdx.x * kWavesPerBlock;
  const int64_t nw = ceil_div(n, (int64_t)kWaveTile);
  uint32_t A[2] = {kNone, kNone}, B[2] = {kNone, kNone};
  bool ok = true;
  auto add = [&](uint32_t (&C)[2], uint32_t c, uint32_t cnt) {
    if (c == kManyClasses) ok = false;
    if (!ok || cnt == 0) return;
    if (C[0] == kNone || C[0] == c) C[0] = c;
    else if (C[1] == kNone || C[1] == c) C[1] = c;
    else ok = false;
  };
  for (int q = 0; q < kWavesPerBlock; ++q) {
    if (w0 + q >= nw) break;
    const WaveClasses c = wcls[w0 + q];
    add(A, c.a0, c.na0);
    add(A, c.a1, c.na1);
    add(B, c.b0, c.nb0);
    add(B, c.b1, c.nb1);
  }
  if (threadIdx.x == 0) general[blockIdx.x] = ok ? 0 : 1;
  if (!ok) return;   // (block-uniform)
  const int t = (int)threadIdx.x, lane = t & (kWave - 1), wv = t / kWave;
  uint32_t ra[kSortIpt], rb[kSortIpt];
  a.raw8(base + (int64_t)t * kSortIpt, n, ra);
  b.raw8(base + (int64_t)t * kSortIpt, n, rb);
  uint32_t ma = 0, mb = 0;   // the thread's class-c1 items
#pragma unroll
  for (int j = 0; j < kSortIpt; ++j) {
    const bool v = t * kSortIpt + j < tile_n;
    if (v && ra[j] == A[1]) ma |= 1u << j;
    if (v && rb[j] == B[1]) mb |= 1u << j;
  }
  // class-c1 items before the thread, both keys in one word (at most
  // kSortTile each)
  const uint32_t cnt = ((uint32_t)__popc(ma) << 16) | (uint32_t)__popc(mb);
  const uint32_t incl = wave_incl(cnt, OpAdd(), 0u);
  if (lane == kWave - 1) s_w[wv] = incl;
  __syncthreads();
  uint32_t pre = incl - cnt, tot = 0;
#pragma unroll
  for (int q = 0; q < kWavesPerBlock; ++q) {
    if (q < wv) pre += s_w[q];
    tot += s_w[q];
  }
  const uint32_t n1a = tot >> 16, n1b = tot & 0xFFFFu;
  const uint32_t n0a = (uint32_t)tile_n - n1a, n0b = (uint32_t)tile_n - n1b;
  // output order in LDS: class c0 first, then class c1, each by rank
#pragma unroll
  for (int j = 0; j < kSortIpt; ++j) {
    const uint32_t pos = (uint32_t)(t * kSortIpt + j);
    if ((int)pos >= tile_n) continue;
    const uint32_t lo = (1u << j) - 1u;
    const uint32_t r1a = (pre >> 16) + (uint32_t)__popc(ma & lo);
    const uint32_t r1b = (pre & 0xFFFFu) + (uint32_t)__popc(mb & lo);
    s_out[0][((ma >> j) & 1u) ? n0a + r1a : pos - r1a] = (uint32_t)base + pos;
    s_out[1][((mb >> j) & 1u) ? n0b + r1b : pos - r1b] = (uint32_t)base + pos;
  }
  // B's rows of the table follow A's; its scanned values include A's n
  const int64_t CA = a.nclass();
  const uint32_t ga0 =
      tileoff[(int64_t)a.cls_of_raw(A[0]) * ntiles + blockIdx.x];
  const uint32_t ga1 =
      A[1] != kNone ? tileoff[(int64_t)a.cls_of_raw(A[1]) * ntiles +
                              blockIdx.x]
                    : 0u;
  const uint32_t gb0 =
      tileoff[(CA + b.cls_of_raw(B[0])) * ntiles + blockIdx.x] - (uint32_t)n;
  const uint32_t gb1 =
      B[1] != kNone
          ? tileoff[(CA + b.cls_of_raw(B[1])) * ntiles + blockIdx.x] -
                (uint32_t)n
          : 0u;
  __syncthreads();
  for (int k = t; k < tile_n; k += kBlock) {
    const uint32_t uk = (uint32_t)k;
    outA[(int64_t)(uk < n0a ? ga0 + uk : ga1 + (uk - n0a))] = s_out[0][k];
    outB[(int64_t)(uk < n0b ? gb0 + uk : gb1 + (uk - n0b))] = s_out[1][k];
  }
}

template <typename AccA, typename AccB>
__global__ __launch_bounds__(kBlock) void k_class_partition2(
    AccA a, AccB b, int64_t n, int64_t ntiles, const uint32_t* tileoff,
    uint32_t* outA, uint32_t* outB, uint32_t* coffA, uint32_t* coffB,
    const uint8_t* general) {
  if (blockIdx.x == 0) {
    // class start offsets of both sorts (B's scanned values include A's n)
    const int CA = a.nclass(), CB = b.nclass();
    for (int c = threadIdx.x; c <= CA; c += kBlock)
      coffA[c] = c < CA ? tileoff[(int64_t)c * ntiles] : (uint32_t)n;
    for (int c = threadIdx.x; c <= CB; c += kBlock)
      coffB[c] = c < CB ? tileoff[(int64_t)(CA + c) * ntiles] - (uint32_t)n
                        : (uint32_t)n;
  }
  if (!general[blockIdx.x]) return;   // done by the two-class pass
  __shared__ RankShared sh;
  __shared__ uint32_t s_val[kSortTile];
  __shared__ uint8_t s_dig[kSortTile];
  __shared__ uint32_t s_gbase[256];
  const int64_t base = (int64_t)blockIdx.x * kSortTile;
  const int64_t tile_n = (n - base) < kSortTile ? (n - base) : kSortTile;
  uint32_t da[kSortIpt], db[kSortIpt], rank[kSortIpt];
  bool valid[kSortIpt];
  striped_classes(a, base, n, s_dig, da, valid);
  striped_classes(b, base, n, s_dig, db, valid);
  const int CA = a.nclass();
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const uint32_t(&dig)[kSortIpt] = q == 0 ? da : db;
    const int C = q == 0 ? CA : b.nclass();
    tile_rank(dig, valid, rank, sh, class_bits(C));
    // B's rows of the table follow A's; its scanned values include A's n
    const int64_t row0 = q == 0 ? 0 : CA;
    const uint32_t sub = q == 0 ? 0u : (uint32_t)n;
    if ((int)threadIdx.x < C)
      s_gbase[threadIdx.x] =
          tileoff[(row0 + threadIdx.x) * ntiles + blockIdx.x] - sub;
    for (int j = 0; j < kSortIpt; ++j) {
      if (!valid[j]) continue;
      const uint32_t lp = sh.start[dig[j]] + rank[j];
      s_val[lp] = (uint32_t)(base + (int64_t)j * kBlock + threadIdx.x);
      s_dig[lp] = (uint8_t)dig[j];
    }
    __syncthreads();
    uint32_t* out = q == 0 ? outA : outB;
    for (int j = 0; j < kSortIpt; ++j) {
      const int qq = j * kBlock + threadIdx.x;
      if (qq >= tile_n) continue;
      const uint32_t d = s_dig[qq];
      out[(int64_t)s_gbase[d] + (qq - sh.start[d])] = s_val[qq];
    }
    __syncthreads();
  }
}

template <typename AccA, typename AccB>
int class_sort2(const AccA& a, const AccB& b, const ClassSortLayout& L,
                uint32_t* outA, uint32_t* coffA, uint32_t* outB,
                uint32_t* coffB, hipStream_t s, const WaveClasses* wcls) {
  const int64_t n = L.n;
  const int CA = a.nclass(), CB = b.nclass();
  const int64_t T = L.ntiles;
  if (n == 0 || CA > 256 || CB > 256 || CA + CB > 256 || !wcls)
    return CHOPPER_EINVAL;
  CHOPPER_HIP(launch("sort_class_hist", k_class_hist2<AccA, AccB>,
                     dim3((unsigned)T), dim3(kBlock), s, a, b, n, T, wcls,
                     L.tilehist));
  CHOPPER_HIP(exclusive_scan<uint32_t>(L.tilehist, L.tileoff,
                                       (int64_t)(CA + CB) * T, L.scantmp,
                                       L.total, s));
  // (a byte per tile: the radix keys' space is free on this path)
  uint8_t* general = reinterpret_cast<uint8_t*>(L.key0);
  CHOPPER_HIP(launch("sort_class_partition",
                     k_class_partition2_two<AccA, AccB>, dim3((unsigned)T),
                     dim3(kBlock), s, a, b, n, T, (const uint32_t*)L.tileoff,
                     wcls, outA, outB, general));
  CHOPPER_HIP(launch("sort_class_partition", k_class_partition2<AccA, AccB>,
                     dim3((unsigned)T), dim3(kBlock), s, a, b, n, T,
                     (const uint32_t*)L.tileoff, outA, outB, coffA, coffB,
                     (const uint8_t*)general));
  return CHOPPER_OK;
}

template int class_sort2<KeyRecStream, KeyRecKind>(
    const KeyRecStream&, const KeyRecKind&, const ClassSortLayout&, uint32_t*,
    uint32_t*, uint32_t*, uint32_t*, hipStream_t, const WaveClasses*);

template int class_sort<KeyRecStream, NoColumns>(
    const KeyRecStream&, const ClassSortLayout&, uint32_t*, uint32_t*, bool*,
    hipStream_t, int, const NoColumns&, bool*);
template int class_sort<KeyRecKind, NoColumns>(
    const KeyRecKind&, const ClassSortLayout&, uint32_t*, uint32_t*, bool*,
    hipStream_t, int, const NoColumns&, bool*);
template int class_sort<KeyMarker, MarkerColumns>(
    const KeyMarker&, const ClassSortLayout&, uint32_t*, uint32_t*, bool*,
    hipStream_t, int, const MarkerColumns&, bool*);
template int class_sort<KeySeqLabel, NoColumns>(
    const KeySeqLabel&, const ClassSortLayout&, uint32_t*, uint32_t*, bool*,
    hipStream_t, int, const NoColumns&, bool*);

}  // namespace chopper
