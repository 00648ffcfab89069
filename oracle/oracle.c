/*
 * CPU ORACLE for the trace pipeline -- TEST INFRASTRUCTURE ONLY.
 *
 * Only tests/, the smoke check and the benchmark's CPU baseline may call this
 * file.  The HIP library never links or calls it, and it shares no code,
 * header, table or helper with that library: each step below is written
 * directly from its definition, single-threaded, with no blocking, fusion or
 * reordering.  Every function names the passage of the paper it follows:
 *
 *   granularities kernel < operation < layer < phase < iteration < GPU < full
 *     workload (Section I, "Proposal");
 *   trace collection with per-kernel start/end and annotations (III-A);
 *   alignment of traces so that counters attach to operations, layers and
 *     iterations (III-B);
 *   aggregation of raw counters and derived metrics, constrained to a
 *     granularity or a selection of GPUs / iterations / operation types
 *     (III-C);
 *   duration = sum of kernel durations, launch overhead = sum of bubbles
 *     before each compute kernel (caption of Fig. "end_to_end");
 *   launch overhead, eqs. (1)-(3), with communication kernels ignored (V-D);
 *   overlap ratio of operations with communication (V-C).
 *
 * Where the paper leaves a choice open, the reading is the one listed in the
 * design notes (clock model and rounding, half-open intervals, attribution by
 * start time, comm-vs-compute by class, gap clamping, row order).
 *
 * Conventions: intervals are half-open [start, end); NONE = 0xFFFFFFFF;
 * kind = 1 (communication) iff class is all_gather (5) or reduce_scatter (6),
 * else 0 (compute).  Status bits: see ORC_* below (same meaning as the
 * library's, by definition of the interface, not by shared code).
 */
#include <stdint.h>
#include <stdlib.h>
#include <math.h>
#include <string.h>

typedef __int128 i128;

#define ORC_NONE 0xFFFFFFFFu

#define ORC_BAD_GPU 1u
#define ORC_BAD_CLASS 2u
#define ORC_NEG_DURATION 4u
#define ORC_MARKER_OVERLAP 8u
#define ORC_RANGE 16u
#define ORC_BAD_LEVEL 64u
#define ORC_PATH_CONFLICT 128u

#define ORC_EOVERFLOW (-3)

static int kind_of(uint8_t cls) { return (cls == 5 || cls == 6) ? 1 : 0; }

/* ------------------------------------------------------------------------ */
/* Clock alignment (III-B; clock model: per-GPU offset plus linear drift)    */
/* ------------------------------------------------------------------------ */

/* round-half-to-even of the exact rational p / q, q > 0, both fit i128. */
static i128 rne_div(i128 p, i128 q) {
  i128 f = p / q, r = p % q;            /* C truncates toward zero */
  if (r < 0) { f -= 1; r += q; }        /* now floor, 0 <= r < q  */
  i128 twice = 2 * r;
  if (twice > q || (twice == q && (f & 1) != 0)) f += 1;
  return f;
}

typedef struct { int64_t x, y; } anchor_t;

static int cmp_anchor(const void* a, const void* b) {
  const anchor_t* p = (const anchor_t*)a;
  const anchor_t* q = (const anchor_t*)b;
  if (p->x != q->x) return p->x < q->x ? -1 : 1;
  if (p->y != q->y) return p->y < q->y ? -1 : 1;
  return 0;
}

/*
 * Least-squares line through a GPU's anchor pairs (local x_j, reference y_j):
 *   y - x  ~  C + D * (x - x0) / 2^48,
 * x0 = smallest local time, D = slope in Q48 and C = intercept, both rounded
 * half-to-even from the exact OLS solution given the rounded D.
 * Returns 0, or ORC_EOVERFLOW when the exact arithmetic guards fail.
 */
int orc_fit(int64_t na, const uint8_t* agpu, const int64_t* ax,
            const int64_t* ay, int32_t n_gpus, int64_t* x0_out,
            int64_t* c_out, int64_t* d_out) {
  anchor_t* buf = (anchor_t*)malloc(sizeof(anchor_t) * (size_t)(na > 0 ? na : 1));
  int rc = 0;
  for (int g = 0; g < n_gpus; ++g) {
    int64_t n = 0;
    for (int64_t j = 0; j < na; ++j)
      if (agpu[j] == g) { buf[n].x = ax[j]; buf[n].y = ay[j]; ++n; }
    x0_out[g] = 0; c_out[g] = 0; d_out[g] = 0;
    if (n == 0) continue;
    qsort(buf, (size_t)n, sizeof(anchor_t), cmp_anchor);
    if (n > ((int64_t)1 << 20)) { rc = ORC_EOVERFLOW; continue; }
    int64_t x0 = buf[0].x;
    i128 su = 0, sw = 0, suu = 0, suw = 0;
    int bad = 0;
    for (int64_t j = 0; j < n; ++j) {
      i128 u = (i128)buf[j].x - x0;
      i128 w = (i128)buf[j].y - buf[j].x;
      if (u >= ((i128)1 << 42) || w >= ((i128)1 << 40) || -w >= ((i128)1 << 40))
        bad = 1;
      su += u; sw += w; suu += u * u; suw += u * w;
    }
    if (bad) { rc = ORC_EOVERFLOW; continue; }
    i128 nn = n;
    i128 num = nn * suw - su * sw;
    i128 den = nn * suu - su * su;
    i128 d = 0;
    if (n > 1 && den != 0) {
      /* D = round(num * 2^48 / den): long division one bit at a time, since
         num * 2^48 itself does not fit in 128 bits. */
      int neg = num < 0;
      i128 a = neg ? -num : num;
      i128 q = a / den, r = a % den;
      if (q >= ((i128)1 << 38)) { rc = ORC_EOVERFLOW; continue; }
      for (int b = 0; b < 48; ++b) {
        r = 2 * r;
        q = 2 * q;
        if (r >= den) { q += 1; r -= den; }
      }
      i128 twice = 2 * r;
      if (twice > den || (twice == den && (q & 1) != 0)) q += 1;
      d = neg ? -q : q;
      if (d >= ((i128)1 << 38) || -d >= ((i128)1 << 38)) {
        rc = ORC_EOVERFLOW; continue;
      }
    }
    i128 cnum = sw * ((i128)1 << 48) - d * su;
    i128 cden = nn * ((i128)1 << 48);
    i128 c = rne_div(cnum, cden);
    x0_out[g] = x0;
    c_out[g] = (int64_t)c;
    d_out[g] = (int64_t)d;
  }
  free(buf);
  return rc;
}

/* floor(p / 2^48) for any sign, written as a plain floor division */
static i128 floor_q48(i128 p) {
  i128 s = (i128)1 << 48;
  i128 q = p / s, r = p % s;
  if (r != 0 && p < 0) q -= 1;
  return q;
}

/*
 * t' = t + C_g + floor((t - x0_g) * D_g / 2^48) for every timestamp of GPU g.
 * Also reports RANGE (|t| >= 2^62 before or after) and BAD_GPU.
 */
uint32_t orc_transform(int64_t n, const uint8_t* gpu, const int64_t* t,
                       int32_t n_gpus, const int64_t* x0, const int64_t* c,
                       const int64_t* d, int64_t* t_out) {
  uint32_t st = 0;
  const i128 lim = (i128)1 << 62;
  for (int64_t k = 0; k < n; ++k) {
    int g = gpu[k];
    if (g >= n_gpus) { st |= ORC_BAD_GPU; t_out[k] = t[k]; continue; }
    i128 v = (i128)t[k] + c[g] + floor_q48(((i128)t[k] - x0[g]) * d[g]);
    if (t[k] >= lim || -(i128)t[k] >= lim || v >= lim || -v >= lim)
      st |= ORC_RANGE;
    t_out[k] = (int64_t)v;
  }
  return st;
}

/* ------------------------------------------------------------------------ */
/* Orders: stable sort by (gpu, stream, start') and by (gpu, kind, start')   */
/* ------------------------------------------------------------------------ */
typedef struct { uint32_t a, b; int64_t t; uint32_t k; } skey_t;

static int cmp_skey(const void* x, const void* y) {
  const skey_t* p = (const skey_t*)x;
  const skey_t* q = (const skey_t*)y;
  if (p->a != q->a) return p->a < q->a ? -1 : 1;
  if (p->b != q->b) return p->b < q->b ? -1 : 1;
  if (p->t != q->t) return p->t < q->t ? -1 : 1;
  if (p->k != q->k) return p->k < q->k ? -1 : 1;  /* ties keep input order */
  return 0;
}

/* by_kind = 0: key (gpu, stream, start'); by_kind = 1: key (gpu, kind, start') */
void orc_order(int64_t n, const uint8_t* gpu, const uint8_t* stream,
               const uint8_t* cls, const int64_t* s, int32_t by_kind,
               uint32_t* out) {
  skey_t* v = (skey_t*)malloc(sizeof(skey_t) * (size_t)(n > 0 ? n : 1));
  for (int64_t k = 0; k < n; ++k) {
    v[k].a = gpu[k];
    v[k].b = by_kind ? (uint32_t)kind_of(cls[k]) : stream[k];
    v[k].t = s[k];
    v[k].k = (uint32_t)k;
  }
  qsort(v, (size_t)n, sizeof(skey_t), cmp_skey);
  for (int64_t p = 0; p < n; ++p) out[p] = v[p].k;
  free(v);
}

/* ------------------------------------------------------------------------ */
/* Attribution (III-A annotations; I granularities): kernel -> marker per    */
/* level by start-time containment                                           */
/* ------------------------------------------------------------------------ */
typedef struct { int64_t s, e; uint32_t id; } mk_t;

static int cmp_mk(const void* x, const void* y) {
  const mk_t* p = (const mk_t*)x;
  const mk_t* q = (const mk_t*)y;
  if (p->s != q->s) return p->s < q->s ? -1 : 1;
  if (p->id != q->id) return p->id < q->id ? -1 : 1;
  return 0;
}

/*
 * For every record k and level l < depth: idx[l*n + k] is the input index of
 * the level-l marker of the record's GPU that contains the record's aligned
 * start, i.e. the last non-empty marker in (start', input index) order with
 * start' <= s'_k, provided s'_k < its end'; otherwise NONE.  Zero-length
 * markers contain no instant and take no part.  MARKER_OVERLAP is raised when
 * two non-empty markers of one (gpu, level) overlap.
 */
uint32_t orc_attribute(int64_t n, const uint8_t* gpu, const int64_t* s,
                       int64_t nm, const uint8_t* mgpu, const uint8_t* mlevel,
                       const int64_t* ms, const int64_t* me, int32_t depth,
                       int32_t n_gpus, uint32_t* idx) {
  uint32_t st = 0;
  for (int64_t j = 0; j < nm; ++j) {
    if (mgpu[j] >= n_gpus) st |= ORC_BAD_GPU;
    if (mlevel[j] >= depth) st |= ORC_BAD_LEVEL;
    if (me[j] < ms[j]) st |= ORC_NEG_DURATION;
  }
  for (int64_t k = 0; k < n; ++k)
    for (int l = 0; l < depth; ++l) idx[(int64_t)l * n + k] = ORC_NONE;
  mk_t* buf = (mk_t*)malloc(sizeof(mk_t) * (size_t)(nm > 0 ? nm : 1));
  for (int g = 0; g < n_gpus; ++g) {
    for (int l = 0; l < depth; ++l) {
      int64_t cnt = 0;
      for (int64_t j = 0; j < nm; ++j)
        if (mgpu[j] == g && mlevel[j] == l && me[j] > ms[j]) {
          buf[cnt].s = ms[j]; buf[cnt].e = me[j]; buf[cnt].id = (uint32_t)j;
          ++cnt;
        }
      qsort(buf, (size_t)cnt, sizeof(mk_t), cmp_mk);
      for (int64_t j = 0; j + 1 < cnt; ++j)
        if (buf[j].e > buf[j + 1].s) st |= ORC_MARKER_OVERLAP;
      for (int64_t k = 0; k < n; ++k) {
        if (gpu[k] != g) continue;
        /* upper_bound: first position whose start' > s'_k */
        int64_t lo = 0, hi = cnt;
        while (lo < hi) {
          int64_t mid = lo + (hi - lo) / 2;
          if (buf[mid].s <= s[k]) lo = mid + 1; else hi = mid;
        }
        int64_t j = lo - 1;
        if (j >= 0 && s[k] < buf[j].e) idx[(int64_t)l * n + k] = buf[j].id;
      }
    }
  }
  free(buf);
  return st;
}

/* ------------------------------------------------------------------------ */
/* Overlap (V-C) and bubbles / launch overhead (Fig. end_to_end, eqs. 1-3)   */
/* ------------------------------------------------------------------------ */
typedef struct { int64_t t; int dc, dm; } ev_t;

static int cmp_ev(const void* x, const void* y) {
  const ev_t* p = (const ev_t*)x;
  const ev_t* q = (const ev_t*)y;
  if (p->t != q->t) return p->t < q->t ? -1 : 1;
  return 0;
}

/* Per-GPU timeline of distinct event times with the state of each segment
   and the cumulative time spent in compute-only (0), comm-only (1) and
   overlapped (2) states before each event time. */
typedef struct {
  int64_t nseg;
  int64_t* t;       /* distinct event times, ascending */
  int* state;       /* state of [t[i], t[i+1]): 0 CO, 1 MO, 2 OV, 3 idle */
  int64_t* cum[3];  /* time in state before t[i] */
} timeline_t;

static void timeline_build(timeline_t* tl, int64_t n, const uint8_t* gpu,
                           const uint8_t* cls, const int64_t* s,
                           const int64_t* e, int g) {
  int64_t cnt = 0;
  for (int64_t k = 0; k < n; ++k)
    if (gpu[k] == g && e[k] > s[k]) cnt += 2;
  ev_t* ev = (ev_t*)malloc(sizeof(ev_t) * (size_t)(cnt > 0 ? cnt : 1));
  int64_t q = 0;
  for (int64_t k = 0; k < n; ++k) {
    if (gpu[k] != g || e[k] <= s[k]) continue;
    int kd = kind_of(cls[k]);
    ev[q].t = s[k]; ev[q].dc = kd ? 0 : 1; ev[q].dm = kd ? 1 : 0; ++q;
    ev[q].t = e[k]; ev[q].dc = kd ? 0 : -1; ev[q].dm = kd ? -1 : 0; ++q;
  }
  qsort(ev, (size_t)cnt, sizeof(ev_t), cmp_ev);
  tl->t = (int64_t*)malloc(sizeof(int64_t) * (size_t)(cnt + 1));
  tl->state = (int*)malloc(sizeof(int) * (size_t)(cnt + 1));
  for (int z = 0; z < 3; ++z)
    tl->cum[z] = (int64_t*)malloc(sizeof(int64_t) * (size_t)(cnt + 1));
  int64_t c = 0, m = 0, ns = 0;
  int64_t acc[3] = {0, 0, 0};
  for (int64_t i = 0; i < cnt;) {
    int64_t t = ev[i].t;
    while (i < cnt && ev[i].t == t) { c += ev[i].dc; m += ev[i].dm; ++i; }
    if (ns > 0) {   /* close the previous segment */
      int stp = tl->state[ns - 1];
      if (stp < 3) acc[stp] += t - tl->t[ns - 1];
    }
    tl->t[ns] = t;
    tl->state[ns] = (c > 0 && m == 0) ? 0 : (c == 0 && m > 0) ? 1
                    : (c > 0 && m > 0) ? 2 : 3;
    for (int z = 0; z < 3; ++z) tl->cum[z][ns] = acc[z];
    ++ns;
  }
  tl->nseg = ns;
  free(ev);
}

static void timeline_free(timeline_t* tl) {
  free(tl->t); free(tl->state);
  for (int z = 0; z < 3; ++z) free(tl->cum[z]);
}

/* time spent in state z (0 CO, 1 MO, 2 OV) strictly before instant t */
static int64_t timeline_F(const timeline_t* tl, int z, int64_t t) {
  int64_t lo = 0, hi = tl->nseg;
  while (lo < hi) {       /* upper_bound of t among event times */
    int64_t mid = lo + (hi - lo) / 2;
    if (tl->t[mid] <= t) lo = mid + 1; else hi = mid;
  }
  int64_t i = lo - 1;
  if (i < 0) return 0;
  int64_t v = tl->cum[z][i];
  if (tl->state[i] == z) v += t - tl->t[i];
  return v;
}

/* window [a, b): out = CO, MO, OV, ID (all zero when b <= a) */
static void timeline_window(const timeline_t* tl, int64_t a, int64_t b,
                            int64_t* out) {
  if (b <= a) { out[0] = out[1] = out[2] = out[3] = 0; return; }
  int64_t tot = 0;
  for (int z = 0; z < 3; ++z) {
    out[z] = timeline_F(tl, z, b) - timeline_F(tl, z, a);
    tot += out[z];
  }
  out[3] = (b - a) - tot;
}

/*
 * ovl[k]: overlapped (compute and comm both active) ns within [s'_k, e'_k).
 * gap[k]: for a compute record, max(0, s'_k - e'_prev) where prev is the
 *   previous compute record in the same (gpu, stream) in (start', index)
 *   order; 0 for comm records and for the first compute record of a stream.
 *   With the host launch time t_l of eqs. (1)-(3), O_prep + O_call equals
 *   this bubble whenever t_l <= t_ks.
 * mwin[4j..]: CO, MO, OV, ID of marker j's aligned window on its GPU.
 * gwin[6g..]: start, end (min start', max end' over the GPU's records, zeros
 *   when it has none), then CO, MO, OV, ID of that window.
 */
uint32_t orc_overlap(int64_t n, const uint8_t* gpu, const uint8_t* stream,
                     const uint8_t* cls, const int64_t* s, const int64_t* e,
                     int64_t nm, const uint8_t* mgpu, const int64_t* ms,
                     const int64_t* me, int32_t n_gpus, int64_t* ovl,
                     int64_t* gap, int64_t* mwin, int64_t* gwin) {
  uint32_t st = 0;
  for (int64_t k = 0; k < n; ++k) {
    if (gpu[k] >= n_gpus) st |= ORC_BAD_GPU;
    if (cls[k] >= 8) st |= ORC_BAD_CLASS;
    if (e[k] < s[k]) st |= ORC_NEG_DURATION;
    ovl[k] = 0;
    gap[k] = 0;
  }
  for (int64_t j = 0; j < nm; ++j)
    for (int z = 0; z < 4; ++z) mwin[4 * j + z] = 0;
  for (int g = 0; g < n_gpus; ++g) {
    timeline_t tl;
    timeline_build(&tl, n, gpu, cls, s, e, g);
    int any = 0;
    int64_t lo = 0, hi = 0;
    for (int64_t k = 0; k < n; ++k) {
      if (gpu[k] != g) continue;
      if (!any || s[k] < lo) lo = s[k];
      if (!any || e[k] > hi) hi = e[k];
      any = 1;
      if (e[k] > s[k])
        ovl[k] = timeline_F(&tl, 2, e[k]) - timeline_F(&tl, 2, s[k]);
    }
    for (int64_t j = 0; j < nm; ++j)
      if (mgpu[j] == g) timeline_window(&tl, ms[j], me[j], &mwin[4 * j]);
    int64_t* gw = &gwin[6 * g];
    gw[0] = any ? lo : 0;
    gw[1] = any ? hi : 0;
    timeline_window(&tl, gw[0], gw[1], &gw[2]);
    timeline_free(&tl);
  }
  /* bubbles: walk each (gpu, stream) in (start', index) order */
  uint32_t* ord = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(n > 0 ? n : 1));
  orc_order(n, gpu, stream, cls, s, 0, ord);
  for (int64_t p = 0; p < n; ++p) {
    uint32_t k = ord[p];
    if (kind_of(cls[k])) continue;
    for (int64_t q = p - 1; q >= 0; --q) {
      uint32_t j = ord[q];
      if (gpu[j] != gpu[k] || stream[j] != stream[k]) break;
      if (kind_of(cls[j])) continue;
      int64_t b = s[k] - e[j];
      gap[k] = b > 0 ? b : 0;
      break;
    }
  }
  free(ord);
  return st;
}

/* ------------------------------------------------------------------------ */
/* Aggregation (III-C) at every granularity (I)                              */
/* ------------------------------------------------------------------------ */
#define ORC_LEVEL_GPU 100
#define ORC_LEVEL_WORKLOAD 101
#define ORC_LEVEL_ALL 255

typedef struct {
  int64_t n_rows;
  int64_t level_offset[16];
  uint32_t status;
  uint32_t* path;   /* [depth][n_rows] */
  uint8_t* gpu;
  uint8_t* kind;
  uint64_t* n;
  int64_t *dur, *gap, *ovl, *tmin, *tmax;
  uint32_t* first;
  uint64_t* ctr;    /* [n_counters][n_rows] */
} orc_rows;

typedef struct {
  uint64_t gpu_mask[4];
  uint32_t class_mask;
  uint32_t use_iter;
  uint32_t iter_lo, iter_hi;
} orc_filter;

/* grouping context for qsort */
static const uint8_t* g_gpu;
static const uint8_t* g_cls;
static const int64_t* g_s;
static const uint32_t* g_idx;
static int64_t g_n;
static int g_plen;      /* number of path entries in the key */
static int g_gpukey;    /* 1: gpu is part of the key */

static int cmp_group(const void* x, const void* y) {
  uint32_t a = *(const uint32_t*)x, b = *(const uint32_t*)y;
  if (g_gpukey && g_gpu[a] != g_gpu[b]) return g_gpu[a] < g_gpu[b] ? -1 : 1;
  for (int l = 0; l < g_plen; ++l) {
    uint32_t pa = g_idx[(int64_t)l * g_n + a], pb = g_idx[(int64_t)l * g_n + b];
    if (pa != pb) return pa < pb ? -1 : 1;
  }
  int ka = kind_of(g_cls[a]), kb = kind_of(g_cls[b]);
  if (ka != kb) return ka < kb ? -1 : 1;
  if (g_s[a] != g_s[b]) return g_s[a] < g_s[b] ? -1 : 1;
  if (a != b) return a < b ? -1 : 1;
  return 0;
}

static int same_group(uint32_t a, uint32_t b) {
  if (g_gpukey && g_gpu[a] != g_gpu[b]) return 0;
  for (int l = 0; l < g_plen; ++l)
    if (g_idx[(int64_t)l * g_n + a] != g_idx[(int64_t)l * g_n + b]) return 0;
  return kind_of(g_cls[a]) == kind_of(g_cls[b]);
}

typedef struct {
  uint32_t gpu, kind;
  int64_t tmin;
  uint32_t first;
  int64_t src;   /* index into the unsorted row arrays */
} rowkey_t;

static int cmp_rowkey(const void* x, const void* y) {
  const rowkey_t* p = (const rowkey_t*)x;
  const rowkey_t* q = (const rowkey_t*)y;
  if (p->gpu != q->gpu) return p->gpu < q->gpu ? -1 : 1;
  if (p->kind != q->kind) return p->kind < q->kind ? -1 : 1;
  if (p->tmin != q->tmin) return p->tmin < q->tmin ? -1 : 1;
  if (p->first != q->first) return p->first < q->first ? -1 : 1;
  return 0;
}

/* slot of record k at level l: deepest non-NONE path entry in 0..l */
static uint32_t slot_of(const uint32_t* idx, int64_t n, int64_t k, int l) {
  for (int j = l; j >= 0; --j)
    if (idx[(int64_t)j * n + k] != ORC_NONE) return idx[(int64_t)j * n + k];
  return ORC_NONE;
}

static int g_lvl;
static int cmp_slot(const void* x, const void* y) {
  uint32_t a = *(const uint32_t*)x, b = *(const uint32_t*)y;
  if (g_gpu[a] != g_gpu[b]) return g_gpu[a] < g_gpu[b] ? -1 : 1;
  uint32_t sa = slot_of(g_idx, g_n, a, g_lvl), sb = slot_of(g_idx, g_n, b, g_lvl);
  if (sa != sb) return sa < sb ? -1 : 1;
  int ka = kind_of(g_cls[a]), kb = kind_of(g_cls[b]);
  if (ka != kb) return ka < kb ? -1 : 1;
  for (int l = 0; l <= g_lvl; ++l) {
    uint32_t pa = g_idx[(int64_t)l * g_n + a], pb = g_idx[(int64_t)l * g_n + b];
    if (pa != pb) return pa < pb ? -1 : 1;
  }
  return 0;
}

/*
 * Rows at one level: the filtered records grouped by
 *   level l in [0, depth):  (gpu, idx_0 .. idx_l, kind)
 *   GPU level:              (gpu, kind)
 *   workload level:         (kind)
 * Per group: record count n, sum of durations e'-s', sum of gaps, sum of
 * overlapped ns, min start', max end', counters summed modulo 2^64, and
 * first = smallest input index among the group's records with start' = min
 * start'.  Rows are ordered by (gpu, kind, min start', first); workload rows
 * carry gpu 0xFF.  Each level is computed from the records, never from
 * another level.  PATH_CONFLICT: at a requested marker level l, two kept
 * records share (gpu, deepest non-NONE marker among levels 0..l, kind) but
 * not the whole path 0..l, so grouping by that marker would merge different
 * groups (markers not nested).
 */
int orc_aggregate(int64_t n, const uint8_t* gpu, const uint8_t* cls,
                  const int64_t* s, const int64_t* e, const uint32_t* idx,
                  const int64_t* gap, const int64_t* ovl,
                  const uint64_t* ctr, int32_t n_counters, int32_t depth,
                  int32_t level, const orc_filter* filt,
                  const uint32_t* mlabel, int64_t nm, orc_rows* out) {
  memset(out, 0, sizeof(*out));
  int levels[16];
  int nlev = 0;
  if (level == ORC_LEVEL_ALL) {
    for (int l = 0; l < depth; ++l) levels[nlev++] = l;
    levels[nlev++] = ORC_LEVEL_GPU;
    levels[nlev++] = ORC_LEVEL_WORKLOAD;
  } else {
    levels[nlev++] = level;
  }
  /* filtered record list (selection of GPUs, classes, iterations; III-C) */
  uint32_t* sel = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(n > 0 ? n : 1));
  int64_t ns = 0;
  for (int64_t k = 0; k < n; ++k) {
    if (filt) {
      int g = gpu[k];
      if (!((filt->gpu_mask[g >> 6] >> (g & 63)) & 1u)) continue;
      if (cls[k] >= 32 || !((filt->class_mask >> cls[k]) & 1u)) continue;
      if (filt->use_iter) {
        uint32_t m0 = depth > 0 ? idx[k] : ORC_NONE;
        if (m0 == ORC_NONE || (int64_t)m0 >= nm) continue;
        if (mlabel[m0] < filt->iter_lo || mlabel[m0] > filt->iter_hi) continue;
      }
    }
    sel[ns++] = (uint32_t)k;
  }
  /* path-conflict check at every requested marker level */
  g_gpu = gpu; g_cls = cls; g_s = s; g_idx = idx; g_n = n;
  uint32_t* tmp = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(ns > 0 ? ns : 1));
  for (int l = 0; l < depth; ++l) {
    if (level != ORC_LEVEL_ALL && level != l) continue;
    memcpy(tmp, sel, sizeof(uint32_t) * (size_t)ns);
    g_lvl = l;
    qsort(tmp, (size_t)ns, sizeof(uint32_t), cmp_slot);
    for (int64_t i = 1; i < ns; ++i) {
      uint32_t a = tmp[i - 1], b = tmp[i];
      if (gpu[a] != gpu[b] || slot_of(idx, n, a, l) != slot_of(idx, n, b, l) ||
          kind_of(cls[a]) != kind_of(cls[b]))
        continue;
      for (int j = 0; j <= l; ++j)
        if (idx[(int64_t)j * n + a] != idx[(int64_t)j * n + b])
          out->status |= ORC_PATH_CONFLICT;
    }
  }
  /* rows per level; capacity: at most ns rows per level */
  int64_t cap = ns * nlev + 1;
  out->path = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(cap * (depth > 0 ? depth : 1)));
  out->gpu = (uint8_t*)malloc((size_t)cap);
  out->kind = (uint8_t*)malloc((size_t)cap);
  out->n = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)cap);
  out->dur = (int64_t*)malloc(sizeof(int64_t) * (size_t)cap);
  out->gap = (int64_t*)malloc(sizeof(int64_t) * (size_t)cap);
  out->ovl = (int64_t*)malloc(sizeof(int64_t) * (size_t)cap);
  out->tmin = (int64_t*)malloc(sizeof(int64_t) * (size_t)cap);
  out->tmax = (int64_t*)malloc(sizeof(int64_t) * (size_t)cap);
  out->first = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)cap);
  out->ctr = (uint64_t*)malloc(sizeof(uint64_t) * (size_t)(cap * (n_counters > 0 ? n_counters : 1)));
  /* temporary unsorted rows of one level */
  rowkey_t* rk = (rowkey_t*)malloc(sizeof(rowkey_t) * (size_t)(ns > 0 ? ns : 1));
  int64_t* bstart = (int64_t*)malloc(sizeof(int64_t) * (size_t)(ns + 1));
  int64_t nrows = 0;
  for (int li = 0; li < nlev; ++li) {
    int lv = levels[li];
    int slot = (lv == ORC_LEVEL_GPU) ? depth : (lv == ORC_LEVEL_WORKLOAD)
               ? depth + 1 : lv;
    out->level_offset[slot] = nrows;
    memcpy(tmp, sel, sizeof(uint32_t) * (size_t)ns);
    g_plen = (lv < depth) ? lv + 1 : 0;
    g_gpukey = (lv != ORC_LEVEL_WORKLOAD);
    qsort(tmp, (size_t)ns, sizeof(uint32_t), cmp_group);
    /* group boundaries */
    int64_t ng = 0;
    for (int64_t i = 0; i < ns; ++i)
      if (i == 0 || !same_group(tmp[i - 1], tmp[i])) bstart[ng++] = i;
    bstart[ng] = ns;
    for (int64_t q = 0; q < ng; ++q) {
      uint32_t k0 = tmp[bstart[q]];
      int64_t mn = s[k0];
      uint32_t fst = k0;
      for (int64_t i = bstart[q]; i < bstart[q + 1]; ++i) {
        uint32_t k = tmp[i];
        if (s[k] < mn || (s[k] == mn && k < fst)) { mn = s[k]; fst = k; }
      }
      rk[q].gpu = (lv == ORC_LEVEL_WORKLOAD) ? 0xFFu : gpu[k0];
      rk[q].kind = (uint32_t)kind_of(cls[k0]);
      rk[q].tmin = mn;
      rk[q].first = fst;
      rk[q].src = q;
    }
    qsort(rk, (size_t)ng, sizeof(rowkey_t), cmp_rowkey);
    for (int64_t r = 0; r < ng; ++r) {
      int64_t q = rk[r].src;
      int64_t o = nrows + r;
      uint32_t k0 = tmp[bstart[q]];
      for (int l = 0; l < depth; ++l)
        out->path[(int64_t)l * cap + o] =
            (lv < depth && l <= lv) ? idx[(int64_t)l * n + k0] : ORC_NONE;
      out->gpu[o] = (uint8_t)rk[r].gpu;
      out->kind[o] = (uint8_t)rk[r].kind;
      uint64_t cnt = 0;
      int64_t sd = 0, sg = 0, so = 0, mx = 0;
      int have = 0;
      for (int c = 0; c < n_counters; ++c) out->ctr[(int64_t)c * cap + o] = 0;
      for (int64_t i = bstart[q]; i < bstart[q + 1]; ++i) {
        uint32_t k = tmp[i];
        cnt += 1;
        sd += e[k] - s[k];
        sg += gap[k];
        so += ovl[k];
        if (!have || e[k] > mx) mx = e[k];
        have = 1;
        for (int c = 0; c < n_counters; ++c)
          out->ctr[(int64_t)c * cap + o] += ctr[(int64_t)c * n + k];
      }
      out->n[o] = cnt;
      out->dur[o] = sd;
      out->gap[o] = sg;
      out->ovl[o] = so;
      out->tmin[o] = rk[r].tmin;
      out->tmax[o] = mx;
      out->first[o] = rk[r].first;
    }
    nrows += ng;
    /* later levels start where this one ends */
    for (int z = slot + 1; z < depth + 3; ++z) out->level_offset[z] = nrows;
  }
  out->n_rows = nrows;
  /* compact the path and counter columns from stride cap to stride n_rows */
  for (int l = 1; l < depth; ++l)
    memmove(&out->path[(int64_t)l * nrows], &out->path[(int64_t)l * cap],
            sizeof(uint32_t) * (size_t)nrows);
  for (int c = 1; c < n_counters; ++c)
    memmove(&out->ctr[(int64_t)c * nrows], &out->ctr[(int64_t)c * cap],
            sizeof(uint64_t) * (size_t)nrows);
  free(rk); free(bstart); free(tmp); free(sel);
  return 0;
}

void orc_rows_free(orc_rows* r) {
  free(r->path); free(r->gpu); free(r->kind); free(r->n); free(r->dur);
  free(r->gap); free(r->ovl); free(r->tmin); free(r->tmax); free(r->first);
  free(r->ctr);
  memset(r, 0, sizeof(*r));
}

/* ------------------------------------------------------------------------ */
/* Derived metrics (III-C: derived from counters and durations; eq. 10)      */
/* ------------------------------------------------------------------------ */
/*
 * Per row, each a plain IEEE double division of integer sums:
 *   out[0] overlap ratio            = ovl / dur
 *   out[1] HBM bandwidth, GB/s      = (rd_bytes + wr_bytes) / dur
 *   out[2] mean SCLK, MHz           = sclk_sum / n
 *   out[3] MFMA utilisation         = mfma_busy / gpu_cycles
 *   out[4] duration at peak clock   = gpu_cycles * 1000 / freq_peak_mhz  (ns)
 *   out[5] actual / peak-clock time = dur / out[4]
 * Counter-based entries are NaN when the rows carry no counters.
 */
void orc_ratios(int64_t nr, const uint64_t* n_, const int64_t* dur,
                const int64_t* ovl, const uint64_t* ctr, int32_t n_counters,
                int64_t ctr_stride, double freq_peak_mhz, double* out) {
  for (int64_t r = 0; r < nr; ++r) {
    double d = (double)dur[r];
    out[0 * nr + r] = (double)ovl[r] / d;
    if (n_counters >= 16) {
      uint64_t cyc = ctr[0 * ctr_stride + r];
      uint64_t mfma = ctr[1 * ctr_stride + r];
      uint64_t rw = ctr[4 * ctr_stride + r] + ctr[5 * ctr_stride + r];
      uint64_t sclk = ctr[13 * ctr_stride + r];
      double dpeak = (double)cyc * 1000.0 / freq_peak_mhz;
      out[1 * nr + r] = (double)rw / d;
      out[2 * nr + r] = (double)sclk / (double)n_[r];
      out[3 * nr + r] = (double)mfma / (double)cyc;
      out[4 * nr + r] = dpeak;
      out[5 * nr + r] = d / dpeak;
    } else {
      double nan = __builtin_nan("");
      for (int z = 1; z < 6; ++z) out[z * nr + r] = nan;
    }
  }
}

/* window fractions: CO, MO, OV, ID over the window length */
void orc_window_fractions(int64_t nw, const int64_t* w, double* out) {
  for (int64_t j = 0; j < nw; ++j) {
    int64_t len = w[4 * j] + w[4 * j + 1] + w[4 * j + 2] + w[4 * j + 3];
    for (int z = 0; z < 4; ++z)
      out[4 * j + z] = (double)w[4 * j + z] / (double)len;
  }
}

/* ------------------------------------------------------------------------
 * Re-keyed views and their statistics.
 *
 * Figure "end_to_end": per phase and kernel class, duration = sum of kernel
 * durations and launch overhead = sum of bubbles, median values across
 * iterations and GPUs; throughput from the largest duration plus launch
 * overhead across GPUs.  Section V-B and Figure "operation_time": operation
 * duration summed across layers with the bubbles between its kernels, one
 * data point per iteration and GPU.  Section IV: the first iterations are
 * warm-up and are not sampled.
 *
 * A unit is one marker of level iter_level (one GPU's iteration), numbered
 * in marker input order.  A record belongs to the unit of its level
 * iter_level marker, to the phase labelled by its level phase_level marker
 * and to the operation labelled by its level op_level marker (NONE: none).
 * Tables (sums wrap modulo 2^64 like every other sum here), one series over
 * the units per group:
 *   cls_tab [3][P * 8][U]      n, dur, gap by (phase label, class; unit)
 *   op_tab  [4][P * O * 2][U]  n, dur, gap, ovl by (phase label, operation
 *                              label, kind; unit)
 *   busy    [U]                sum of dur + gap of the unit's compute records
 *   iter_max [NI]              max of busy over the units whose iteration
 *                              label is i, -1 if there is none
 * A record counts in cls_tab when it has a unit and a phase label < P, in
 * op_tab when also its operation label < O; busy needs only the unit.
 * Medians (st = dur, gap, dur + gap): over the units whose iteration label
 * is >= warmup and whose table entry has n > 0, the middle values lo =
 * v[(m - 1) / 2] and hi = v[m / 2] of the m sorted values, median =
 * ((double)lo + (double)hi) / 2 (NaN when m = 0).  iter_med: the same over
 * iter_max[i] >= 0 for warmup <= i < NI.
 * ------------------------------------------------------------------------ */
static int cmp_i64(const void* x, const void* y) {
  const int64_t a = *(const int64_t*)x, b = *(const int64_t*)y;
  return a < b ? -1 : a > b;
}

static double median_of(int64_t* v, int64_t m) {
  if (m == 0) return __builtin_nan("");
  qsort(v, (size_t)m, sizeof(int64_t), cmp_i64);
  return ((double)v[(m - 1) / 2] + (double)v[m / 2]) / 2.0;
}

int orc_views(int64_t n, const uint8_t* cls, const int64_t* s,
              const int64_t* e, const uint32_t* idx, int depth,
              const int64_t* gap, const int64_t* ovl, int64_t nm,
              const uint8_t* m_level, const uint32_t* m_label, int iter_level,
              int phase_level, int op_level, int P, int O, int NI,
              uint32_t warmup, int64_t unit_cap, int64_t* n_units,
              uint32_t* unit_marker, uint64_t* cls_tab, uint64_t* op_tab,
              int64_t* busy, int64_t* iter_max, double* cls_med,
              int64_t* cls_cnt, double* op_med, int64_t* op_cnt,
              double* iter_med, int64_t* iter_cnt) {
  /* units: the iteration markers in input order */
  int64_t U = 0;
  uint32_t* unit_of = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(nm + 1));
  for (int64_t m = 0; m < nm; ++m) {
    unit_of[m] = ORC_NONE;
    if (m_level[m] == (uint8_t)iter_level) {
      if (U < unit_cap) unit_marker[U] = (uint32_t)m;
      unit_of[m] = (uint32_t)U;
      ++U;
    }
  }
  *n_units = U;
  if (U > unit_cap) {
    free(unit_of);
    return -1;
  }
  const int64_t nc = U * P * 8, no = U * P * O * 2;
  memset(cls_tab, 0, sizeof(uint64_t) * (size_t)(3 * nc));
  memset(op_tab, 0, sizeof(uint64_t) * (size_t)(4 * no));
  for (int64_t u = 0; u < U; ++u) busy[u] = 0;
  /* one pass over the records */
  for (int64_t r = 0; r < n; ++r) {
    const uint32_t mi = idx[(int64_t)iter_level * n + r];
    if (mi == ORC_NONE) continue;
    const int64_t u = unit_of[mi];
    const int64_t dur = e[r] - s[r];
    const int kd = kind_of(cls[r]);
    if (kd == 0)
      busy[u] = (int64_t)((uint64_t)busy[u] + (uint64_t)dur + (uint64_t)gap[r]);
    const uint32_t mp = idx[(int64_t)phase_level * n + r];
    if (mp == ORC_NONE || m_label[mp] >= (uint32_t)P) continue;
    const int64_t p = m_label[mp];
    if (cls[r] < 8) {
      const int64_t k = (p * 8 + cls[r]) * U + u;
      cls_tab[k] += 1;
      cls_tab[nc + k] += (uint64_t)dur;
      cls_tab[2 * nc + k] += (uint64_t)gap[r];
    }
    const uint32_t mo = idx[(int64_t)op_level * n + r];
    if (mo == ORC_NONE || m_label[mo] >= (uint32_t)O) continue;
    const int64_t k = ((p * O + m_label[mo]) * 2 + kd) * U + u;
    op_tab[k] += 1;
    op_tab[no + k] += (uint64_t)dur;
    op_tab[2 * no + k] += (uint64_t)gap[r];
    op_tab[3 * no + k] += (uint64_t)ovl[r];
  }
  for (int i = 0; i < NI; ++i) iter_max[i] = -1;
  for (int64_t u = 0; u < U; ++u) {
    const uint32_t lab = m_label[unit_marker[u]];
    if (lab < (uint32_t)NI && busy[u] > iter_max[lab]) iter_max[lab] = busy[u];
  }
  /* medians over the kept units */
  int64_t* v = (int64_t*)malloc(sizeof(int64_t) * (size_t)(U + NI + 1));
  for (int g = 0; g < P * 8; ++g) {
    for (int st = 0; st < 3; ++st) {
      int64_t m = 0;
      for (int64_t u = 0; u < U; ++u) {
        const int64_t k = g * U + u;
        if (m_label[unit_marker[u]] < warmup || cls_tab[k] == 0) continue;
        const uint64_t d = cls_tab[nc + k], b = cls_tab[2 * nc + k];
        v[m++] = (int64_t)(st == 0 ? d : st == 1 ? b : d + b);
      }
      cls_cnt[g] = m;
      cls_med[(int64_t)st * P * 8 + g] = median_of(v, m);
    }
  }
  for (int64_t g = 0; g < (int64_t)P * O * 2; ++g) {
    for (int st = 0; st < 3; ++st) {
      int64_t m = 0;
      for (int64_t u = 0; u < U; ++u) {
        const int64_t k = g * U + u;
        if (m_label[unit_marker[u]] < warmup || op_tab[k] == 0) continue;
        const uint64_t d = op_tab[no + k], b = op_tab[2 * no + k];
        v[m++] = (int64_t)(st == 0 ? d : st == 1 ? b : d + b);
      }
      op_cnt[g] = m;
      op_med[(int64_t)st * P * O * 2 + g] = median_of(v, m);
    }
  }
  int64_t m = 0;
  for (int i = (int)warmup; i < NI; ++i)
    if (i >= 0 && iter_max[i] >= 0) v[m++] = iter_max[i];
  *iter_cnt = m;
  *iter_med = median_of(v, m);
  free(v);
  free(unit_of);
  return 0;
}

/* ------------------------------------------------------------------------
 * Launch overhead split (Section V-D eqs. 1-3).  For a compute record i with
 * previous compute record p of the same (gpu, stream) in (start', index)
 * order, with dispatch time tl (aligned):
 *   O_prep = max(tl - e_p, 0), O_call = min(s_i - tl, s_i - e_p),
 *   O_launch = O_prep + O_call.
 * Reading: when the bubble s_i - e_p is not positive (abutting or
 * overlapping kernels), for the first compute record of a stream and for
 * communication records both parts are 0; otherwise O_prep is capped at the
 * bubble and O_call is the rest, which are the equations' values whenever
 * tl <= s_i.
 * ------------------------------------------------------------------------ */
void orc_launch_split(int64_t n, const uint8_t* gpu, const uint8_t* stream,
                      const uint8_t* cls, const int64_t* s, const int64_t* e,
                      const int64_t* tl, int64_t* prep, int64_t* call) {
  uint32_t* ord = (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(n > 0 ? n : 1));
  orc_order(n, gpu, stream, cls, s, 0, ord);
  int have = 0;
  uint32_t cur_g = 0, cur_st = 0;
  int64_t last_e = 0;
  for (int64_t q = 0; q < n; ++q) {
    const uint32_t i = ord[q];
    if (q == 0 || gpu[i] != cur_g || stream[i] != cur_st) {
      cur_g = gpu[i];
      cur_st = stream[i];
      have = 0;
    }
    prep[i] = 0;
    call[i] = 0;
    if (kind_of(cls[i])) continue;
    if (have) {
      const int64_t ep = last_e;
      const int64_t bubble = s[i] - ep;
      if (bubble > 0) {
        int64_t p = tl[i] - ep;                 /* eq. 1 */
        if (p < 0) p = 0;
        int64_t c = s[i] - tl[i];               /* eq. 2 */
        if (s[i] - ep < c) c = s[i] - ep;
        /* a dispatch after the start (tl > s_i): the whole bubble is
           preparation */
        if (p > bubble) {
          p = bubble;
          c = 0;
        }
        prep[i] = p;
        call[i] = c;
      }
    }
    have = 1;
    last_e = e[i];
  }
  free(ord);
}

/* ------------------------------------------------------------------------
 * Counter-pass join (Section III-A hardware profiling: counters come from
 * serialized passes of two or three counters each, without valid
 * timestamps; Section III-B: alignment attaches them to the runtime trace's
 * kernels).
 *
 * A runtime record's key is (gpu, stream, iteration label, ordinal), the
 * ordinal being the number of records with the same (gpu, stream, label)
 * and a smaller (start', index); a pass entry's key is (gpu, stream, label,
 * ordinal), the ordinal counting earlier entries of the pass with the same
 * (gpu, stream, label).  Record and entry match when the keys are equal and
 * their classes agree; then each of the pass's value columns goes to its
 * destination counter column of the record and bit p of matched is set.
 * Columns no matched entry fills are 0.  Records and entries without an
 * iteration (label NONE) are never matched.  JOIN_MISS: some record with an
 * iteration found no matching entry in some pass.  JOIN_ORDER (a warning:
 * the join above is defined for any label order): along (gpu, stream) in
 * (start', index) order, or along a pass's own order, an iteration label is
 * smaller than an earlier one (NONE labels aside) -- iterations are
 * annotated in time order (III-A), so the trace or the pass is out of order.
 * ------------------------------------------------------------------------ */
#define ORC_JOIN_MISS 256u
#define ORC_JOIN_ORDER 512u

typedef struct {
  uint32_t g, st, lab;
  int64_t t;      /* start' (records) or position (entries) */
  uint32_t k;     /* index */
  uint32_t ord;
} jrow_t;

static int cmp_jrow_time(const void* x, const void* y) {
  const jrow_t* a = (const jrow_t*)x;
  const jrow_t* b = (const jrow_t*)y;
  if (a->g != b->g) return a->g < b->g ? -1 : 1;
  if (a->st != b->st) return a->st < b->st ? -1 : 1;
  if (a->t != b->t) return a->t < b->t ? -1 : 1;
  return a->k < b->k ? -1 : a->k > b->k;
}

static int cmp_jrow_key(const void* x, const void* y) {
  const jrow_t* a = (const jrow_t*)x;
  const jrow_t* b = (const jrow_t*)y;
  if (a->g != b->g) return a->g < b->g ? -1 : 1;
  if (a->st != b->st) return a->st < b->st ? -1 : 1;
  if (a->lab != b->lab) return a->lab < b->lab ? -1 : 1;
  if (a->ord != b->ord) return a->ord < b->ord ? -1 : 1;
  return a->k < b->k ? -1 : a->k > b->k;
}

/* ordinals: sort by (g, st, t, k), check the labels, then count within
   each (g, st, lab) */
static uint32_t join_ordinals(jrow_t* v, int64_t n) {
  uint32_t st = 0;
  qsort(v, (size_t)n, sizeof(jrow_t), cmp_jrow_time);
  {
    /* along each (g, st): a label below the last label seen */
    uint32_t last = ORC_NONE;   /* last label with an iteration */
    for (int64_t i = 0; i < n; ++i) {
      if (i == 0 || v[i].g != v[i - 1].g || v[i].st != v[i - 1].st)
        last = ORC_NONE;
      if (v[i].lab == ORC_NONE) continue;
      if (last != ORC_NONE && v[i].lab < last) st |= ORC_JOIN_ORDER;
      last = v[i].lab;
    }
  }
  /* counts per (g, st, lab) in time order, whatever the label order */
  for (int64_t i = 0; i < n; ++i) v[i].ord = 0;
  {
    /* group equal (g, st, lab) keeping time order: a stable pass over a
       copy sorted by (g, st, lab, t, k) */
    jrow_t* w = (jrow_t*)malloc(sizeof(jrow_t) * (size_t)(n > 0 ? n : 1));
    memcpy(w, v, sizeof(jrow_t) * (size_t)n);
    for (int64_t i = 0; i < n; ++i) w[i].ord = (uint32_t)i; /* time rank */
    qsort(w, (size_t)n, sizeof(jrow_t), cmp_jrow_key);
    /* cmp_jrow_key orders by ord = time rank inside equal (g, st, lab) */
    uint32_t c = 0;
    for (int64_t i = 0; i < n; ++i) {
      if (i > 0 && (w[i].g != w[i - 1].g || w[i].st != w[i - 1].st ||
                    w[i].lab != w[i - 1].lab))
        c = 0;
      v[w[i].ord].ord = c++;
    }
    free(w);
  }
  return st;
}

uint32_t orc_join(int64_t n, const uint8_t* gpu, const uint8_t* stream,
                  const uint8_t* cls, const int64_t* s, const uint32_t* lab,
                  int32_t n_passes, const int64_t* pn, const int32_t* pcols,
                  const int32_t* pdst, const uint8_t* const* pgpu,
                  const uint8_t* const* pstream, const uint8_t* const* pcls,
                  const uint32_t* const* plab,
                  const uint64_t* const* pval, uint64_t* counters,
                  uint8_t* matched) {
  uint32_t status = 0;
  memset(counters, 0, sizeof(uint64_t) * 16 * (size_t)n);
  memset(matched, 0, (size_t)n);
  jrow_t* R = (jrow_t*)malloc(sizeof(jrow_t) * (size_t)(n > 0 ? n : 1));
  for (int64_t i = 0; i < n; ++i)
    R[i] = (jrow_t){gpu[i], stream[i], lab[i], s[i], (uint32_t)i, 0};
  status |= join_ordinals(R, n);
  qsort(R, (size_t)n, sizeof(jrow_t), cmp_jrow_key);
  for (int p = 0; p < n_passes; ++p) {
    const int64_t m = pn[p];
    jrow_t* Q = (jrow_t*)malloc(sizeof(jrow_t) * (size_t)(m > 0 ? m : 1));
    for (int64_t i = 0; i < m; ++i)
      Q[i] = (jrow_t){pgpu[p][i], pstream[p][i], plab[p][i], i, (uint32_t)i,
                      0};
    status |= join_ordinals(Q, m);
    qsort(Q, (size_t)m, sizeof(jrow_t), cmp_jrow_key);
    /* merge the two key-sorted lists */
    int64_t j = 0;
    for (int64_t i = 0; i < n; ++i) {
      const jrow_t* a = &R[i];
      if (a->lab == ORC_NONE) continue;
      while (j < m) {
        const jrow_t* b = &Q[j];
        if (b->g != a->g ? b->g < a->g
            : b->st != a->st ? b->st < a->st
            : b->lab != a->lab ? b->lab < a->lab : b->ord < a->ord)
          ++j;
        else
          break;
      }
      int hit = 0;
      if (j < m && Q[j].g == a->g && Q[j].st == a->st && Q[j].lab == a->lab &&
          Q[j].ord == a->ord && pcls[p][Q[j].k] == cls[a->k]) {
        hit = 1;
        for (int c = 0; c < pcols[p]; ++c)
          counters[(int64_t)pdst[16 * p + c] * n + a->k] =
              pval[p][(int64_t)c * m + Q[j].k];
        matched[a->k] |= (uint8_t)(1u << p);
      }
      if (!hit) status |= ORC_JOIN_MISS;
    }
    free(Q);
  }
  free(R);
  return status;
}

/* ------------------------------------------------------------------------
 * Overlap statistics and overhead breakdown of operations (Fig.
 * gemm_overlap: overlap ratio against duration of operations, their
 * correlation, 25-75 % and min-max fills of the overlap ratio; Section VI
 * duration breakdown, eqs. 6-10).
 *
 * Instances: compute rows (kind 0) of the operation level with dur > 0 --
 * one operation of one layer in one GPU's iteration -- grouped by
 * g = p * O + o, p and o the labels of the row's phase- and operation-level
 * markers (p < P, o < O).  Per instance
 *   x = floor(ovl * 2^30 / dur)    overlap ratio in Q30 (ovl <= dur)
 *   y = dur + gap                   operation duration with its bubbles (V-B)
 * Per group with m instances, from exact sums Sx, Sy, Sxx, Syy, Sxy:
 *   cov = m Sxy - Sx Sy, vx = m Sxx - Sx^2, vy = m Syy - Sy^2 (exact),
 *   pearson = (double)cov / sqrt((double)vx * (double)vy)   (NaN if m < 2 or
 *             a variance is 0: constant overlap gives NaN),
 *   slope = (double)cov / (double)vx (per Q30 unit), intercept
 *   a = ((double)Sy - slope (double)Sx) / m: the least-squares line of
 *   duration on overlap; D0 = a, D50 = a + slope 2^29 (duration at 0 % and
 *   50 % overlap), Ovr_overlap = D50 / D0 (eq. 9);
 *   quantiles of x / 2^30: v[0], v[(m-1)/4], (v[(m-1)/2] + v[m/2]) / 2,
 *   v[3(m-1)/4], v[m-1] of the sorted values;
 *   D_act = Sy / m, D_peak = (sum of ctr[0]) * 1000 / freq_peak / m (ns,
 *   eq. 10), MFMA_util = sum ctr[1] / sum ctr[0], Ovr_util = 1 / MFMA_util
 *   (eq. 8), F_perf = sum ctr[11] / m, Ovr_inst = F_perf / F_gemm[o]
 *   (eq. 7), D_thr = F_gemm[o] / TPT_peak (eq. 6), Ovr_freq = D_act /
 *   D_peak / Ovr_overlap (eq. 10); F_gemm[o] is given per operation label
 *   (NaN: not given).  Counter sums wrap modulo 2^64; with fewer than 16
 *   counters the counter-based values are NaN.
 * out [17][P * O]: pearson, slope, intercept, D0, D50, q0, q25, q50, q75,
 * q100, D_act, D_peak, Ovr_util, Ovr_inst, Ovr_overlap, Ovr_freq, D_thr;
 * cnt [P * O] = m.  Limits: y < 2^34, m < 2^26 per group.
 *
 * Per-GPU overlap CDF (Fig. per_gpu_overlap_variation: per GPU, the CDF of
 * an operation's overlap ratio against its duration normalised to that
 * GPU's minimum; Section VI "Overlap overhead": D_50% and D_0% are read off
 * such a CDF, eq. 9).  The instances of (p, o) on GPU h (row gpu h < NG) in
 * CDF order: ascending x, equal x in row order (rows of a GPU are in time
 * order).  With v_k the k-th instance in that order (k = 0 .. m_h - 1) and
 * y_min the smallest y of the group:
 *   q0, q25, q50, q75, q100 of x / 2^30 as above;
 *   D_0%  = y(v_0) / y_min                 (the CDF at 0),
 *   D_50% = (y(v_(m-1)/2) / y_min + y(v_m/2) / y_min) / 2  (the CDF at 1/2),
 *   Ovr_h = D_50% / D_0%.
 * gout [9][P * O * NG] at g * NG + h: q0, q25, q50, q75, q100, y_min, D_0%,
 * D_50%, Ovr_h (NaN when m_h = 0); gcnt = m_h.  The operation's
 * Ovr_overlap (out 14, eq. 9) is the median over the GPUs with m_h > 0 of
 * Ovr_h (sorted, (v[(k-1)/2] + v[k/2]) / 2), and Ovr_freq (out 15, eq. 10)
 * divides by it.  D0 and D50 (out 3, 4) stay the least-squares line's
 * values at 0 and 50 % overlap.
 * ------------------------------------------------------------------------ */
typedef unsigned __int128 u128;

typedef struct { uint32_t x; int64_t r, y; } cdf_item;

static int cmp_cdf(const void* a_, const void* b_) {
  const cdf_item* a = (const cdf_item*)a_;
  const cdf_item* b = (const cdf_item*)b_;
  if (a->x != b->x) return a->x < b->x ? -1 : 1;
  return a->r < b->r ? -1 : a->r > b->r;
}

static int cmp_f64(const void* a_, const void* b_) {
  const double a = *(const double*)a_, b = *(const double*)b_;
  return a < b ? -1 : a > b;
}

static int cmp_u32(const void* x, const void* y) {
  const uint32_t a = *(const uint32_t*)x, b = *(const uint32_t*)y;
  return a < b ? -1 : a > b;
}

void orc_op_stats(int64_t lo, int64_t hi, int64_t cap, const uint32_t* path,
                  int phase_level, int op_level, const uint8_t* kind,
                  const int64_t* dur, const int64_t* gap, const int64_t* ovl,
                  const uint64_t* ctr, int nc, const uint32_t* m_label,
                  int P, int O, double freq_peak, double tpt_peak,
                  const double* f_gemm, double* out, int64_t* cnt,
                  const uint8_t* rgpu, int NG, double* gout,
                  int64_t* gcnt) {
  const int G = P * O;
  const double nan = __builtin_nan("");
  /* the group of every row (-1: not an instance), then each group's rows */
  const int64_t nr = hi > lo ? hi - lo : 0;
  int32_t* grp = (int32_t*)malloc(sizeof(int32_t) * (size_t)(nr + 1));
  int64_t* start = (int64_t*)calloc((size_t)G + 1, sizeof(int64_t));
  for (int64_t r = lo; r < hi; ++r) {
    int32_t gg = -1;
    if (kind[r] == 0 && dur[r] > 0) {
      const uint32_t mp = path[(int64_t)phase_level * cap + r];
      const uint32_t mo = path[(int64_t)op_level * cap + r];
      if (mp != ORC_NONE && mo != ORC_NONE) {
        const uint32_t p = m_label[mp], o = m_label[mo];
        if (p < (uint32_t)P && o < (uint32_t)O) gg = (int32_t)(p * O + o);
      }
    }
    grp[r - lo] = gg;
    if (gg >= 0) start[gg + 1]++;
  }
  for (int g = 0; g < G; ++g) start[g + 1] += start[g];
  int64_t* rows = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nr + 1));
  int64_t* fillp = (int64_t*)malloc(sizeof(int64_t) * (size_t)(G + 1));
  memcpy(fillp, start, sizeof(int64_t) * (size_t)(G + 1));
  for (int64_t r = lo; r < hi; ++r)
    if (grp[r - lo] >= 0) rows[fillp[grp[r - lo]]++] = r;
  for (int g = 0; g < G; ++g) {
    int64_t m = 0;
    i128 sx = 0, sy = 0, sxx = 0, syy = 0, sxy = 0;
    uint64_t cyc = 0, busy = 0, flops = 0;
    uint32_t* xs =
        (uint32_t*)malloc(sizeof(uint32_t) * (size_t)(start[g + 1] - start[g] + 1));
    for (int64_t q = start[g]; q < start[g + 1]; ++q) {
      const int64_t r = rows[q];
      const i128 x = ((i128)ovl[r] << 30) / dur[r];
      const i128 y = (i128)dur[r] + gap[r];
      xs[m++] = (uint32_t)x;
      sx += x;
      sy += y;
      sxx += x * x;
      syy += y * y;
      sxy += x * y;
      if (nc >= 16) {
        cyc += ctr[0 * cap + r];
        busy += ctr[1 * cap + r];
        flops += ctr[11 * cap + r];
      }
    }
    cnt[g] = m;
    double* o_ = out;
    for (int k = 0; k < 17; ++k) o_[(int64_t)k * G + g] = nan;
    for (int h = 0; h < NG; ++h) {
      gcnt[(int64_t)g * NG + h] = 0;
      for (int z = 0; z < 9; ++z)
        gout[(int64_t)z * G * NG + (int64_t)g * NG + h] = nan;
    }
    if (m > 0) {
      const i128 cov = (i128)m * sxy - sx * sy;
      const i128 vx = (i128)m * sxx - sx * sx;
      const i128 vy = (i128)m * syy - sy * sy;
      const double dm = (double)m;
      if (m >= 2 && vx != 0 && vy != 0)
        o_[0 * G + g] = (double)cov / sqrt((double)vx * (double)vy);
      double slope = nan, a = nan;
      if (vx != 0) {
        slope = (double)cov / (double)vx;
        a = ((double)sy - slope * (double)sx) / dm;
      }
      o_[1 * G + g] = slope;
      o_[2 * G + g] = a;
      const double d0 = a, d50 = a + slope * 536870912.0;
      o_[3 * G + g] = d0;
      o_[4 * G + g] = d50;
      qsort(xs, (size_t)m, sizeof(uint32_t), cmp_u32);
      const double q = 1.0 / 1073741824.0;
      o_[5 * G + g] = (double)xs[0] * q;
      o_[6 * G + g] = (double)xs[(m - 1) / 4] * q;
      o_[7 * G + g] = ((double)xs[(m - 1) / 2] + (double)xs[m / 2]) / 2.0 * q;
      o_[8 * G + g] = (double)xs[3 * (m - 1) / 4] * q;
      o_[9 * G + g] = (double)xs[m - 1] * q;
      const double dact = (double)sy / dm;
      o_[10 * G + g] = dact;
      /* per-GPU CDFs of the group, and eq. 9 as their median over GPUs */
      cdf_item* it = (cdf_item*)malloc(sizeof(cdf_item) * (size_t)m);
      double* ovr_h = (double*)malloc(sizeof(double) * (size_t)(NG > 0 ? NG : 1));
      int k_h = 0;
      for (int h = 0; h < NG; ++h) {
        const int64_t gi = (int64_t)g * NG + h;
        int64_t mh = 0;
        for (int64_t q2 = start[g]; q2 < start[g + 1]; ++q2) {
          const int64_t r = rows[q2];
          if (rgpu[r] != h) continue;
          it[mh].x = (uint32_t)(((i128)ovl[r] << 30) / dur[r]);
          it[mh].r = r;
          it[mh].y = dur[r] + gap[r];
          ++mh;
        }
        gcnt[gi] = mh;
        for (int z = 0; z < 9; ++z) gout[(int64_t)z * G * NG + gi] = nan;
        if (mh == 0) continue;
        qsort(it, (size_t)mh, sizeof(cdf_item), cmp_cdf);
        int64_t ymin = it[0].y;
        for (int64_t k = 1; k < mh; ++k)
          if (it[k].y < ymin) ymin = it[k].y;
        const double qq = 1.0 / 1073741824.0, dy = (double)ymin;
        double* go = gout + gi;
        const int64_t GN = (int64_t)G * NG;
        go[0 * GN] = (double)it[0].x * qq;
        go[1 * GN] = (double)it[(mh - 1) / 4].x * qq;
        go[2 * GN] = ((double)it[(mh - 1) / 2].x + (double)it[mh / 2].x) /
                     2.0 * qq;
        go[3 * GN] = (double)it[3 * (mh - 1) / 4].x * qq;
        go[4 * GN] = (double)it[mh - 1].x * qq;
        go[5 * GN] = dy;
        const double c0 = (double)it[0].y / dy;
        const double c50 = ((double)it[(mh - 1) / 2].y / dy +
                            (double)it[mh / 2].y / dy) / 2.0;
        go[6 * GN] = c0;
        go[7 * GN] = c50;
        go[8 * GN] = c50 / c0;
        ovr_h[k_h++] = c50 / c0;
      }
      double ovr_ov = nan;
      if (k_h > 0) {
        qsort(ovr_h, (size_t)k_h, sizeof(double), cmp_f64);
        ovr_ov = (ovr_h[(k_h - 1) / 2] + ovr_h[k_h / 2]) / 2.0;
      }
      free(it);
      free(ovr_h);
      o_[14 * G + g] = ovr_ov;
      if (nc >= 16) {
        const double dpeak = (double)cyc * 1000.0 / freq_peak / dm;
        o_[11 * G + g] = dpeak;
        o_[12 * G + g] = 1.0 / ((double)busy / (double)cyc);
        const double fg = f_gemm ? f_gemm[g % O] : nan;
        o_[13 * G + g] = ((double)flops / dm) / fg;
        o_[15 * G + g] = dact / dpeak / ovr_ov;
      }
      o_[16 * G + g] = (f_gemm ? f_gemm[g % O] : nan) / tpt_peak;
    }
    free(xs);
  }
  free(grp);
  free(start);
  free(rows);
  free(fillp);
}
