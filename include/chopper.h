/*
 * chopper.h -- C ABI of libchopper, the GPU trace pipeline for MI355X (gfx950).
 *
 * The library turns per-kernel records of a multi-GPU training run into the
 * multi-granularity view described in the paper (Chopper, arXiv 2512.08242):
 *
 *   chopper_align      puts every record and annotation marker on one clock
 *                      and sorts the records      (Section III-B, alignment)
 *   chopper_attribute  assigns each kernel to its iteration / phase / layer /
 *                      operation marker           (Section I granularities,
 *                                                  III-A annotations)
 *   chopper_overlap    splits wall time into compute-only, comm-only,
 *                      overlapped and idle; per-kernel overlapped time and
 *                      launch bubbles              (Section V-C; V-D eqs. 1-3;
 *                                                  caption of Fig. end_to_end)
 *   chopper_aggregate  sums durations, bubbles, overlap and counters at every
 *                      granularity, optionally filtered by GPU / class /
 *                      iteration                  (Section III-C)
 *   chopper_ratios     derived metrics per aggregated row (III-C; eq. 10)
 *   chopper_join_counters  counters of serialized profiling passes matched
 *                      to the runtime kernels (III-A, III-B)
 *   chopper_launch_split  preparation / call split of the launch overhead
 *                      from dispatch times (V-D eqs. 1-3)
 *   chopper_op_stats   overlap statistics and overhead breakdown per
 *                      operation (Fig. gemm_overlap; VI eqs. 6-10)
 *   chopper_views      per-phase/class and per-operation views with medians
 *                      over iterations and GPUs, iteration throughput
 *                      (Fig. end_to_end, Fig. operation_time)
 *
 * Memory.  Every pointer is a DEVICE pointer unless marked [host].  The caller
 * owns every buffer.  The library allocates no device memory, frees nothing
 * and keeps no data between calls; all temporary storage comes from the
 * caller's `scratch` (chopper_launch_split_noalloc alone uses a static 6 KiB
 * device table of the library instead).  One exception, on the host: for
 * its read-backs (below) the library keeps, per device, four 256-byte slots
 * of pinned host memory (hipHostMalloc) with one HIP event each, created on
 * first use and held until the process ends; a read-back finds its value
 * there and copies it out, and no slot holds anything between calls.  When
 * the pinned memory cannot be had, the read-backs copy into the call's own
 * variables instead.  Scratch protocol (every call taking scratch): pass
 * scratch == NULL to receive the required size in *scratch_bytes (nothing
 * else is read or written, no GPU work is done, CHOPPER_OK is returned); then
 * call again with a buffer of at least that many bytes, 256-byte aligned.
 *
 * Streams.  `stream` is a hipStream_t.  Work is enqueued on it.  Some calls
 * read back a few words (counts and flags that size or choose later
 * launches): a one-wave kernel stores them into a pinned slot, and the host
 * waits for an event recorded after it, not for the whole stream, while
 * work that does not depend on them is already queued behind it:
 * chopper_align once (record classes and whether the input is in start
 * order; the markers' clock transform runs meanwhile), chopper_attribute
 * once (whether the markers are in start order; their class partition runs
 * meanwhile), chopper_aggregate once when the records come grouped by GPU
 * in start order (row counts per level, whether groups are runs; the
 * records reduction runs meanwhile and exits on the device if the flags
 * rule it out), twice otherwise and twice more on the general path,
 * chopper_join_counters twice; the sorts wait again when their input is not
 * in time order.  chopper_overlap, the derived metrics, the launch split
 * and the statistics never wait.  So do not capture the waiting calls in a
 * HIP graph.  Outputs are valid after the stream has been synchronized.
 * Concurrent calls must use distinct scratch buffers.  Calls on different
 * streams are ordered by the caller's events; chopper_aggregate also takes
 * one (ready) for inputs computed on another stream.
 *
 * Errors.  Argument errors are detected on the host before any GPU work and
 * returned synchronously (negative codes below).  Problems in the DATA are
 * reported as bits OR-ed into the device word *status (the caller clears it);
 * when one of the "error" bits is set the affected outputs are unspecified
 * but every kernel stays within its buffers.
 *
 * Conventions.  Times are int64 nanoseconds; intervals are half-open
 * [start, end).  NONE = 0xFFFFFFFF.  Record classes: 0 GEMM, 1 attention,
 * 2 elementwise, 3 RMSNorm, 4 RoPE, 5 all_gather, 6 reduce_scatter,
 * 7 optimizer; kind = 1 (communication) iff class is 5 or 6, else 0
 * (compute) -- communication is decided by class, not by stream (V-D).
 * Arrays are structure-of-arrays; multi-column outputs are column-major
 * ([column][row]).
 */
#ifndef CHOPPER_H
#define CHOPPER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define CHOPPER_NONE 0xFFFFFFFFu

/* return codes */
enum {
  CHOPPER_OK = 0,
  CHOPPER_EINVAL = -1,     /* null pointer, negative size, bad depth/level */
  CHOPPER_ESCRATCH = -2,   /* scratch smaller than the size reported       */
  CHOPPER_EOVERFLOW = -3,  /* clock fit outside its exact-arithmetic range */
  CHOPPER_EHIP = -4        /* a HIP runtime call failed                    */
};

/* *status bits */
enum {
  CHOPPER_ST_BAD_GPU = 1u,         /* gpu >= n_gpus (record or marker)      */
  CHOPPER_ST_BAD_CLASS = 2u,       /* record class >= 8                     */
  CHOPPER_ST_NEG_DURATION = 4u,    /* end < start (record or marker)        */
  CHOPPER_ST_MARKER_OVERLAP = 8u,  /* two non-empty markers of one (gpu,
                                      level) overlap: warning only, the
                                      attribution is still exactly defined  */
  CHOPPER_ST_RANGE = 16u,          /* |t| >= 2^62 before or after alignment,
                                      or a time span too wide for the keys  */
  CHOPPER_ST_ROWS_OVERFLOW = 32u,  /* aggregate rows exceed rows->cap; the
                                      level offsets hold the needed counts  */
  CHOPPER_ST_BAD_LEVEL = 64u,      /* marker level >= depth                 */
  CHOPPER_ST_PATH_CONFLICT = 128u, /* records sharing a deepest marker have
                                      different marker paths (markers not
                                      nested): warning only, rows are still
                                      grouped by the whole path            */
  CHOPPER_ST_JOIN_MISS = 256u,     /* a record with an iteration found no
                                      entry of some counter pass           */
  CHOPPER_ST_JOIN_ORDER = 512u     /* an iteration label below an earlier
                                      one along a (gpu, stream): warning
                                      only, the join is exactly defined    */
};

/* aggregation levels besides the marker levels 0 .. depth-1 */
enum {
  CHOPPER_LEVEL_GPU = 100,
  CHOPPER_LEVEL_WORKLOAD = 101,
  CHOPPER_LEVEL_ALL = 255
};

/* Kernel records of all GPUs of a run (runtime + hardware profiling,
   Section III-A).  gpu < n_gpus <= 256.  counters: n_counters (0..16)
   columns of n values each, column-major, or NULL when n_counters == 0.
   op_id is carried for the caller and not read by the library. */
typedef struct {
  int64_t n;
  int32_t n_gpus;
  int32_t n_counters;
  const uint8_t* gpu;
  const uint8_t* stream;
  const uint8_t* cls;
  const uint32_t* op_id;
  const int64_t* start_ns;
  const int64_t* end_ns;
  const uint64_t* counters;
} chopper_records;

/* Annotation markers (iteration, phase, layer, operation ... ranges,
   Section III-A), in each GPU's local clock.  level 0 is the outermost;
   depth = number of levels (1..8). */
typedef struct {
  int64_t n;
  int32_t depth;
  int32_t reserved;
  const uint8_t* gpu;
  const uint8_t* level;
  const int64_t* start_ns;
  const int64_t* end_ns;
  const uint32_t* label;
} chopper_markers;

/* [host] Clock anchor pairs: the same instant read on a GPU's local clock
   and on the reference clock. */
typedef struct {
  int64_t n;
  const uint8_t* gpu;
  const int64_t* local_ns;
  const int64_t* ref_ns;
} chopper_anchors;

/* [host] Per-GPU clock: t_ref = t + c + floor((t - x0) * d_q48 / 2^48). */
typedef struct {
  int64_t x0;
  int64_t c;
  int64_t d_q48;
} chopper_clock;

/* [host] Selection before grouping (III-C): a record is kept iff bit gpu of
   gpu_mask, bit cls of class_mask and, when use_iter != 0, its level-0
   marker exists and iter_lo <= label <= iter_hi. */
typedef struct {
  uint64_t gpu_mask[4];
  uint32_t class_mask;
  uint32_t use_iter;
  uint32_t iter_lo;
  uint32_t iter_hi;
} chopper_filter;

/* Aggregated rows (device arrays of capacity cap).  level_offset has
   depth + 3 entries: first row of marker levels 0..depth-1, of the GPU level,
   of the workload level, and the total.  path has depth columns; entries
   deeper than the row's level, and all entries of GPU / workload rows, are
   NONE.  ctr has n_counters columns (may be NULL when n_counters == 0). */
typedef struct {
  int64_t cap;
  int64_t* level_offset;
  uint32_t* path;
  uint8_t* gpu;
  uint8_t* kind;
  uint64_t* n;
  int64_t* dur;
  int64_t* gap;
  int64_t* ovl;
  int64_t* tmin;
  int64_t* tmax;
  uint32_t* first;
  uint64_t* ctr;
} chopper_rows;

/*
 * chopper_align -- clock alignment and the two record orders
 * (Section III-B: traces are aligned so that counters attach to operations,
 * layers and iterations).
 *
 * Fit (host): for each GPU g, its anchors (x = local, y = ref) sorted by
 * (x, y); x0 = first x; u = x - x0, w = y - x; exact least squares of w on u
 * with the slope rounded half-to-even to Q48 (d_q48) and the intercept c
 * rounded half-to-even given d_q48.  No anchors: identity; one anchor or all
 * x equal: d_q48 = 0.  Limits: <= 2^20 anchors per GPU, u < 2^42,
 * |w| < 2^40, |d_q48| < 2^38, else CHOPPER_EOVERFLOW.
 * Transform (GPU): every record start/end and marker start/end of GPU g:
 * t' = t + c + floor((t - x0) * d_q48 / 2^48), exact 64x64->128-bit product.
 *
 * Outputs: clocks_out [host][n_gpus]; start_out/end_out [n] and
 * mstart_out/mend_out [markers->n] aligned times in input order;
 * order_out [n]: permutation sorting records stably by (gpu, stream,
 * start'); korder_out [n]: stable by (gpu, kind, start').  Ties keep input
 * order.  markers may be NULL (no marker outputs); anchors may be NULL
 * (identity clocks).
 */
int chopper_align(const chopper_records* records,
                  const chopper_markers* markers,
                  const chopper_anchors* anchors, chopper_clock* clocks_out,
                  int64_t* start_out, int64_t* end_out, int64_t* mstart_out,
                  int64_t* mend_out, uint32_t* order_out, uint32_t* korder_out,
                  void* scratch, size_t* scratch_bytes, uint32_t* status,
                  void* stream);

/*
 * chopper_attribute -- kernel -> marker per granularity level
 * (Section I: kernel, operation, layer, phase, iteration; III-A annotations).
 *
 * idx_out [depth][n] (column l = level l, input order): the input index of
 * the last non-empty level-l marker of the record's GPU, in (start', input
 * index) order, whose aligned start is <= the record's aligned start, if the
 * record's start is before that marker's end; otherwise NONE.  For markers
 * that do not overlap this is simply the marker containing the kernel start.
 * Zero-length markers contain no instant and are ignored.  start_al,
 * mstart_al, mend_al come from chopper_align.  Sets MARKER_OVERLAP,
 * BAD_GPU, BAD_LEVEL.
 */
int chopper_attribute(const chopper_records* records, const int64_t* start_al,
                      const chopper_markers* markers, const int64_t* mstart_al,
                      const int64_t* mend_al, uint32_t* idx_out,
                      void* scratch, size_t* scratch_bytes, uint32_t* status,
                      void* stream);

/*
 * chopper_overlap -- compute/communication overlap and launch bubbles
 * (Section V-C overlap ratio; V-D eqs. 1-3 and caption of Fig. end_to_end:
 * launch overhead is the bubble before each compute kernel, communication
 * kernels are ignored).
 *
 * Per GPU and instant t, c(t) / m(t) = number of compute / communication
 * kernels with s' <= t < e'.  States: CO (c>0, m=0), MO (c=0, m>0),
 * OV (both), ID (neither).
 *   ovl_out [n]   ns of state OV inside [s', e') of each record;
 *   gap_out [n]   compute record: max(0, s' - e'_prev), prev = previous
 *                 compute record of the same (gpu, stream) in order_out;
 *                 0 for the first one and for communication records;
 *   mwin_out [markers->n][4]  CO, MO, OV, ID ns in each marker window
 *                 [mstart', mend') (row-major 4 per marker; zeros when empty);
 *   gwin_out [n_gpus][6]  start = min s', end = max e' over the GPU's records
 *                 (zeros if none), then CO, MO, OV, ID of that window.
 * order / korder come from chopper_align; markers may be NULL.
 */
int chopper_overlap(const chopper_records* records, const int64_t* start_al,
                    const int64_t* end_al, const uint32_t* order,
                    const uint32_t* korder, const chopper_markers* markers,
                    const int64_t* mstart_al, const int64_t* mend_al,
                    int64_t* ovl_out, int64_t* gap_out, int64_t* mwin_out,
                    int64_t* gwin_out, void* scratch, size_t* scratch_bytes,
                    uint32_t* status, void* stream);

/*
 * chopper_aggregate -- metric aggregation at a granularity (Section III-C;
 * granularities of Section I; duration = sum of kernel durations and launch
 * overhead = sum of bubbles, caption of Fig. end_to_end).
 *
 * Groups of the records kept by `filter` (NULL keeps all):
 *   level l in [0, depth):  (gpu, idx_0 .. idx_l, kind)
 *   CHOPPER_LEVEL_GPU:      (gpu, kind)
 *   CHOPPER_LEVEL_WORKLOAD: (kind), gpu written as 0xFF
 *   CHOPPER_LEVEL_ALL:      all of the above, in that order.
 * Per row: n records, dur = sum(e'-s'), gap = sum(gap), ovl = sum(ovl),
 * tmin = min s', tmax = max e', first = smallest input index among the
 * group's records with s' = tmin, ctr = counters summed modulo 2^64.
 * Rows of a level are ordered by (gpu, kind, tmin, first).
 * idx is chopper_attribute's output (depth columns of n); gap / ovl are
 * chopper_overlap's; korder is chopper_align's.  markers supplies n and the
 * labels read by the iteration filter (may be NULL if depth == 0 paths are
 * all NONE and no iteration filter is used).
 * rows->level_offset is always written.  If the total exceeds rows->cap,
 * ROWS_OVERFLOW is set and the rows are unspecified.  When markers are not
 * nested so that two records with the same deepest marker have different
 * paths, PATH_CONFLICT is set (a warning); the rows are still those of the
 * whole paths (the call then waits for `stream` once more and sorts the
 * records by path, level by level).
 * ready: NULL, or a hipEvent_t that gap and ovl are complete at (recorded by
 * the caller, typically after chopper_overlap on another stream, before this
 * call).  Every pass that reads gap or ovl is queued behind a
 * hipStreamWaitEvent on it; the passes before them (the order check, the
 * head counts, the row offsets and their read-back) are not, so they run
 * while gap and ovl are still being computed.
 */
int chopper_aggregate(const chopper_records* records, const int64_t* start_al,
                      const int64_t* end_al, const uint32_t* korder,
                      const uint32_t* idx, int32_t depth, const int64_t* gap,
                      const int64_t* ovl, const chopper_markers* markers,
                      int32_t level, const chopper_filter* filter,
                      chopper_rows* rows, void* scratch, size_t* scratch_bytes,
                      uint32_t* status, void* ready, void* stream);

/*
 * chopper_ratios -- derived metrics per aggregated row (III-C: metrics derived
 * from counters and duration, e.g. bandwidth; eq. 10 peak-clock duration).
 * out [6][rows->cap] (doubles, column-major), rows 0 .. total-1 where total
 * = rows->level_offset[depth + 2]:
 *   0 overlap ratio           ovl / dur
 *   1 HBM bandwidth (GB/s)    (ctr[4] + ctr[5]) / dur
 *   2 mean SCLK (MHz)         ctr[13] / n
 *   3 MFMA utilisation        ctr[1] / ctr[0]
 *   4 peak-clock duration ns  ctr[0] * 1000 / freq_peak_mhz
 *   5 actual / peak-clock     dur / column 4
 * Each is IEEE double arithmetic on the integer sums converted to double
 * (round to nearest), in exactly this operation order; x/0 follows IEEE.
 * Columns 1-5 are NaN when n_counters < 16.
 */
int chopper_ratios(const chopper_rows* rows, int32_t depth, int32_t n_counters,
                   double freq_peak_mhz, double* out, void* stream);

/*
 * chopper_window_fractions -- CO, MO, OV, ID of n windows (4 int64 each, as
 * written by chopper_overlap) divided by their sum; out [n][4] doubles.
 */
int chopper_window_fractions(int64_t n, const int64_t* win, double* out,
                             void* stream);

/*
 * chopper_views -- re-keyed views of the aggregated run and their statistics
 * (caption of Fig. end_to_end: duration = sum of kernel durations, launch
 * overhead = sum of bubbles, per phase and kernel class, median values
 * across iterations and GPUs, throughput from the largest duration plus
 * launch overhead across GPUs; Section V-B and Fig. operation_time:
 * operation duration summed across layers including the bubbles between its
 * kernels, one data point per iteration and GPU; Section IV: the first
 * iterations are warm-up and not sampled).
 *
 * A unit is one marker of level spec->iter_level (one GPU's iteration),
 * numbered in marker input order; out->unit_marker[u] is its marker index
 * and *out->n_units the number of units.  A record belongs to the unit of
 * its level iter_level marker, to the phase labelled by its level
 * phase_level marker and to the operation labelled by its level op_level
 * marker (no marker: none).  With P = n_phases, O = n_ops, C = unit_cap:
 *   cls_tab [3][P * 8][C]       n, dur, gap summed by (phase label, class;
 *                               unit): entry (p * 8 + class) * C + u
 *   op_tab  [4][P * O * 2][C]   n, dur, gap, ovl summed by (phase label,
 *                               operation label, kind; unit): entry
 *                               ((p * O + o) * 2 + kind) * C + u
 *   busy    [C]                 sum of dur + gap of the unit's compute
 *                               records (whatever their phase)
 *   iter_max [n_iters]          the largest busy among the units whose
 *                               iteration label is i, -1 if none
 * Records without a unit, or with a phase label >= P, are in neither table;
 * op_tab also needs an operation label < O.  Sums wrap modulo 2^64.
 *   cls_med [3][P * 8], op_med [3][P * O * 2]: for dur, gap and dur + gap,
 *   the median over the units whose iteration label is >= warmup and whose
 *   entry has n > 0: with the m values sorted, ((double)v[(m-1)/2] +
 *   (double)v[m/2]) / 2, NaN when m = 0; cls_cnt / op_cnt hold m.
 *   iter_med [1], iter_cnt [1]: the same over iter_max[i] >= 0 for
 *   warmup <= i < n_iters (throughput = tokens per iteration / iter_med).
 * Inputs: start_al / end_al / idx / gap from chopper_align, chopper_attribute
 * and chopper_overlap; rows from chopper_aggregate of the same records
 * without a filter, at level op_level or CHOPPER_LEVEL_ALL (op_tab is the
 * re-keyed level op_level rows).  Levels < depth <= markers->depth;
 * 1 <= n_phases <= 16, 1 <= n_ops <= 128, n_iters >= 0, unit_cap * n_phases
 * < 2^32.  More units than unit_cap: ROWS_OVERFLOW, *n_units holds the
 * count, outputs unspecified.  Every output array is written.
 */
typedef struct {
  int32_t iter_level;
  int32_t phase_level;
  int32_t op_level;
  int32_t n_phases;
  int32_t n_ops;
  int32_t n_iters;
  uint32_t warmup;
  int32_t reserved;
} chopper_view_spec;

typedef struct {
  int64_t unit_cap;
  int64_t* n_units;
  uint32_t* unit_marker;
  uint64_t* cls_tab;
  uint64_t* op_tab;
  int64_t* busy;
  int64_t* iter_max;
  double* cls_med;
  int64_t* cls_cnt;
  double* op_med;
  int64_t* op_cnt;
  double* iter_med;
  int64_t* iter_cnt;
} chopper_view_out;

int chopper_views(const chopper_records* records, const int64_t* start_al,
                  const int64_t* end_al, const uint32_t* idx, int32_t depth,
                  const int64_t* gap, const chopper_markers* markers,
                  const chopper_rows* rows, const chopper_view_spec* spec,
                  const chopper_view_out* out, void* scratch,
                  size_t* scratch_bytes, uint32_t* status, void* stream);

/*
 * chopper_launch_split -- launch overhead split into preparation and call
 * overhead (Section V-D eqs. 1-3) from the kernels' dispatch times.
 *
 * launch_ns [n]: dispatch time t_l of every record on its GPU's local clock
 * (the clock of start_ns / end_ns); it is aligned with clocks (n_gpus
 * entries, [host], chopper_align's clocks_out) exactly like start and end.
 * gap [n] is chopper_overlap's bubble and start_al chopper_align's start'.
 * For a compute record with gap g > 0 the previous compute kernel of its
 * stream ended at e = s' - g, and
 *   prep_out = min(max(t_l' - e, 0), g)      (eq. 1, at most the bubble)
 *   call_out = g - prep_out                   (eq. 2: min(s' - t_l', s' - e))
 * so that prep + call = g (eq. 3) whenever e <= s', as in every trace;
 * records with g = 0 (communication kernels, the first kernel of a stream,
 * abutting or overlapping kernels) get 0 and 0.  Outputs in input order.
 * Per-row sums: pass prep_out / call_out to chopper_aggregate as counter
 * columns.  Sets BAD_GPU, and RANGE when |t_l| or |t_l'| >= 2^62.  Scratch
 * protocol as above (n_gpus clock entries).
 */
int chopper_launch_split(const chopper_records* records,
                         const chopper_clock* clocks,
                         const int64_t* launch_ns, const int64_t* start_al,
                         const int64_t* gap, int64_t* prep_out,
                         int64_t* call_out, void* scratch,
                         size_t* scratch_bytes, uint32_t* status,
                         void* stream);

/*
 * chopper_launch_split_noalloc -- chopper_launch_split for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): same arguments and results, but
 * no scratch argument.  The clock table that chopper_launch_split keeps in
 * the caller's scratch lives here in a static device array of the library
 * (256 entries of 24 bytes, 6 KiB per device, held by every device the
 * library runs on until the process ends).  The call allocates and frees
 * nothing; the device address of the array is looked up once per device, on
 * the first call made on it.  Limits: n_gpus <= 256 (CHOPPER_ESCRATCH
 * otherwise, nothing enqueued); `stream` must belong to the current device
 * (CHOPPER_EHIP otherwise).  The table is rewritten by every call before its
 * kernel reads it, so nothing needs clearing, but calls that overlap on one
 * GPU (different streams, or threads) race on it: serialize them.
 */
int chopper_launch_split_noalloc(const chopper_records* records,
                                 const chopper_clock* clocks,
                                 const int64_t* launch_ns,
                                 const int64_t* start_al, const int64_t* gap,
                                 int64_t* prep_out, int64_t* call_out,
                                 uint32_t* status, void* stream);

/*
 * chopper_join_counters -- counters of serialized hardware-profiling passes
 * attached to the runtime trace's kernels (Section III-A: two or three
 * counters per pass, kernels serialized, no valid timestamps; Section III-B:
 * alignment attaches counters to operations, layers and iterations).
 *
 * A pass ([host] struct, device arrays) lists kernels in its own order with
 * gpu, stream, class and iteration label (NONE: none) and n_cols value
 * columns ([n_cols][n], u64) that go to counter columns dst[0 .. n_cols-1]
 * (each destination used by at most one pass).  A record's key is
 * (gpu, stream, label, ordinal): label = label of its level iter_level
 * marker (idx from chopper_attribute), ordinal = number of records with the
 * same (gpu, stream, label) before it in (start', index) order (`order` from
 * chopper_align); an entry's ordinal counts earlier entries of its pass with
 * the same (gpu, stream, label).  Equal keys and equal classes match:
 * counters_out [16][n] gets the entry's values in the pass's columns (0 when
 * nothing matches, and in columns no pass fills), bit p of matched_out [n]
 * is set for pass p.  Records and entries without an iteration never match.
 * The ordinal is defined for any order of the labels: a label's kernels
 * need not be consecutive along their (gpu, stream).
 * JOIN_MISS: a record with an iteration found no entry in some pass.
 * JOIN_ORDER (warning): along a (gpu, stream), in either order, an iteration
 * label is below an earlier one (iterations out of time order).
 * n_passes <= 8; the records may hold at most 255 (gpu, stream) pairs
 * (CHOPPER_EINVAL otherwise; entries of other pairs never match).  Scratch
 * protocol as above (grows with n, the largest pass and n x 8 bytes per
 * value column of all passes: records far from their sorted order are
 * gathered in that order into a row-major stage and copied back).  The
 * call waits for `stream` twice: the number of the records' pairs is read
 * back, then one word saying which sides hold a label in more than one run
 * (those sides are sorted by label, which waits again inside the sort) and
 * whether the records lie far from their sorted order.
 */
typedef struct {
  int64_t n;
  int32_t n_cols;
  int32_t reserved;
  const uint8_t* gpu;
  const uint8_t* stream;
  const uint8_t* cls;
  const uint32_t* label;
  const uint64_t* values;
  int32_t dst[16];
} chopper_counter_pass;

int chopper_join_counters(const chopper_records* records,
                          const int64_t* start_al, const uint32_t* order,
                          const uint32_t* idx, int32_t depth,
                          int32_t iter_level, const chopper_markers* markers,
                          const chopper_counter_pass* passes,
                          int32_t n_passes, uint64_t* counters_out,
                          uint8_t* matched_out, void* scratch,
                          size_t* scratch_bytes, uint32_t* status,
                          void* stream);

/*
 * chopper_op_stats -- overlap statistics and overhead breakdown of
 * operations (Fig. gemm_overlap: overlap ratio against operation duration,
 * their correlation, 25-75 % and min-max fills of the ratio; Section VI
 * duration breakdown, eqs. 6-10).
 *
 * Instances: compute rows (kind 0, dur > 0) of chopper_aggregate's level
 * op_level -- one operation of one layer in one GPU's iteration -- in group
 * g = p * n_ops + o of their phase and operation labels (p < n_phases,
 * o < n_ops).  Per instance x = floor(ovl * 2^30 / dur) (overlap ratio,
 * Q30) and y = dur + gap (duration with its bubbles, V-B).  From exact
 * 128-bit sums Sx, Sy, Sxx, Syy, Sxy of a group of m instances:
 * cov = m Sxy - Sx Sy, vx = m Sxx - Sx^2, vy = m Syy - Sy^2 (exact), each
 * converted to the nearest double, and out [17][n_phases * n_ops] =
 *   0 pearson    cov / sqrt(vx * vy)  (NaN if m < 2 or a variance is 0)
 *   1 slope      cov / vx  (least-squares duration per Q30 unit of ratio)
 *   2 intercept  (Sy - slope * Sx) / m
 *   3 D0 = intercept, 4 D50 = intercept + slope * 2^29  (eq. 9)
 *   5..9 ratio quantiles v[0], v[(m-1)/4], (v[(m-1)/2] + v[m/2]) / 2,
 *        v[3(m-1)/4], v[m-1] of the sorted x, times 2^-30
 *   10 D_act = Sy / m;  11 D_peak = sum ctr[0] * 1000 / freq_peak_mhz / m
 *   12 Ovr_util = 1 / (sum ctr[1] / sum ctr[0])  (eq. 8)
 *   13 Ovr_inst = (sum ctr[11] / m) / f_gemm[o]  (eq. 7)
 *   14 Ovr_overlap (eq. 9): the median over the GPUs with instances of
 *      their per-GPU D_50% / D_0% (below), sorted, (v[(k-1)/2] + v[k/2]) / 2
 *   15 Ovr_freq = D_act / D_peak / Ovr_overlap  (eq. 10)
 *   16 D_thr = f_gemm[o] / tpt_peak  (eq. 6)
 * (3 and 4 are the least-squares line at 0 and 50 % overlap.)
 *
 * Per-GPU overlap CDF (Fig. per_gpu_overlap_variation: overlap ratio from 0
 * to 1 against duration normalised to the GPU's minimum; Section VI
 * "Overlap overhead": D_50% and D_0% are read off such a CDF).  The
 * instances of group g on GPU h < n_gpus, c = g * n_gpus + h, in CDF order
 * (ascending x, equal x in row order, which is time order on a GPU): with
 * v_k the k-th of m_h instances and y_min their smallest y,
 * gpu_out [9][n_phases * n_ops * n_gpus] at c =
 *   0..4 quantiles v[0], v[(m-1)/4], (v[(m-1)/2] + v[m/2]) / 2, v[3(m-1)/4],
 *        v[m-1] of x, times 2^-30
 *   5 y_min   6 D_0% = y(v_0) / y_min
 *   7 D_50% = (y(v_(m-1)/2) / y_min + y(v_m/2) / y_min) / 2
 *   8 D_50% / D_0%
 * (NaN when m_h = 0); gpu_cnt [n_phases * n_ops * n_gpus] = m_h.  Both
 * may be NULL (computed in scratch, not returned).
 * in exactly these IEEE operations; cnt [n_phases * n_ops] = m.  Empty
 * groups: NaN.  11-13 and 15 need n_counters = 16 (else NaN); f_gemm
 * ([host], n_ops theoretical FLOP counts, per operation label) may be NULL
 * (13 and 16 NaN).  Limits: y < 2^34 and x <= 2^30 (else RANGE, result
 * unspecified), m < 2^26 per group.
 *
 * rows: chopper_aggregate's output (device arrays) for `depth` marker
 * levels, of which level op_level is read; markers: the same markers
 * (device; labels read); n_counters: the rows' counter columns (0 .. 16).
 * out and cnt: device arrays, every element written.  Scratch:
 * caller-owned device memory, size query with scratch == NULL (grows with
 * rows->cap and n_phases * n_ops * n_gpus), 256-byte aligned.  status: device word
 * (RANGE bit).  Enqueued on `stream` without synchronizing.  Returns
 * CHOPPER_EINVAL for a level outside 0 .. depth-1, depth above the markers'
 * depth, sizes out of range (n_gpus included) or a missing pointer
 * (rows->gpu is read), CHOPPER_ESCRATCH for a
 * short scratch buffer.
 */
typedef struct {
  int32_t phase_level;
  int32_t op_level;
  int32_t n_phases;   /* 1 .. 16 */
  int32_t n_ops;      /* 1 .. 128 */
  double freq_peak_mhz;
  double tpt_peak;    /* FLOP per ns */
  const double* f_gemm;
  int32_t n_gpus;     /* 1 .. 256: GPUs of the per-GPU CDFs */
  int32_t reserved;
} chopper_stats_spec;

int chopper_op_stats(const chopper_rows* rows, int32_t depth,
                     int32_t n_counters, const chopper_markers* markers,
                     const chopper_stats_spec* spec, double* out,
                     int64_t* cnt, double* gpu_out, int64_t* gpu_cnt,
                     void* scratch, size_t* scratch_bytes,
                     uint32_t* status, void* stream);

/* Text for a return code. */
const char* chopper_strerror(int code);

/* ABI version (major * 10000 + minor * 100 + patch). */
int chopper_version(void);

/*
 * chopper_time_kernel -- measurement hook.  Until called again, every launch
 * of the library kernel named `name` is bracketed by hipEventRecord(start)
 * and hipEventRecord(stop) on the launch stream (start_event / stop_event
 * are hipEvent_t created by the caller).  name == NULL switches it off.
 * Returns CHOPPER_EINVAL for an unknown name.  chopper_kernel_name(i) lists
 * the names (NULL past the end).
 */
int chopper_time_kernel(const char* name, void* start_event, void* stop_event);
const char* chopper_kernel_name(int i);

#ifdef __cplusplus
}
#endif

#endif /* CHOPPER_H */
