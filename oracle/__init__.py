"""CPU oracle for the trace pipeline -- TEST INFRASTRUCTURE ONLY.

Only tests/, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never imports, links or calls it, and the two share no code.

The arithmetic lives in ``oracle.c`` (plain, single-threaded C, written from
the paper's definitions); this module builds it with gcc and marshals numpy
arrays in and out.

Pinned by tests/test_oracle_pins.py against brute force (per-nanosecond
timelines, linear scans, exact rational least squares), closed forms and
invariants.  Comparison with the paper's own numbers is "parity unpinned":
the paper's traces are not available and its figures carry no data.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

NONE = 0xFFFFFFFF
LEVEL_GPU, LEVEL_WORKLOAD, LEVEL_ALL = 100, 101, 255
BAD_GPU, BAD_CLASS, NEG_DURATION, MARKER_OVERLAP, RANGE = 1, 2, 4, 8, 16
BAD_LEVEL, PATH_CONFLICT = 64, 128
EOVERFLOW = -3


def build(force: bool = True) -> str:
    """Compile oracle.c into liboracle.so (gcc, -O2, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-fPIC", "-shared",
                               "-ffp-contract=off", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


class _Rows(ctypes.Structure):
    _fields_ = [("n_rows", ctypes.c_int64),
                ("level_offset", ctypes.c_int64 * 16),
                ("status", ctypes.c_uint32),
                ("path", ctypes.POINTER(ctypes.c_uint32)),
                ("gpu", ctypes.POINTER(ctypes.c_uint8)),
                ("kind", ctypes.POINTER(ctypes.c_uint8)),
                ("n", ctypes.POINTER(ctypes.c_uint64)),
                ("dur", ctypes.POINTER(ctypes.c_int64)),
                ("gap", ctypes.POINTER(ctypes.c_int64)),
                ("ovl", ctypes.POINTER(ctypes.c_int64)),
                ("tmin", ctypes.POINTER(ctypes.c_int64)),
                ("tmax", ctypes.POINTER(ctypes.c_int64)),
                ("first", ctypes.POINTER(ctypes.c_uint32)),
                ("ctr", ctypes.POINTER(ctypes.c_uint64))]


class Filter(ctypes.Structure):
    """Selection applied before grouping (paper III-C): GPU bit mask, class
    bit mask, optional inclusive range of iteration labels."""
    _fields_ = [("gpu_mask", ctypes.c_uint64 * 4),
                ("class_mask", ctypes.c_uint32),
                ("use_iter", ctypes.c_uint32),
                ("iter_lo", ctypes.c_uint32),
                ("iter_hi", ctypes.c_uint32)]


def make_filter(gpus=None, classes=None, iters=None) -> Filter:
    f = Filter()
    mask = [0, 0, 0, 0]
    for g in (range(256) if gpus is None else gpus):
        mask[g >> 6] |= 1 << (g & 63)
    for i in range(4):
        f.gpu_mask[i] = mask[i]
    cm = 0
    for c in (range(32) if classes is None else classes):
        cm |= 1 << c
    f.class_mask = cm
    if iters is not None:
        f.use_iter = 1
        f.iter_lo, f.iter_hi = int(iters[0]), int(iters[1])
    return f


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if (not os.path.exists(_LIB) or
            os.path.getmtime(_LIB) < os.path.getmtime(_SRC)):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i64, i32 = ctypes.c_int64, ctypes.c_int32
    lib.orc_fit.argtypes = [i64, P, P, P, i32, P, P, P]
    lib.orc_fit.restype = ctypes.c_int
    lib.orc_transform.argtypes = [i64, P, P, i32, P, P, P, P]
    lib.orc_transform.restype = ctypes.c_uint32
    lib.orc_order.argtypes = [i64, P, P, P, P, i32, P]
    lib.orc_order.restype = None
    lib.orc_attribute.argtypes = [i64, P, P, i64, P, P, P, P, i32, i32, P]
    lib.orc_attribute.restype = ctypes.c_uint32
    lib.orc_overlap.argtypes = [i64, P, P, P, P, P, i64, P, P, P, i32, P, P,
                                P, P]
    lib.orc_overlap.restype = ctypes.c_uint32
    lib.orc_aggregate.argtypes = [i64, P, P, P, P, P, P, P, P, i32, i32, i32,
                                  P, P, i64, ctypes.POINTER(_Rows)]
    lib.orc_aggregate.restype = ctypes.c_int
    lib.orc_rows_free.argtypes = [ctypes.POINTER(_Rows)]
    lib.orc_rows_free.restype = None
    lib.orc_ratios.argtypes = [i64, P, P, P, P, i32, i64, ctypes.c_double, P]
    lib.orc_ratios.restype = None
    lib.orc_window_fractions.argtypes = [i64, P, P]
    lib.orc_window_fractions.restype = None
    lib.orc_views.argtypes = [i64, P, P, P, P, i32, P, P, i64, P, P, i32, i32,
                              i32, i32, i32, i32, ctypes.c_uint32, i64, P, P,
                              P, P, P, P, P, P, P, P, P, P]
    lib.orc_views.restype = ctypes.c_int
    lib.orc_launch_split.argtypes = [i64, P, P, P, P, P, P, P, P]
    lib.orc_launch_split.restype = None
    lib.orc_join.argtypes = [i64, P, P, P, P, P, i32, P, P, P, P, P, P, P, P,
                             P, P]
    lib.orc_join.restype = ctypes.c_uint32
    lib.orc_op_stats.argtypes = [i64, i64, i64, P, i32, i32, P, P, P, P, P,
                                 i32, P, i32, i32, ctypes.c_double,
                                 ctypes.c_double, P, P, P, P, i32, P, P]
    lib.orc_op_stats.restype = None
    _lib = lib
    return lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


# ---------------------------------------------------------------------------
def fit(a_gpu, a_local, a_ref, n_gpus: int):
    """Per-GPU clock parameters (x0, C, D_q48) and the return code."""
    lib = _load()
    a_gpu, a_local, a_ref = (_c(a_gpu, np.uint8), _c(a_local, np.int64),
                             _c(a_ref, np.int64))
    x0 = np.zeros(n_gpus, np.int64)
    c = np.zeros(n_gpus, np.int64)
    d = np.zeros(n_gpus, np.int64)
    rc = lib.orc_fit(a_gpu.shape[0], _p(a_gpu), _p(a_local), _p(a_ref),
                     n_gpus, _p(x0), _p(c), _p(d))
    return x0, c, d, rc


def transform(gpu, t, n_gpus, x0, c, d):
    lib = _load()
    gpu, t = _c(gpu, np.uint8), _c(t, np.int64)
    out = np.empty_like(t)
    st = lib.orc_transform(t.shape[0], _p(gpu), _p(t), n_gpus,
                           _p(_c(x0, np.int64)), _p(_c(c, np.int64)),
                           _p(_c(d, np.int64)), _p(out))
    return out, int(st)


def order(gpu, stream, cls, s, by_kind: bool):
    lib = _load()
    gpu, stream, cls, s = (_c(gpu, np.uint8), _c(stream, np.uint8),
                           _c(cls, np.uint8), _c(s, np.int64))
    out = np.empty(gpu.shape[0], np.uint32)
    lib.orc_order(gpu.shape[0], _p(gpu), _p(stream), _p(cls), _p(s),
                  1 if by_kind else 0, _p(out))
    return out


def attribute(gpu, s, m_gpu, m_level, ms, me, depth, n_gpus):
    lib = _load()
    gpu, s = _c(gpu, np.uint8), _c(s, np.int64)
    m_gpu, m_level = _c(m_gpu, np.uint8), _c(m_level, np.uint8)
    ms, me = _c(ms, np.int64), _c(me, np.int64)
    n = gpu.shape[0]
    idx = np.empty((depth, n), np.uint32)
    st = lib.orc_attribute(n, _p(gpu), _p(s), m_gpu.shape[0], _p(m_gpu),
                           _p(m_level), _p(ms), _p(me), depth, n_gpus,
                           _p(idx))
    return idx, int(st)


def overlap(gpu, stream, cls, s, e, m_gpu, ms, me, n_gpus):
    lib = _load()
    gpu, stream, cls = (_c(gpu, np.uint8), _c(stream, np.uint8),
                        _c(cls, np.uint8))
    s, e = _c(s, np.int64), _c(e, np.int64)
    m_gpu, ms, me = _c(m_gpu, np.uint8), _c(ms, np.int64), _c(me, np.int64)
    n, nm = gpu.shape[0], m_gpu.shape[0]
    ovl = np.empty(n, np.int64)
    gap = np.empty(n, np.int64)
    mwin = np.empty((nm, 4), np.int64)
    gwin = np.empty((n_gpus, 6), np.int64)
    st = lib.orc_overlap(n, _p(gpu), _p(stream), _p(cls), _p(s), _p(e), nm,
                         _p(m_gpu), _p(ms), _p(me), n_gpus, _p(ovl), _p(gap),
                         _p(mwin), _p(gwin))
    return dict(ovl=ovl, gap=gap, mwin=mwin, gwin=gwin, status=int(st))


def aggregate(gpu, cls, s, e, idx, gap, ovl, counters, depth, level=LEVEL_ALL,
              filt: Optional[Filter] = None, m_label=None) -> Dict:
    lib = _load()
    gpu, cls = _c(gpu, np.uint8), _c(cls, np.uint8)
    s, e = _c(s, np.int64), _c(e, np.int64)
    idx = _c(idx, np.uint32)
    gap, ovl = _c(gap, np.int64), _c(ovl, np.int64)
    n = gpu.shape[0]
    nc = 0 if counters is None else counters.shape[0]
    ctr = None if counters is None else _c(counters, np.uint64)
    ml = _c(m_label if m_label is not None else np.zeros(0), np.uint32)
    rows = _Rows()
    lib.orc_aggregate(n, _p(gpu), _p(cls), _p(s), _p(e), _p(idx), _p(gap),
                      _p(ovl), _p(ctr), nc, depth, level,
                      None if filt is None else ctypes.byref(filt), _p(ml),
                      ml.shape[0], ctypes.byref(rows))
    nr = rows.n_rows

    def arr(ptr, count, dt):
        if count == 0:
            return np.zeros(0, dt)
        return np.ctypeslib.as_array(ptr, shape=(count,)).astype(dt, copy=True)

    out = dict(
        n_rows=nr,
        level_offset=np.array(rows.level_offset[:depth + 3], np.int64),
        status=int(rows.status),
        path=arr(rows.path, nr * depth, np.uint32).reshape(depth, nr),
        gpu=arr(rows.gpu, nr, np.uint8), kind=arr(rows.kind, nr, np.uint8),
        n=arr(rows.n, nr, np.uint64), dur=arr(rows.dur, nr, np.int64),
        gap=arr(rows.gap, nr, np.int64), ovl=arr(rows.ovl, nr, np.int64),
        tmin=arr(rows.tmin, nr, np.int64), tmax=arr(rows.tmax, nr, np.int64),
        first=arr(rows.first, nr, np.uint32),
        ctr=arr(rows.ctr, nr * nc, np.uint64).reshape(nc, nr))
    lib.orc_rows_free(ctypes.byref(rows))
    return out


def ratios(rows: Dict, freq_peak_mhz: float = 2100.0) -> np.ndarray:
    lib = _load()
    nr = int(rows["n_rows"])
    nc = rows["ctr"].shape[0]
    out = np.empty((6, nr), np.float64)
    ctr = _c(rows["ctr"], np.uint64)
    lib.orc_ratios(nr, _p(_c(rows["n"], np.uint64)),
                   _p(_c(rows["dur"], np.int64)), _p(_c(rows["ovl"], np.int64)),
                   _p(ctr), nc, nr, float(freq_peak_mhz), _p(out))
    return out


def window_fractions(w: np.ndarray) -> np.ndarray:
    lib = _load()
    w = _c(w, np.int64).reshape(-1, 4)
    out = np.empty(w.shape, np.float64)
    lib.orc_window_fractions(w.shape[0], _p(w), _p(out))
    return out


OP_STATS = ("pearson", "slope", "intercept", "d0", "d50", "q0", "q25",
            "q50", "q75", "q100", "d_act", "d_peak", "ovr_util", "ovr_inst",
            "ovr_overlap", "ovr_freq", "d_thr")


OP_CDF = ("q0", "q25", "q50", "q75", "q100", "y_min", "d0", "d50", "ovr")


def op_stats(rows: Dict, m_label, depth, phase_level=1, op_level=3,
             n_phases=3, n_ops=64, freq_peak_mhz=2100.0, tpt_peak=1.0,
             f_gemm=None, n_gpus=None, per_gpu=False):
    """Overlap statistics and overhead breakdown per (phase, operation)
    (Fig. gemm_overlap, Section VI eqs. 6-10) from the rows of the
    operation level, with the per-GPU overlap CDFs (Fig.
    per_gpu_overlap_variation) that eq. 9 is read from; definitions in
    oracle.c.  Returns (out [17][P*O], cnt [P*O]), and with per_gpu also
    (gout [9][P*O*NG], gcnt [P*O*NG]).  n_gpus defaults to one more than
    the largest GPU id of the rows."""
    lib = _load()
    gpu = _c(rows["gpu"], np.uint8) if "gpu" in rows else \
        np.zeros(int(rows["n"].shape[0]), np.uint8)
    if n_gpus is None:
        n_gpus = int(gpu.max()) + 1 if gpu.size else 1
    lo = rows["level_offset"]
    nr = int(rows["n"].shape[0])
    path = _c(rows["path"], np.uint32)
    nc = int(rows["ctr"].shape[0]) if rows["ctr"] is not None else 0
    ctr = _c(rows["ctr"], np.uint64) if nc else np.zeros(1, np.uint64)
    P_, O_ = int(n_phases), int(n_ops)
    NG = int(n_gpus)
    out = np.zeros((17, P_ * O_))
    cnt = np.zeros(P_ * O_, np.int64)
    gout = np.zeros((9, P_ * O_ * NG))
    gcnt = np.zeros(P_ * O_ * NG, np.int64)
    fg = None if f_gemm is None else _c(f_gemm, np.float64)
    a = [path, _c(rows["kind"], np.uint8), _c(rows["dur"], np.int64),
         _c(rows["gap"], np.int64), _c(rows["ovl"], np.int64), ctr,
         _c(m_label, np.uint32)]
    lib.orc_op_stats(int(lo[op_level]), int(lo[op_level + 1]), nr,
                     _p(a[0]), phase_level, op_level, _p(a[1]), _p(a[2]),
                     _p(a[3]), _p(a[4]), _p(a[5]), nc, _p(a[6]), P_, O_,
                     float(freq_peak_mhz), float(tpt_peak), _p(fg), _p(out),
                     _p(cnt), _p(gpu), NG, _p(gout), _p(gcnt))
    if per_gpu:
        return out, cnt, gout, gcnt
    return out, cnt


JOIN_MISS, JOIN_ORDER = 256, 512


def join(gpu, stream, cls, s, lab, passes):
    """Counter-pass join (III-A, III-B): counters [16][n] u64 and the matched
    pass bits [n] of every record, and the status; definitions in
    oracle.c.  passes: dicts with gpu, stream, cls, lab ([m] each), values
    ([c][m] u64) and dst (c destination columns)."""
    lib = _load()
    n = int(np.asarray(s).shape[0])
    P_ = len(passes)
    keep = []
    arr = lambda vals, dt: (ctypes.c_void_p * max(P_, 1))(*[
        _p(v) for v in vals])
    g = [_c(q["gpu"], np.uint8) for q in passes]
    st = [_c(q["stream"], np.uint8) for q in passes]
    cl = [_c(q["cls"], np.uint8) for q in passes]
    lb = [_c(q["lab"], np.uint32) for q in passes]
    vl = [_c(q["values"], np.uint64) for q in passes]
    keep += [g, st, cl, lb, vl]
    pn = np.array([int(np.asarray(q["gpu"]).shape[0]) for q in passes] or [0],
                  np.int64)
    pc = np.array([len(q["dst"]) for q in passes] or [0], np.int32)
    pd = np.zeros(16 * max(P_, 1), np.int32)
    for i, q in enumerate(passes):
        pd[16 * i:16 * i + len(q["dst"])] = q["dst"]
    counters = np.zeros((16, n), np.uint64)
    matched = np.zeros(n, np.uint8)
    a = [_c(gpu, np.uint8), _c(stream, np.uint8), _c(cls, np.uint8),
         _c(s, np.int64), _c(lab, np.uint32)]
    st_ = lib.orc_join(n, *[_p(x) for x in a], P_, _p(pn), _p(pc), _p(pd),
                       arr(g, None), arr(st, None), arr(cl, None),
                       arr(lb, None), arr(vl, None), _p(counters),
                       _p(matched))
    return counters, matched, int(st_)


def launch_split(gpu, stream, cls, s, e, tl):
    """Preparation and call overhead of every record (V-D eqs. 1-3) from
    aligned start, end and dispatch times; definitions in oracle.c."""
    lib = _load()
    n = int(np.asarray(s).shape[0])
    a = [_c(gpu, np.uint8), _c(stream, np.uint8), _c(cls, np.uint8),
         _c(s, np.int64), _c(e, np.int64), _c(tl, np.int64)]
    prep = np.zeros(n, np.int64)
    call = np.zeros(n, np.int64)
    lib.orc_launch_split(n, *[_p(x) for x in a], _p(prep), _p(call))
    return prep, call


def views(cls, s, e, idx, gap, ovl, m_level, m_label, iter_level=0,
          phase_level=1, op_level=3, n_phases=3, n_ops=64, n_iters=1,
          warmup=0) -> Dict:
    """Re-keyed views and medians (Fig. end_to_end, V-B / Fig.
    operation_time, warm-up iterations of IV); definitions in oracle.c."""
    lib = _load()
    n = int(np.asarray(s).shape[0])
    nm = int(np.asarray(m_level).shape[0])
    idx = _c(idx, np.uint32).reshape(-1)
    depth = idx.shape[0] // n if n else 0
    U = int((np.asarray(m_level) == iter_level).sum())
    P, O, NI = int(n_phases), int(n_ops), int(n_iters)
    out = dict(
        n_units=np.zeros(1, np.int64), unit_marker=np.zeros(U, np.uint32),
        cls_tab=np.zeros((3, U * P * 8), np.uint64),
        op_tab=np.zeros((4, U * P * O * 2), np.uint64),
        busy=np.zeros(U, np.int64), iter_max=np.zeros(NI, np.int64),
        cls_med=np.zeros((3, P * 8)), cls_cnt=np.zeros(P * 8, np.int64),
        op_med=np.zeros((3, P * O * 2)), op_cnt=np.zeros(P * O * 2, np.int64),
        iter_med=np.zeros(1), iter_cnt=np.zeros(1, np.int64))
    a = [_c(cls, np.uint8), _c(s, np.int64), _c(e, np.int64), idx,
         _c(gap, np.int64), _c(ovl, np.int64), _c(m_level, np.uint8),
         _c(m_label, np.uint32)]
    rc = lib.orc_views(n, _p(a[0]), _p(a[1]), _p(a[2]), _p(a[3]), depth,
                       _p(a[4]), _p(a[5]), nm, _p(a[6]), _p(a[7]), iter_level,
                       phase_level, op_level, P, O, NI, warmup, U,
                       *[_p(out[k]) for k in (
                           "n_units", "unit_marker", "cls_tab", "op_tab",
                           "busy", "iter_max", "cls_med", "cls_cnt", "op_med",
                           "op_cnt", "iter_med", "iter_cnt")])
    assert rc == 0
    out["n_units"] = int(out["n_units"][0])
    out["iter_med"] = float(out["iter_med"][0])
    out["iter_cnt"] = int(out["iter_cnt"][0])
    return out


# ---------------------------------------------------------------------------
def run(tr, level: int = LEVEL_ALL, filt: Optional[Filter] = None,
        freq_peak_mhz: float = 2100.0) -> Dict:
    """The whole pipeline on a tracegen.Trace: align, attribute, overlap,
    aggregate, derived ratios."""
    G = tr.n_gpus
    x0, c, d, rc = fit(tr.a_gpu, tr.a_local, tr.a_ref, G)
    s, st1 = transform(tr.gpu, tr.start, G, x0, c, d)
    e, st2 = transform(tr.gpu, tr.end, G, x0, c, d)
    ms, st3 = transform(tr.m_gpu, tr.m_start, G, x0, c, d)
    me, st4 = transform(tr.m_gpu, tr.m_end, G, x0, c, d)
    status = st1 | st2 | st3 | st4
    if (e < s).any() or (tr.end < tr.start).any():
        status |= NEG_DURATION
    if (tr.cls >= 8).any():
        status |= BAD_CLASS
    ordr = order(tr.gpu, tr.stream, tr.cls, s, False)
    kord = order(tr.gpu, tr.stream, tr.cls, s, True)
    idx, st5 = attribute(tr.gpu, s, tr.m_gpu, tr.m_level, ms, me, tr.depth, G)
    ov = overlap(tr.gpu, tr.stream, tr.cls, s, e, tr.m_gpu, ms, me, G)
    rows = aggregate(tr.gpu, tr.cls, s, e, idx, ov["gap"], ov["ovl"],
                     tr.counters, tr.depth, level, filt, tr.m_label)
    rat = ratios(rows, freq_peak_mhz)
    wf = window_fractions(ov["mwin"])
    status |= st5 | ov["status"] | rows["status"]
    return dict(x0=x0, c=c, d=d, fit_rc=rc, start=s, end=e, mstart=ms,
                mend=me, order=ordr, korder=kord, idx=idx, ovl=ov["ovl"],
                gap=ov["gap"], mwin=ov["mwin"], gwin=ov["gwin"], rows=rows,
                ratios=rat, wfrac=wf, status=status)
