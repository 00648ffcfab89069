"""ctypes binding of libchopper: argument marshalling only.

Every step runs in the HIP library; this module passes device pointers of
torch tensors, the current HIP stream and host structs, and raises on error
codes.  There is no fallback: without libchopper.so the import fails.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libchopper.so")

NONE = 0xFFFFFFFF
LEVEL_GPU, LEVEL_WORKLOAD, LEVEL_ALL = 100, 101, 255
ST_BAD_GPU, ST_BAD_CLASS, ST_NEG_DURATION, ST_MARKER_OVERLAP = 1, 2, 4, 8
ST_RANGE, ST_ROWS_OVERFLOW, ST_BAD_LEVEL, ST_PATH_CONFLICT = 16, 32, 64, 128
OK, EINVAL, ESCRATCH, EOVERFLOW, EHIP = 0, -1, -2, -3, -4

P = ctypes.c_void_p


class Records(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("n_gpus", ctypes.c_int32),
                ("n_counters", ctypes.c_int32), ("gpu", P), ("stream", P),
                ("cls", P), ("op_id", P), ("start_ns", P), ("end_ns", P),
                ("counters", P)]


class Markers(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("depth", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("gpu", P), ("level", P),
                ("start_ns", P), ("end_ns", P), ("label", P)]


class Anchors(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("gpu", P), ("local_ns", P),
                ("ref_ns", P)]


class Clock(ctypes.Structure):
    _fields_ = [("x0", ctypes.c_int64), ("c", ctypes.c_int64),
                ("d_q48", ctypes.c_int64)]


class Filter(ctypes.Structure):
    _fields_ = [("gpu_mask", ctypes.c_uint64 * 4),
                ("class_mask", ctypes.c_uint32), ("use_iter", ctypes.c_uint32),
                ("iter_lo", ctypes.c_uint32), ("iter_hi", ctypes.c_uint32)]


class Rows(ctypes.Structure):
    _fields_ = [("cap", ctypes.c_int64), ("level_offset", P), ("path", P),
                ("gpu", P), ("kind", P), ("n", P), ("dur", P), ("gap", P),
                ("ovl", P), ("tmin", P), ("tmax", P), ("first", P),
                ("ctr", P)]


class ViewSpec(ctypes.Structure):
    _fields_ = [("iter_level", ctypes.c_int32), ("phase_level", ctypes.c_int32),
                ("op_level", ctypes.c_int32), ("n_phases", ctypes.c_int32),
                ("n_ops", ctypes.c_int32), ("n_iters", ctypes.c_int32),
                ("warmup", ctypes.c_uint32), ("reserved", ctypes.c_int32)]


_VIEW_OUT = ("n_units", "unit_marker", "cls_tab", "op_tab", "busy",
             "iter_max", "cls_med", "cls_cnt", "op_med", "op_cnt", "iter_med",
             "iter_cnt")


class ViewOut(ctypes.Structure):
    _fields_ = [("unit_cap", ctypes.c_int64)] + [(k, P) for k in _VIEW_OUT]


class StatsSpec(ctypes.Structure):
    _fields_ = [("phase_level", ctypes.c_int32), ("op_level", ctypes.c_int32),
                ("n_phases", ctypes.c_int32), ("n_ops", ctypes.c_int32),
                ("freq_peak_mhz", ctypes.c_double),
                ("tpt_peak", ctypes.c_double),
                ("f_gemm", ctypes.POINTER(ctypes.c_double)),
                ("n_gpus", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class CounterPass(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("n_cols", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("gpu", P), ("stream", P),
                ("cls", P), ("label", P), ("values", P),
                ("dst", ctypes.c_int32 * 16)]


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
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it first "
            "(python -m paper_2512_08242_amd.build or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    i64, i32 = ctypes.c_int64, ctypes.c_int32
    SZ = ctypes.POINTER(ctypes.c_size_t)
    lib.chopper_align.argtypes = [ctypes.POINTER(Records),
                                  ctypes.POINTER(Markers),
                                  ctypes.POINTER(Anchors),
                                  ctypes.POINTER(Clock), P, P, P, P, P, P, P,
                                  SZ, P, P]
    lib.chopper_attribute.argtypes = [ctypes.POINTER(Records), P,
                                      ctypes.POINTER(Markers), P, P, P, P, SZ,
                                      P, P]
    lib.chopper_overlap.argtypes = [ctypes.POINTER(Records), P, P, P, P,
                                    ctypes.POINTER(Markers), P, P, P, P, P, P,
                                    P, SZ, P, P]
    lib.chopper_aggregate.argtypes = [ctypes.POINTER(Records), P, P, P, P, i32,
                                      P, P, ctypes.POINTER(Markers), i32,
                                      ctypes.POINTER(Filter),
                                      ctypes.POINTER(Rows), P, SZ, P, P, P]
    lib.chopper_ratios.argtypes = [ctypes.POINTER(Rows), i32, i32,
                                   ctypes.c_double, P, P]
    lib.chopper_window_fractions.argtypes = [i64, P, P, P]
    lib.chopper_launch_split.argtypes = [ctypes.POINTER(Records),
                                         ctypes.POINTER(Clock), P, P, P, P, P,
                                         P, SZ, P, P]
    lib.chopper_launch_split_noalloc.argtypes = [ctypes.POINTER(Records),
                                                 ctypes.POINTER(Clock), P, P,
                                                 P, P, P, P, P]
    lib.chopper_op_stats.argtypes = [ctypes.POINTER(Rows), i32, i32,
                                     ctypes.POINTER(Markers),
                                     ctypes.POINTER(StatsSpec), P, P, P, P,
                                     P, SZ, P, P]
    lib.chopper_join_counters.argtypes = [ctypes.POINTER(Records), P, P, P,
                                          i32, i32, ctypes.POINTER(Markers),
                                          ctypes.POINTER(CounterPass), i32, P,
                                          P, P, SZ, P, P]
    lib.chopper_views.argtypes = [ctypes.POINTER(Records), P, P, P, i32, P,
                                  ctypes.POINTER(Markers),
                                  ctypes.POINTER(Rows),
                                  ctypes.POINTER(ViewSpec),
                                  ctypes.POINTER(ViewOut), P, SZ, P, P]
    lib.chopper_strerror.argtypes = [ctypes.c_int]
    lib.chopper_strerror.restype = ctypes.c_char_p
    lib.chopper_version.restype = ctypes.c_int
    lib.chopper_kernel_name.argtypes = [ctypes.c_int]
    lib.chopper_kernel_name.restype = ctypes.c_char_p
    lib.chopper_time_kernel.argtypes = [ctypes.c_char_p, P, P]
    for name in ("chopper_align", "chopper_attribute", "chopper_overlap",
                 "chopper_aggregate", "chopper_ratios",
                 "chopper_window_fractions", "chopper_version",
                 "chopper_time_kernel", "chopper_views",
                 "chopper_launch_split", "chopper_launch_split_noalloc",
                 "chopper_join_counters",
                 "chopper_op_stats"):
        getattr(lib, name).restype = ctypes.c_int
    return lib


lib = _load()


def _check(rc: int, what: str):
    if rc != OK:
        raise RuntimeError(f"{what}: {lib.chopper_strerror(rc).decode()} "
                           f"({rc})")


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def kernel_names():
    out, i = [], 0
    while True:
        s = lib.chopper_kernel_name(i)
        if s is None:
            return out
        out.append(s.decode())
        i += 1


def time_kernel(name: Optional[str], start=None, stop=None):
    """Bracket every launch of library kernel `name` with two torch/HIP
    events (None switches it off)."""
    if name is None:
        _check(lib.chopper_time_kernel(None, None, None), "time_kernel")
        return
    for ev in (start, stop):
        if not ev.cuda_event:      # torch creates the HIP event lazily
            ev.record()
    _check(lib.chopper_time_kernel(name.encode(),
                                   ctypes.c_void_p(start.cuda_event),
                                   ctypes.c_void_p(stop.cuda_event)),
           "time_kernel")


# ---------------------------------------------------------------------------
class DeviceTrace:
    """A trace resident in device memory (structure of arrays)."""

    def __init__(self, tr, device="cuda"):
        dev = torch.device(device)
        t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
        self.n_gpus = int(tr.n_gpus)
        self.depth = int(tr.depth)
        self.n = int(tr.n)
        self.n_markers = int(tr.n_markers)
        self.gpu, self.stream, self.cls = t(tr.gpu), t(tr.stream), t(tr.cls)
        self.op_id = t(tr.op_id.astype(np.int32).view(np.int32))
        self.start, self.end = t(tr.start), t(tr.end)
        self.counters = (None if tr.counters is None else
                         t(tr.counters.view(np.int64)))
        self.n_counters = 0 if tr.counters is None else tr.counters.shape[0]
        self.m_gpu, self.m_level = t(tr.m_gpu), t(tr.m_level)
        self.m_start, self.m_end = t(tr.m_start), t(tr.m_end)
        self.m_label = t(tr.m_label.view(np.int32))
        # anchors stay on the host
        self.a_gpu = np.ascontiguousarray(tr.a_gpu, np.uint8)
        self.a_local = np.ascontiguousarray(tr.a_local, np.int64)
        self.a_ref = np.ascontiguousarray(tr.a_ref, np.int64)

    def records(self) -> Records:
        r = Records()
        r.n, r.n_gpus, r.n_counters = self.n, self.n_gpus, self.n_counters
        r.gpu, r.stream, r.cls = _ptr(self.gpu), _ptr(self.stream), _ptr(
            self.cls)
        r.op_id = _ptr(self.op_id)
        r.start_ns, r.end_ns = _ptr(self.start), _ptr(self.end)
        r.counters = _ptr(self.counters)
        return r

    def markers(self) -> Markers:
        m = Markers()
        m.n, m.depth = self.n_markers, self.depth
        m.gpu, m.level = _ptr(self.m_gpu), _ptr(self.m_level)
        m.start_ns, m.end_ns = _ptr(self.m_start), _ptr(self.m_end)
        m.label = _ptr(self.m_label)
        return m

    def anchors(self) -> Anchors:
        a = Anchors()
        a.n = int(self.a_gpu.shape[0])
        a.gpu = self.a_gpu.ctypes.data_as(P)
        a.local_ns = self.a_local.ctypes.data_as(P)
        a.ref_ns = self.a_ref.ctypes.data_as(P)
        return a

    def nbytes(self) -> int:
        tot = 0
        for v in self.__dict__.values():
            if isinstance(v, torch.Tensor):
                tot += v.numel() * v.element_size()
        return tot


def _scratch(query, dev) -> torch.Tensor:
    sz = ctypes.c_size_t(0)
    _check(query(None, ctypes.byref(sz)), "scratch query")
    return torch.empty(max(int(sz.value), 256) + 256, dtype=torch.uint8,
                       device=dev)


def _aligned(buf: torch.Tensor):
    p = buf.data_ptr()
    return ctypes.c_void_p((p + 255) & ~255), ctypes.c_size_t(
        buf.numel() - ((-p) % 256))


class RowsBuffer:
    """Device arrays for aggregated rows of capacity `cap`."""

    def __init__(self, cap: int, depth: int, n_counters: int, device):
        cap = max(int(cap), 0)
        e = lambda *shape, dt: torch.empty(*shape, dtype=dt, device=device)
        self.cap, self.depth, self.n_counters = cap, depth, n_counters
        self.level_offset = torch.zeros(depth + 3, dtype=torch.int64,
                                        device=device)
        self.path = e(max(depth, 1), max(cap, 1), dt=torch.int32)
        self.gpu = e(max(cap, 1), dt=torch.uint8)
        self.kind = e(max(cap, 1), dt=torch.uint8)
        self.n = e(max(cap, 1), dt=torch.int64)
        self.dur = e(max(cap, 1), dt=torch.int64)
        self.gap = e(max(cap, 1), dt=torch.int64)
        self.ovl = e(max(cap, 1), dt=torch.int64)
        self.tmin = e(max(cap, 1), dt=torch.int64)
        self.tmax = e(max(cap, 1), dt=torch.int64)
        self.first = e(max(cap, 1), dt=torch.int32)
        self.ctr = e(max(n_counters, 1), max(cap, 1), dt=torch.int64)

    def struct(self) -> Rows:
        r = Rows()
        r.cap = self.cap
        for name in ("level_offset", "path", "gpu", "kind", "n", "dur", "gap",
                     "ovl", "tmin", "tmax", "first", "ctr"):
            setattr(r, name, _ptr(getattr(self, name)))
        if self.cap == 0:
            for name in ("path", "gpu", "kind", "n", "dur", "gap", "ovl",
                         "tmin", "tmax", "first", "ctr"):
                setattr(r, name, None)
        return r

    def to_numpy(self) -> Dict[str, np.ndarray]:
        lo = self.level_offset.cpu().numpy()
        nr = int(min(lo[-1], self.cap))
        u = lambda t, dt: t.cpu().numpy().view(dt)
        return dict(
            n_rows=nr, level_offset=lo,
            path=u(self.path[:self.depth, :nr], np.uint32).reshape(
                self.depth, nr),
            gpu=u(self.gpu[:nr], np.uint8), kind=u(self.kind[:nr], np.uint8),
            n=u(self.n[:nr], np.uint64), dur=u(self.dur[:nr], np.int64),
            gap=u(self.gap[:nr], np.int64), ovl=u(self.ovl[:nr], np.int64),
            tmin=u(self.tmin[:nr], np.int64), tmax=u(self.tmax[:nr], np.int64),
            first=u(self.first[:nr], np.uint32),
            ctr=u(self.ctr[:self.n_counters, :nr], np.uint64).reshape(
                self.n_counters, nr))


class Pipeline:
    """align -> attribute -> overlap -> aggregate -> ratios over one
    DeviceTrace with preallocated outputs and scratch."""

    def __init__(self, dt: DeviceTrace, level: int = LEVEL_ALL,
                 filt: Optional[Filter] = None, freq_peak_mhz: float = 2100.0):
        self.dt = dt
        self.level, self.filt, self.freq = level, filt, float(freq_peak_mhz)
        dev = dt.start.device
        n, nm, D = dt.n, dt.n_markers, dt.depth
        e = lambda *s, dt_: torch.empty(*s, dtype=dt_, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.start = e(max(n, 1), dt_=torch.int64)
        self.end = e(max(n, 1), dt_=torch.int64)
        self.mstart = e(max(nm, 1), dt_=torch.int64)
        self.mend = e(max(nm, 1), dt_=torch.int64)
        self.order = e(max(n, 1), dt_=torch.int32)
        self.korder = e(max(n, 1), dt_=torch.int32)
        self.idx = e(D, max(n, 1), dt_=torch.int32)
        self.ovl = e(max(n, 1), dt_=torch.int64)
        self.gap = e(max(n, 1), dt_=torch.int64)
        self.mwin = e(max(nm, 1), 4, dt_=torch.int64)
        self.gwin = e(dt.n_gpus, 6, dt_=torch.int64)
        self.wfrac = e(max(nm, 1), 4, dt_=torch.float64)
        self.clocks = (Clock * dt.n_gpus)()
        self._rec, self._mk, self._anc = dt.records(), dt.markers(), \
            dt.anchors()
        self.rows = RowsBuffer(0, D, dt.n_counters, dev)
        self.ratios = e(6, 1, dt_=torch.float64)
        self._scr = {}
        self._ready = None      # event gap / ovl are complete at (see step)
        for name in ("align", "attribute", "overlap"):
            self._scr[name] = _scratch(
                lambda s, b, nm_=name: self._call(nm_, s, b), dev)
        # size the rows from a first aggregation
        self._scr["aggregate"] = _scratch(
            lambda s, b: self._call("aggregate", s, b), dev)
        self.align()
        self.attribute()
        self.overlap()
        self.aggregate()
        torch.cuda.synchronize()
        need = int(self.rows.level_offset[-1].item())
        self.rows = RowsBuffer(need, D, dt.n_counters, dev)
        self._scr["aggregate"] = _scratch(
            lambda s, b: self._call("aggregate", s, b), dev)
        self.ratios = e(6, max(need, 1), dt_=torch.float64)
        self.status.zero_()       # drop the sizing call's ROWS_OVERFLOW

    # raw entry points -------------------------------------------------------
    def _call(self, name, scratch, sbytes):
        dt = self.dt
        rec, mk = self._rec, self._mk
        st = _ptr(self.status)
        s = _stream()
        if name == "align":
            return lib.chopper_align(
                ctypes.byref(rec), ctypes.byref(mk), ctypes.byref(self._anc),
                self.clocks, _ptr(self.start), _ptr(self.end),
                _ptr(self.mstart), _ptr(self.mend), _ptr(self.order),
                _ptr(self.korder), scratch, sbytes, st, s)
        if name == "attribute":
            return lib.chopper_attribute(
                ctypes.byref(rec), _ptr(self.start), ctypes.byref(mk),
                _ptr(self.mstart), _ptr(self.mend), _ptr(self.idx), scratch,
                sbytes, st, s)
        if name == "overlap":
            return lib.chopper_overlap(
                ctypes.byref(rec), _ptr(self.start), _ptr(self.end),
                _ptr(self.order), _ptr(self.korder), ctypes.byref(mk),
                _ptr(self.mstart), _ptr(self.mend), _ptr(self.ovl),
                _ptr(self.gap), _ptr(self.mwin), _ptr(self.gwin), scratch,
                sbytes, st, s)
        if name == "aggregate":
            rows = self.rows.struct()
            self._rows_struct = rows
            return lib.chopper_aggregate(
                ctypes.byref(rec), _ptr(self.start), _ptr(self.end),
                _ptr(self.korder), _ptr(self.idx), dt.depth, _ptr(self.gap),
                _ptr(self.ovl), ctypes.byref(mk), self.level,
                None if self.filt is None else ctypes.byref(self.filt),
                ctypes.byref(rows), scratch, sbytes, st,
                None if self._ready is None
                else ctypes.c_void_p(self._ready.cuda_event), s)
        raise ValueError(name)

    def _run(self, name):
        scr, sb = _aligned(self._scr[name])
        _check(self._call(name, scr, ctypes.byref(sb)), name)

    def align(self):
        self._run("align")

    def attribute(self):
        self._run("attribute")

    def overlap(self):
        self._run("overlap")

    def aggregate(self):
        self._run("aggregate")

    def derive(self):
        self.derive_rows()
        self.derive_windows()

    def derive_rows(self):
        rows = self.rows.struct()
        _check(lib.chopper_ratios(ctypes.byref(rows), self.dt.depth,
                                  self.dt.n_counters, self.freq,
                                  _ptr(self.ratios), _stream()), "ratios")

    def derive_windows(self):
        _check(lib.chopper_window_fractions(self.dt.n_markers,
                                            _ptr(self.mwin), _ptr(self.wfrac),
                                            _stream()), "window_fractions")

    def launch_split(self, launch_ns: torch.Tensor):
        """Preparation and call overhead of every record (chopper_launch_split)
        from dispatch times on each GPU's local clock; returns (prep, call)
        device tensors in input order.  Needs align and overlap to have
        run."""
        dt = self.dt
        dev = dt.start.device
        prep = torch.empty(max(dt.n, 1), dtype=torch.int64, device=dev)
        call = torch.empty(max(dt.n, 1), dtype=torch.int64, device=dev)

        def go(scratch, sbytes):
            return lib.chopper_launch_split(
                ctypes.byref(self._rec), self.clocks, _ptr(launch_ns),
                _ptr(self.start), _ptr(self.gap), _ptr(prep), _ptr(call),
                scratch, sbytes, _ptr(self.status), _stream())
        if "launch" not in self._scr:
            self._scr["launch"] = _scratch(go, dev)
        scr, sb = _aligned(self._scr["launch"])
        _check(go(scr, ctypes.byref(sb)), "launch_split")
        return prep[:dt.n], call[:dt.n]

    def launch_split_noalloc(self, launch_ns: torch.Tensor, prep=None,
                             call=None):
        """chopper_launch_split_noalloc: the same split without scratch (the
        library's static device table); writes into prep / call when given,
        else into new tensors, and returns them."""
        dt = self.dt
        dev = dt.start.device
        if prep is None:
            prep = torch.empty(max(dt.n, 1), dtype=torch.int64, device=dev)
        if call is None:
            call = torch.empty(max(dt.n, 1), dtype=torch.int64, device=dev)
        _check(lib.chopper_launch_split_noalloc(
            ctypes.byref(self._rec), self.clocks, _ptr(launch_ns),
            _ptr(self.start), _ptr(self.gap), _ptr(prep), _ptr(call),
            _ptr(self.status), _stream()), "launch_split_noalloc")
        return prep[:dt.n], call[:dt.n]

    def op_stats(self, phase_level: int = 1, op_level: int = 3,
                 n_phases: int = 3, n_ops: int = 64,
                 freq_peak_mhz: float = 2100.0, tpt_peak: float = 1.0,
                 f_gemm=None, per_gpu: bool = False):
        """Overlap statistics and overhead breakdown per (phase, operation)
        from the aggregated rows (chopper_op_stats); returns device tensors
        out [17][n_phases * n_ops] and cnt [n_phases * n_ops], and with
        per_gpu also the per-GPU overlap CDFs gout [9][n_phases * n_ops *
        n_gpus] and gcnt [n_phases * n_ops * n_gpus]."""
        dt = self.dt
        dev = dt.start.device
        G = n_phases * n_ops
        NG = dt.n_gpus
        out = torch.empty(17, G, dtype=torch.float64, device=dev)
        cnt = torch.empty(G, dtype=torch.int64, device=dev)
        gout = torch.empty(9, G * NG, dtype=torch.float64, device=dev)
        gcnt = torch.empty(G * NG, dtype=torch.int64, device=dev)
        fg = None
        if f_gemm is not None:
            fg = (ctypes.c_double * n_ops)(*[float(v) for v in f_gemm])
        spec = StatsSpec(phase_level, op_level, n_phases, n_ops,
                         float(freq_peak_mhz), float(tpt_peak),
                         ctypes.cast(fg, ctypes.POINTER(ctypes.c_double))
                         if fg is not None else None, NG, 0)
        rows = self.rows.struct()

        def go(scratch, sbytes):
            return lib.chopper_op_stats(
                ctypes.byref(rows), dt.depth, dt.n_counters,
                ctypes.byref(self._mk), ctypes.byref(spec), _ptr(out),
                _ptr(cnt), _ptr(gout), _ptr(gcnt), scratch, sbytes,
                _ptr(self.status), _stream())
        if "stats" not in self._scr:
            self._scr["stats"] = _scratch(go, dev)
        scr, sb = _aligned(self._scr["stats"])
        _check(go(scr, ctypes.byref(sb)), "op_stats")
        if per_gpu:
            return out, cnt, gout, gcnt
        return out, cnt

    def join_counters(self, passes, iter_level: int = 0):
        """Counters of serialized profiling passes matched to the records
        (chopper_join_counters).  passes: dicts of device tensors gpu,
        stream, cls (u8), label (i32 holding u32), values ([c][m] i64
        holding u64) and the list dst of destination columns.  Returns
        (counters [16][n], matched [n]) device tensors.  Needs align and
        attribute to have run."""
        dt = self.dt
        dev = dt.start.device
        n = dt.n
        arr = (CounterPass * max(len(passes), 1))()
        for i, q in enumerate(passes):
            c = arr[i]
            c.n = int(q["gpu"].numel())
            c.n_cols = len(q["dst"])
            c.gpu, c.stream, c.cls = _ptr(q["gpu"]), _ptr(q["stream"]), \
                _ptr(q["cls"])
            c.label, c.values = _ptr(q["label"]), _ptr(q["values"])
            for j, d in enumerate(q["dst"]):
                c.dst[j] = int(d)
        ctr = torch.empty(16, max(n, 1), dtype=torch.int64, device=dev)
        matched = torch.empty(max(n, 1), dtype=torch.uint8, device=dev)

        def go(scratch, sbytes):
            return lib.chopper_join_counters(
                ctypes.byref(self._rec), _ptr(self.start), _ptr(self.order),
                _ptr(self.idx), dt.depth, iter_level, ctypes.byref(self._mk),
                arr, len(passes), _ptr(ctr), _ptr(matched), scratch, sbytes,
                _ptr(self.status), _stream())
        scr = _scratch(go, dev)
        a, sb = _aligned(scr)
        _check(go(a, ctypes.byref(sb)), "join_counters")
        return ctr[:, :n], matched[:n]

    def step(self):
        """One pass of the whole pipeline.  Attribution and the overlap
        queries both need only the aligned times, orders and markers, so the
        overlap call goes on a second stream (default priority) beside the
        attribution on the caller's.  The aggregation is queued after the
        attribution with the event recorded after the overlap call, which
        only its passes that read gap and ovl wait for, so the records
        reduction starts once both streams are done and has the GPU to
        itself; the ratios and the window fractions follow on the caller's
        stream.  Traces below 2^20 records run the calls in sequence on the
        caller's stream: there the waits between streams cost about as much
        as the work they let overlap."""
        if self.dt.n < (1 << 20):
            self.align()
            self.attribute()
            self.overlap()
            self.aggregate()
            self.derive()
            return
        main = torch.cuda.current_stream()
        if getattr(self, "_side", None) is None:
            self._side = torch.cuda.Stream(device=main.device)
            self._ov_done = torch.cuda.Event()
        self.align()
        self._side.wait_stream(main)
        try:
            with torch.cuda.stream(self._side):
                self.overlap()
                self._ov_done.record(self._side)
            self.attribute()
            self._ready = self._ov_done
            self.aggregate()
        finally:
            # (also when a call failed: nothing later on the caller's stream
            # may run beside the second stream's work)
            self._ready = None
            main.wait_stream(self._side)
        self.derive_rows()
        self.derive_windows()

    def results(self) -> Dict:
        torch.cuda.synchronize()
        n, nm, D = self.dt.n, self.dt.n_markers, self.dt.depth
        u = lambda t, dt_: t.cpu().numpy().view(dt_)
        rows = self.rows.to_numpy()
        nr = rows["n_rows"]
        return dict(
            x0=np.array([c.x0 for c in self.clocks], np.int64),
            c=np.array([c.c for c in self.clocks], np.int64),
            d=np.array([c.d_q48 for c in self.clocks], np.int64),
            start=u(self.start[:n], np.int64), end=u(self.end[:n], np.int64),
            mstart=u(self.mstart[:nm], np.int64),
            mend=u(self.mend[:nm], np.int64),
            order=u(self.order[:n], np.uint32),
            korder=u(self.korder[:n], np.uint32),
            idx=u(self.idx[:, :n], np.uint32).reshape(D, n),
            ovl=u(self.ovl[:n], np.int64), gap=u(self.gap[:n], np.int64),
            mwin=u(self.mwin[:nm], np.int64).reshape(nm, 4),
            gwin=u(self.gwin, np.int64),
            rows=rows,
            ratios=u(self.ratios[:, :nr], np.float64).reshape(6, nr),
            wfrac=u(self.wfrac[:nm], np.float64).reshape(nm, 4),
            status=int(self.status.item()) & 0xFFFFFFFF)


class Views:
    """Re-keyed views of a Pipeline's run (chopper_views): per (iteration
    unit, phase, class) and (unit, phase, operation, kind) sums, busy time
    per unit, its maximum per iteration, and medians over the units."""

    def __init__(self, pipe: Pipeline, iter_level: int = 0,
                 phase_level: int = 1, op_level: int = 3, n_phases: int = 3,
                 n_ops: int = 64, n_iters: int = 1, warmup: int = 0):
        self.pipe = pipe
        dt = pipe.dt
        dev = dt.start.device
        self.spec = ViewSpec(iter_level, phase_level, op_level, n_phases,
                             n_ops, n_iters, warmup, 0)
        U = int((dt.m_level == iter_level).sum().item()) if dt.n_markers else 0
        Pn, O, NI = n_phases, n_ops, n_iters
        e = lambda n, dt_: torch.empty(max(n, 1), dtype=dt_, device=dev)
        self.U, self.P, self.O, self.NI = U, Pn, O, NI
        self.t = dict(
            n_units=e(1, torch.int64), unit_marker=e(U, torch.int32),
            cls_tab=e(3 * U * Pn * 8, torch.int64),
            op_tab=e(4 * U * Pn * O * 2, torch.int64),
            busy=e(U, torch.int64), iter_max=e(NI, torch.int64),
            cls_med=e(3 * Pn * 8, torch.float64),
            cls_cnt=e(Pn * 8, torch.int64),
            op_med=e(3 * Pn * O * 2, torch.float64),
            op_cnt=e(Pn * O * 2, torch.int64),
            iter_med=e(1, torch.float64), iter_cnt=e(1, torch.int64))
        self.out = ViewOut()
        self.out.unit_cap = U
        for k in _VIEW_OUT:
            setattr(self.out, k, _ptr(self.t[k]))
        self._scr = _scratch(lambda s, b: self._call(s, b), dev)

    def _call(self, scratch, sbytes):
        pp, dt = self.pipe, self.pipe.dt
        rows = pp.rows.struct()
        self._rows = rows
        return lib.chopper_views(
            ctypes.byref(pp._rec), _ptr(pp.start), _ptr(pp.end), _ptr(pp.idx),
            dt.depth, _ptr(pp.gap), ctypes.byref(pp._mk), ctypes.byref(rows),
            ctypes.byref(self.spec), ctypes.byref(self.out), scratch, sbytes,
            _ptr(pp.status), _stream())

    def run(self):
        scr, sb = _aligned(self._scr)
        _check(self._call(scr, ctypes.byref(sb)), "views")

    def results(self) -> Dict:
        torch.cuda.synchronize()
        U, Pn, O, NI = self.U, self.P, self.O, self.NI
        u = lambda k, n, dt_: self.t[k][:n].cpu().numpy().view(dt_)
        return dict(
            n_units=int(self.t["n_units"][0].item()),
            unit_marker=u("unit_marker", U, np.uint32),
            cls_tab=u("cls_tab", 3 * U * Pn * 8, np.uint64).reshape(3, -1),
            op_tab=u("op_tab", 4 * U * Pn * O * 2, np.uint64).reshape(4, -1),
            busy=u("busy", U, np.int64), iter_max=u("iter_max", NI, np.int64),
            cls_med=u("cls_med", 3 * Pn * 8, np.float64).reshape(3, -1),
            cls_cnt=u("cls_cnt", Pn * 8, np.int64),
            op_med=u("op_med", 3 * Pn * O * 2, np.float64).reshape(3, -1),
            op_cnt=u("op_cnt", Pn * O * 2, np.int64),
            iter_med=float(self.t["iter_med"][0].item()),
            iter_cnt=int(self.t["iter_cnt"][0].item()))
