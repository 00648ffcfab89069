"""The C ABI without a GPU: the library loads, exports every function the
header declares, answers scratch-size queries and rejects bad arguments on
the host before any GPU work."""
import ctypes
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "chopper.h")
LIB = os.path.join(ROOT, "paper_2512_08242_amd", "libchopper.so")


def declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(chopper_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def ch():
    if not os.path.exists(LIB):
        import __graft_entry__
        __graft_entry__.build()
    import paper_2512_08242_amd as m
    return m


def test_header_declares_the_four_steps():
    names = declared()
    for n in ("chopper_align", "chopper_attribute", "chopper_overlap",
              "chopper_aggregate", "chopper_ratios",
              "chopper_window_fractions", "chopper_strerror",
              "chopper_version", "chopper_time_kernel", "chopper_kernel_name",
              "chopper_views", "chopper_launch_split",
              "chopper_join_counters", "chopper_op_stats"):
        assert n in names


def test_library_exports_every_declared_symbol(ch):
    lib = ctypes.CDLL(LIB)
    for name in declared():
        assert hasattr(lib, name), name


def test_strerror_and_version(ch):
    lib = ch.lib
    assert lib.chopper_strerror(0) == b"ok"
    assert lib.chopper_strerror(-2) == b"scratch buffer too small"
    assert lib.chopper_version() >= 100


def _records(ch, n=10, n_gpus=2, n_counters=0):
    r = ch.binding.Records()
    r.n, r.n_gpus, r.n_counters = n, n_gpus, n_counters
    fake = ctypes.c_void_p(0x1000)   # never dereferenced by a size query
    for f in ("gpu", "stream", "cls", "op_id", "start_ns", "end_ns"):
        setattr(r, f, fake)
    r.counters = fake if n_counters else None
    return r


def _markers(ch, n=5, depth=3):
    m = ch.binding.Markers()
    m.n, m.depth = n, depth
    fake = ctypes.c_void_p(0x1000)
    for f in ("gpu", "level", "start_ns", "end_ns", "label"):
        setattr(m, f, fake)
    return m


def test_scratch_queries_need_no_gpu(ch):
    lib, b = ch.lib, ch.binding
    fake = ctypes.c_void_p(0x1000)
    rec, mk = _records(ch, 1000), _markers(ch, 300)
    sz = ctypes.c_size_t(0)
    clocks = (b.Clock * 2)()
    rc = lib.chopper_align(ctypes.byref(rec), ctypes.byref(mk), None, clocks,
                           fake, fake, fake, fake, fake, fake, None,
                           ctypes.byref(sz), None, None)
    assert rc == 0 and sz.value > 1000 * 8
    small = sz.value
    rec2 = _records(ch, 100000)
    rc = lib.chopper_align(ctypes.byref(rec2), ctypes.byref(mk), None, clocks,
                           fake, fake, fake, fake, fake, fake, None,
                           ctypes.byref(sz), None, None)
    assert rc == 0 and sz.value > small
    for call in (
        lambda: lib.chopper_attribute(ctypes.byref(rec), fake,
                                      ctypes.byref(mk), fake, fake, fake,
                                      None, ctypes.byref(sz), None, None),
        lambda: lib.chopper_overlap(ctypes.byref(rec), fake, fake, fake, fake,
                                    ctypes.byref(mk), fake, fake, fake, fake,
                                    fake, fake, None, ctypes.byref(sz), None,
                                    None),
    ):
        sz.value = 0
        assert call() == 0 and sz.value > 0
    rows = b.Rows()
    rows.cap = 0
    rows.level_offset = fake
    sz.value = 0
    assert lib.chopper_aggregate(ctypes.byref(rec), fake, fake, fake, fake, 3,
                                 fake, fake, ctypes.byref(mk), 255, None,
                                 ctypes.byref(rows), None, ctypes.byref(sz),
                                 None, None, None) == 0
    assert sz.value > 0


def test_argument_errors_are_synchronous(ch):
    lib, b = ch.lib, ch.binding
    fake = ctypes.c_void_p(0x1000)
    sz = ctypes.c_size_t(0)
    clocks = (b.Clock * 2)()
    EINVAL, ESCRATCH = -1, -2
    bad = _records(ch, 10)
    bad.n = -1
    assert lib.chopper_align(ctypes.byref(bad), None, None, clocks, fake,
                             fake, None, None, fake, fake, None,
                             ctypes.byref(sz), None, None) == EINVAL
    bad = _records(ch, 10, n_gpus=0)
    assert lib.chopper_align(ctypes.byref(bad), None, None, clocks, fake,
                             fake, None, None, fake, fake, None,
                             ctypes.byref(sz), None, None) == EINVAL
    bad = _records(ch, 10, n_counters=17)
    assert lib.chopper_align(ctypes.byref(bad), None, None, clocks, fake,
                             fake, None, None, fake, fake, None,
                             ctypes.byref(sz), None, None) == EINVAL
    rec = _records(ch, 10)
    mk = _markers(ch, 5, depth=9)
    assert lib.chopper_attribute(ctypes.byref(rec), fake, ctypes.byref(mk),
                                 fake, fake, fake, None, ctypes.byref(sz),
                                 None, None) == EINVAL
    # missing output pointer
    mk = _markers(ch, 5, depth=3)
    assert lib.chopper_attribute(ctypes.byref(rec), fake, ctypes.byref(mk),
                                 fake, fake, None, None, ctypes.byref(sz),
                                 None, None) == EINVAL
    # a scratch smaller than required
    sz.value = 0
    assert lib.chopper_attribute(ctypes.byref(rec), fake, ctypes.byref(mk),
                                 fake, fake, fake, None, ctypes.byref(sz),
                                 None, None) == 0
    need = sz.value
    small = ctypes.c_size_t(need - 1)
    assert lib.chopper_attribute(ctypes.byref(rec), fake, ctypes.byref(mk),
                                 fake, fake, fake, ctypes.c_void_p(0x100000),
                                 ctypes.byref(small), fake, None) == ESCRATCH
    # misaligned scratch
    big = ctypes.c_size_t(need + 1024)
    assert lib.chopper_attribute(ctypes.byref(rec), fake, ctypes.byref(mk),
                                 fake, fake, fake, ctypes.c_void_p(0x100001),
                                 ctypes.byref(big), fake, None) == EINVAL
    # unknown aggregation level, depth mismatch
    rows = b.Rows()
    rows.cap = 0
    rows.level_offset = fake
    for lvl, depth in ((7, 3), (99, 3), (255, 2)):
        assert lib.chopper_aggregate(ctypes.byref(rec), fake, fake, fake,
                                     fake, depth, fake, fake,
                                     ctypes.byref(mk), lvl, None,
                                     ctypes.byref(rows), None,
                                     ctypes.byref(sz), None, None,
                                     None) == EINVAL
    # time hook: unknown kernel name
    assert lib.chopper_time_kernel(b"no_such_kernel", fake, fake) == EINVAL
    assert lib.chopper_time_kernel(None, None, None) == 0


def test_anchor_errors_are_reported_before_gpu_work(ch):
    lib, b = ch.lib, ch.binding
    fake = ctypes.c_void_p(0x1000)
    clocks = (b.Clock * 1)()
    rec = _records(ch, 0, n_gpus=1)
    # gpu index of an anchor beyond n_gpus
    g = np.array([3], np.uint8)
    x = np.array([0], np.int64)
    a = b.Anchors()
    a.n = 1
    a.gpu = g.ctypes.data_as(ctypes.c_void_p)
    a.local_ns = x.ctypes.data_as(ctypes.c_void_p)
    a.ref_ns = x.ctypes.data_as(ctypes.c_void_p)
    sz = ctypes.c_size_t(0)
    assert lib.chopper_align(ctypes.byref(rec), None, ctypes.byref(a), clocks,
                             None, None, None, None, None, None, None,
                             ctypes.byref(sz), None, None) == 0
    status = ctypes.c_void_p(0x2000)
    rc = lib.chopper_align(ctypes.byref(rec), None, ctypes.byref(a), clocks,
                           None, None, None, None, None, None,
                           ctypes.c_void_p(0x100000), ctypes.byref(sz), status,
                           None)
    assert rc == -1
    # a slope beyond the Q48 range
    g = np.array([0, 0], np.uint8)
    x = np.array([0, 10**9], np.int64)
    y = np.array([0, 10**9 + 10**7], np.int64)
    a.n = 2
    a.gpu = g.ctypes.data_as(ctypes.c_void_p)
    a.local_ns = x.ctypes.data_as(ctypes.c_void_p)
    a.ref_ns = y.ctypes.data_as(ctypes.c_void_p)
    rc = lib.chopper_align(ctypes.byref(rec), None, ctypes.byref(a), clocks,
                           None, None, None, None, None, None,
                           ctypes.c_void_p(0x100000), ctypes.byref(sz), status,
                           None)
    assert rc == -3


def test_views_scratch_query_and_argument_errors(ch):
    """chopper_views answers the scratch query without GPU work and rejects
    bad specs synchronously."""
    lib, b = ch.lib, ch.binding
    fake = ctypes.c_void_p(0x1000)
    rec = b.Records()
    rec.n, rec.n_gpus, rec.n_counters = 1000, 2, 0
    rec.gpu = rec.stream = rec.cls = rec.start_ns = rec.end_ns = fake
    mk = b.Markers()
    mk.n, mk.depth = 500, 4
    mk.gpu = mk.level = mk.start_ns = mk.end_ns = mk.label = fake
    rows = b.Rows()
    rows.cap = 10
    for k in ("level_offset", "path", "gpu", "kind", "n", "dur", "gap", "ovl",
              "tmin", "tmax", "first"):
        setattr(rows, k, fake)
    out = b.ViewOut()
    out.unit_cap = 16
    for k in b._VIEW_OUT:
        setattr(out, k, fake)

    def call(spec, out_=out, scratch=None):
        sz = ctypes.c_size_t(0)
        rc = lib.chopper_views(ctypes.byref(rec), fake, fake, fake, 4, fake,
                               ctypes.byref(mk), ctypes.byref(rows),
                               ctypes.byref(spec), ctypes.byref(out_),
                               scratch, ctypes.byref(sz), None, None)
        return rc, sz.value

    good = b.ViewSpec(0, 1, 3, 3, 64, 10, 0, 0)
    rc, sz = call(good)
    assert rc == 0 and sz > 0
    for bad in (b.ViewSpec(0, 1, 4, 3, 64, 10, 0, 0),    # level >= depth
                b.ViewSpec(-1, 1, 3, 3, 64, 10, 0, 0),
                b.ViewSpec(0, 1, 3, 0, 64, 10, 0, 0),    # no phase
                b.ViewSpec(0, 1, 3, 17, 64, 10, 0, 0),   # > 16 phases
                b.ViewSpec(0, 1, 3, 3, 129, 10, 0, 0),   # > 128 operations
                b.ViewSpec(0, 1, 3, 3, 64, -1, 0, 0)):
        assert call(bad)[0] == -1
    o2 = b.ViewOut()
    o2.unit_cap = 16
    for k in b._VIEW_OUT:
        setattr(o2, k, fake)
    o2.op_med = None
    assert call(good, o2)[0] == -1
    # too small a scratch buffer
    sz = ctypes.c_size_t(8)
    assert lib.chopper_views(ctypes.byref(rec), fake, fake, fake, 4, fake,
                             ctypes.byref(mk), ctypes.byref(rows),
                             ctypes.byref(good), ctypes.byref(out),
                             ctypes.c_void_p(0x10000), ctypes.byref(sz), fake,
                             None) == -2


def test_launch_split_scratch_query_and_argument_errors(ch):
    lib, b = ch.lib, ch.binding
    fake = ctypes.c_void_p(0x1000)
    rec = _records(ch, 1000)
    clocks = (b.Clock * 2)()
    sz = ctypes.c_size_t(0)
    assert lib.chopper_launch_split(ctypes.byref(rec), clocks, fake, fake,
                                    fake, fake, fake, None, ctypes.byref(sz),
                                    None, None) == 0
    assert sz.value > 0
    for args in ((None, fake), (fake, None)):
        assert lib.chopper_launch_split(ctypes.byref(rec), clocks, args[0],
                                        fake, fake, fake, args[1], None,
                                        ctypes.byref(sz), None, None) == -1
    assert lib.chopper_launch_split(ctypes.byref(rec), None, fake, fake, fake,
                                    fake, fake, None, ctypes.byref(sz), None,
                                    None) == -1


def test_launch_split_noalloc_argument_errors(ch):
    """The allocation-free variant rejects missing pointers synchronously,
    before any HIP call (no GPU here)."""
    lib, b = ch.lib, ch.binding
    fake = ctypes.c_void_p(0x1000)
    rec = _records(ch, 1000)
    clocks = (b.Clock * 2)()
    for i in range(6):
        args = [fake] * 6
        args[i] = None
        assert lib.chopper_launch_split_noalloc(
            ctypes.byref(rec), clocks, *args[:5], fake if i < 5 else None,
            None) == -1, i
    assert lib.chopper_launch_split_noalloc(ctypes.byref(rec), None, fake,
                                            fake, fake, fake, fake, fake,
                                            None) == -1
    rec.n_gpus = 257
    assert lib.chopper_launch_split_noalloc(ctypes.byref(rec), clocks, fake,
                                            fake, fake, fake, fake, fake,
                                            None) == -1


def test_op_stats_scratch_query_and_argument_errors(ch):
    """chopper_op_stats answers the scratch query without GPU work, sizes
    its scratch from the row capacity, and rejects bad specs synchronously."""
    lib, b = ch.lib, ch.binding
    fake = ctypes.c_void_p(0x1000)
    mk = b.Markers()
    mk.n, mk.depth = 500, 4
    mk.gpu = mk.level = mk.start_ns = mk.end_ns = mk.label = fake
    rows = b.Rows()
    rows.cap = 10
    for k in ("level_offset", "path", "gpu", "kind", "n", "dur", "gap", "ovl",
              "tmin", "tmax", "first", "ctr"):
        setattr(rows, k, fake)

    def call(spec, depth=4, nc=16, out=fake, cap=10):
        rows.cap = cap
        sz = ctypes.c_size_t(0)
        rc = lib.chopper_op_stats(ctypes.byref(rows), depth, nc,
                                  ctypes.byref(mk), ctypes.byref(spec), out,
                                  fake, None, None, None, ctypes.byref(sz),
                                  None, None)
        return rc, sz.value

    def spec(*a, n_gpus=8):
        return b.StatsSpec(*a, None, n_gpus, 0)

    good = spec(1, 3, 3, 64, 2100.0, 1.0)
    rc, sz = call(good)
    assert rc == 0 and sz > 0
    rc2, sz2 = call(good, cap=10**6)
    assert rc2 == 0 and sz2 > sz + 4 * 10**6
    # the per-GPU CDF tables grow with the GPUs
    rc3, sz3 = call(spec(1, 3, 3, 64, 2100.0, 1.0, n_gpus=256))
    assert rc3 == 0 and sz3 > sz
    for bad in (spec(1, 4, 3, 64, 2100.0, 1.0),   # level >= depth
                spec(-1, 3, 3, 64, 2100.0, 1.0),
                spec(1, 3, 0, 64, 2100.0, 1.0),   # no phase
                spec(1, 3, 17, 64, 2100.0, 1.0),  # > 16 phases
                spec(1, 3, 3, 0, 2100.0, 1.0),
                spec(1, 3, 3, 129, 2100.0, 1.0),  # > 128 ops
                spec(1, 3, 3, 64, 2100.0, 1.0, n_gpus=0),
                spec(1, 3, 3, 64, 2100.0, 1.0, n_gpus=257)):
        assert call(bad)[0] == -1
    assert call(good, depth=5)[0] == -1          # deeper than the markers
    assert call(good, nc=17)[0] == -1
    assert call(good, out=None)[0] == -1
    sz = ctypes.c_size_t(8)
    assert lib.chopper_op_stats(ctypes.byref(rows), 4, 16, ctypes.byref(mk),
                                ctypes.byref(good), fake, fake, None, None,
                                ctypes.c_void_p(0x10000), ctypes.byref(sz),
                                fake, None) == -2
