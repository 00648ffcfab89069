"""Parity of the HIP pipeline with the CPU oracle, element by element, through
the C ABI.  Integer outputs must be bit-exact; derived doubles must be equal
(NaN matching NaN), which is within the 1e-12 relative tolerance required for
them since both sides perform the same IEEE operations."""
import dataclasses
import sys

import numpy as np
import pytest

import oracle
import tracegen as tg

pytestmark = pytest.mark.gpu

REC_KEYS = ("start", "end", "mstart", "mend", "order", "korder", "idx", "ovl",
            "gap", "mwin", "gwin")
ROW_KEYS = ("path", "gpu", "kind", "n", "dur", "gap", "ovl", "tmin", "tmax",
            "first", "ctr")


@pytest.fixture(scope="module")
def ch():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    import paper_2512_08242_amd as m
    return m


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def run_gpu(ch, tr, level=255, filt=None):
    pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"), level=level, filt=filt)
    pipe.status.zero_()
    pipe.step()
    return pipe.results()


def assert_same_float(a, b, what):
    a, b = np.asarray(a), np.asarray(b)
    assert a.shape == b.shape, what
    same = (a == b) | (np.isnan(a) & np.isnan(b))
    if not same.all():
        i = np.nonzero(~same.reshape(-1))[0][0]
        raise AssertionError(f"{what}: first difference at {i}: "
                             f"{a.reshape(-1)[i]!r} vs {b.reshape(-1)[i]!r}")


def assert_parity(got, ref, rows=True, name=""):
    assert got["status"] == ref["status"], (name, got["status"], ref["status"])
    for k in ("x0", "c", "d"):
        assert np.array_equal(got[k], ref[k]), (name, k)
    for k in REC_KEYS:
        g, r = np.asarray(got[k]), np.asarray(ref[k])
        assert g.shape == r.shape, (name, k, g.shape, r.shape)
        if not np.array_equal(g, r):
            diff = np.nonzero((g != r).reshape(-1))[0]
            raise AssertionError(f"{name}: {k}: {diff.size} differences, "
                                 f"first at {diff[0]}: {g.reshape(-1)[diff[0]]} "
                                 f"vs {r.reshape(-1)[diff[0]]}")
    if not rows:
        return
    gr, rr = got["rows"], ref["rows"]
    assert np.array_equal(gr["level_offset"], rr["level_offset"]), (
        name, gr["level_offset"], rr["level_offset"])
    for k in ROW_KEYS:
        if not np.array_equal(gr[k], rr[k]):
            diff = np.nonzero((np.asarray(gr[k]) != np.asarray(rr[k])
                               ).reshape(-1))[0]
            raise AssertionError(f"{name}: rows.{k}: {diff.size} differences,"
                                 f" first at {diff[0]}")
    assert_same_float(got["ratios"], ref["ratios"], f"{name}: ratios")
    assert_same_float(got["wfrac"], ref["wfrac"], f"{name}: window fractions")


MICRO = [dict(n_gpus=1, n_kernels=40, n_streams=1, depth=2),
         dict(n_gpus=2, n_kernels=120, n_streams=3, depth=3, n_counters=16,
              anchors=5),
         dict(n_gpus=3, n_kernels=300, n_streams=4, depth=4, n_counters=3,
              anchors=2),
         dict(n_gpus=4, n_kernels=600, n_streams=2, depth=5, n_counters=16,
              anchors=8, mixed_stream_kinds=False),
         dict(n_gpus=2, n_kernels=5000, n_streams=3, depth=4, n_counters=16,
              anchors=9, span=60000)]


@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("shape", range(len(MICRO)))
def test_micro_nested(ch, seed, shape):
    tr = tg.make_micro(seed * 7 + shape, **MICRO[shape])
    say("micro nested", seed, shape, tr.n, tr.n_markers)
    ref = oracle.run(tr)
    assert not ref["status"] & oracle.PATH_CONFLICT
    assert_parity(run_gpu(ch, tr), ref, name=tr.name)


@pytest.mark.parametrize("seed", range(8))
def test_micro_unnested(ch, seed):
    """Arbitrary marker intervals: attribution, overlap and the rows of
    every level (grouped by the whole marker path) stay exact; PATH_CONFLICT
    is a warning."""
    tr = tg.make_micro(500 + seed, n_gpus=2, n_kernels=200, n_streams=3,
                       depth=3, nested=False, n_counters=2)
    say("micro unnested", seed)
    got, ref = run_gpu(ch, tr), oracle.run(tr)
    assert_parity(got, ref, name=tr.name)


def test_unnested_conflicts_are_exercised(ch):
    """Most of the un-nested micro traces really hold records that share
    their deepest marker but not their path, on both row paths (input in
    start order and shuffled), at single levels and with a filter."""
    hits = 0
    for seed in range(8):
        tr = tg.make_micro(500 + seed, n_gpus=2, n_kernels=200, n_streams=3,
                           depth=3, nested=False, n_counters=2)
        ref = oracle.run(tr)
        hits += bool(ref["status"] & oracle.PATH_CONFLICT)
    assert hits >= 4, hits
    tr = tg.make_micro(777, n_gpus=3, n_kernels=3000, n_streams=2, depth=4,
                       nested=False, n_counters=16, anchors=3)
    say("unnested, 3000 records")
    ref = oracle.run(tr)
    assert ref["status"] & oracle.PATH_CONFLICT
    assert_parity(run_gpu(ch, tr), ref, name="unnested 3000")
    for level in (0, 1, 3, 100):
        say("unnested level", level)
        assert_parity(run_gpu(ch, tr, level=level),
                      oracle.run(tr, level=level), name=f"unnested l{level}")
    f_or = oracle.make_filter(gpus=[0, 2], classes=[0, 2, 3, 5, 6])
    f_ch = ch.make_filter(gpus=[0, 2], classes=[0, 2, 3, 5, 6])
    say("unnested filter")
    assert_parity(run_gpu(ch, tr, filt=f_ch), oracle.run(tr, filt=f_or),
                  name="unnested filter")


@pytest.mark.parametrize("cid", [0, 1, 2])
def test_config_full_parity(ch, cid):
    tr = tg.make_config(cid)
    say("config", cid, tr.n, tr.n_markers)
    ref = oracle.run(tr)
    got = run_gpu(ch, tr)
    assert_parity(got, ref, name=f"config{cid}")


def _flat(res):
    out = {}
    for k, v in res.items():
        if isinstance(v, dict):
            for kk, vv in v.items():
                out[k + "." + kk] = vv
        else:
            out[k] = v
    return out


def test_two_stream_step_equals_calls_in_sequence(ch):
    # config 2 (2,457,600 records) takes the two-stream step; the same
    # calls one after the other on one stream must give the same bits
    tr = tg.make_config(2, with_truth=False)
    assert tr.n >= 1 << 20
    dt = ch.DeviceTrace(tr, "cuda")
    a = ch.Pipeline(dt)
    a.status.zero_()
    a.step()
    a.step()          # twice: the second reuses the streams and the event
    ra = _flat(a.results())
    b = ch.Pipeline(dt)
    b.status.zero_()
    b.align()
    b.attribute()
    b.overlap()
    b.aggregate()
    b.derive()
    rb = _flat(b.results())
    assert ra.keys() == rb.keys()
    for k in ra:
        x, y = ra[k], rb[k]
        if isinstance(x, np.ndarray) and x.dtype.kind == "f":
            assert_same_float(x, y, k)
        elif isinstance(x, np.ndarray):
            assert np.array_equal(x, y), k
        else:
            assert x == y, k


@pytest.mark.parametrize("level", [0, 1, 2, 100, 101])
def test_single_level_requests(ch, level):
    tr = tg.make_micro(77, n_gpus=3, n_kernels=400, depth=3, n_counters=4,
                       anchors=3)
    say("level", level)
    assert_parity(run_gpu(ch, tr, level=level), oracle.run(tr, level=level),
                  name=f"level{level}")


def test_filter(ch):
    tr = tg.make_config(0)
    say("filter")
    f_or = oracle.make_filter(gpus=[0], classes=[0, 1, 2, 5], iters=(1, 1))
    f_ch = ch.make_filter(gpus=[0], classes=[0, 1, 2, 5], iters=(1, 1))
    assert_parity(run_gpu(ch, tr, filt=f_ch), oracle.run(tr, filt=f_or),
                  name="filter")
    tr = tg.make_micro(12, n_gpus=3, n_kernels=300, depth=3, n_counters=2)
    f_or = oracle.make_filter(gpus=[0, 2], classes=[0, 3, 5, 6, 7])
    f_ch = ch.make_filter(gpus=[0, 2], classes=[0, 3, 5, 6, 7])
    assert_parity(run_gpu(ch, tr, filt=f_ch), oracle.run(tr, filt=f_or),
                  name="filter2")


# ---------------------------------------------------------------------------
# Input grouped by GPU and in start order inside each GPU (the order a
# profiler writes): the aggregation then reads the records in input order.
# ---------------------------------------------------------------------------
def natural_order(tr, gpu_map=None, n_gpus=None):
    """The records stably sorted by (gpu, start); optionally GPU ids renamed
    through gpu_map (records, markers and anchors alike)."""
    if gpu_map is not None:
        gm = np.asarray(gpu_map, np.uint8)
        tr = dataclasses.replace(tr, gpu=gm[tr.gpu], m_gpu=gm[tr.m_gpu],
                                 a_gpu=gm[tr.a_gpu], n_gpus=n_gpus)
    p = np.lexsort((tr.start, tr.gpu))
    return dataclasses.replace(
        tr, gpu=tr.gpu[p], stream=tr.stream[p], start=tr.start[p],
        end=tr.end[p], cls=tr.cls[p], op_id=tr.op_id[p],
        counters=None if tr.counters is None else tr.counters[:, p].copy(),
        name=tr.name + "/natural")


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("shape", range(len(MICRO)))
def test_natural_order_micro(ch, seed, shape):
    tr = natural_order(tg.make_micro(900 + seed * 7 + shape, **MICRO[shape]))
    say("natural micro", seed, shape, tr.n)
    assert_parity(run_gpu(ch, tr), oracle.run(tr), name=tr.name)


@pytest.mark.parametrize("seed", range(6))
def test_natural_order_unnested(ch, seed):
    """Arbitrary marker intervals with the records grouped by GPU in start
    order: the natural-tile heads pass must find the shared deepest markers
    of different paths (PATH_CONFLICT) and send the rows to the general
    path."""
    tr = natural_order(tg.make_micro(600 + seed, n_gpus=2, n_kernels=3000,
                                     n_streams=3, depth=3, nested=False,
                                     n_counters=2, span=30000))
    say("natural unnested", seed, tr.n)
    ref = oracle.run(tr)
    assert_parity(run_gpu(ch, tr), ref, name=tr.name)


@pytest.mark.parametrize("seed", range(4))
def test_natural_order_markers_shuffled(ch, seed):
    """Records grouped by GPU in start order, markers numbered in no order:
    the marker slots of a run do not increase, which the natural-tile heads
    pass must notice (the rows then come from the general path)."""
    tr = natural_order(tg.make_micro(620 + seed, n_gpus=2, n_kernels=3000,
                                     n_streams=2, depth=3, n_counters=2,
                                     span=30000))
    p = np.random.default_rng(seed).permutation(tr.n_markers)
    tr = dataclasses.replace(tr, m_gpu=tr.m_gpu[p], m_level=tr.m_level[p],
                             m_start=tr.m_start[p], m_end=tr.m_end[p],
                             m_label=tr.m_label[p], name=tr.name + "/mshuf")
    say("natural, markers shuffled", seed, tr.n, tr.n_markers)
    assert_parity(run_gpu(ch, tr), oracle.run(tr), name=tr.name)


@pytest.mark.parametrize("seed", range(3))
def test_natural_order_many_small_gpus(ch, seed):
    """Forty GPUs of about fifty records: most tiles hold several GPUs."""
    tr = natural_order(tg.make_micro(950 + seed, n_gpus=40, n_kernels=2000,
                                     n_streams=3, depth=3, n_counters=16,
                                     span=3000))
    say("natural many gpus", seed, tr.n)
    assert_parity(run_gpu(ch, tr), oracle.run(tr), name=tr.name)


def test_natural_order_sparse_gpu_ids(ch):
    """GPUs 1, 4 and 6 of 8 have records; the others none."""
    tr = natural_order(tg.make_micro(960, n_gpus=3, n_kernels=3000,
                                     n_streams=3, depth=4, n_counters=16,
                                     anchors=4, span=40000),
                       gpu_map=[1, 4, 6], n_gpus=8)
    say("natural sparse gpus", tr.n)
    assert_parity(run_gpu(ch, tr), oracle.run(tr), name=tr.name)


@pytest.mark.parametrize("level", [0, 2, 100])
def test_natural_order_single_level(ch, level):
    tr = natural_order(tg.make_micro(970, n_gpus=2, n_kernels=3000,
                                     depth=3, n_counters=4, span=30000))
    say("natural level", level)
    assert_parity(run_gpu(ch, tr, level=level), oracle.run(tr, level=level),
                  name=f"natural level{level}")


def test_natural_order_broken_inside_a_gpu(ch):
    """Two records of one GPU out of start order: the korder tiles apply."""
    tr = natural_order(tg.make_micro(980, n_gpus=2, n_kernels=3000,
                                     depth=3, n_counters=16, span=30000))
    g0 = np.nonzero(tr.gpu == tr.gpu[1000])[0]
    i = int(g0[g0 > 1000][0])
    j = next(int(k) for k in g0[g0 > i] if tr.start[k] != tr.start[i])
    for a in ("gpu", "stream", "start", "end", "cls", "op_id"):
        v = getattr(tr, a)
        v[[i, j]] = v[[j, i]]
    tr.counters[:, [i, j]] = tr.counters[:, [j, i]]
    say("natural broken", i, j)
    assert_parity(run_gpu(ch, tr), oracle.run(tr), name="natural broken")


def _tiny(n, m=3, G=1, depth=2, overlapping=False):
    """n records in [0, 1000) on one GPU; markers: one level-0 marker over
    everything and m - 1 level-1 markers tiling it (nested), or m markers of
    alternating levels and length 700 every 300 ns (overlapping)."""
    rng = np.random.default_rng(n)
    s = np.sort(rng.integers(0, 1000, size=n)).astype(np.int64)
    if overlapping:
        lev = (np.arange(m) % depth).astype(np.uint8)
        ms = np.arange(m, dtype=np.int64) * 300
        me = ms + 700
    elif m > 0:
        cuts = np.linspace(0, 1000, m).astype(np.int64)
        lev = np.array([0] + [1] * (m - 1), np.uint8)
        ms = np.concatenate([[0], cuts[:-1]]).astype(np.int64)
        me = np.concatenate([[1000], cuts[1:]]).astype(np.int64)
    else:
        lev, ms, me = (np.zeros(0, np.uint8), np.zeros(0, np.int64),
                       np.zeros(0, np.int64))
    return tg.Trace(
        n_gpus=G, depth=depth, gpu=np.zeros(n, np.uint8),
        stream=(np.arange(n) % 2).astype(np.uint8), start=s,
        end=s + rng.integers(0, 50, size=n), cls=(np.arange(n) % 7
                                                   ).astype(np.uint8),
        op_id=np.zeros(n, np.uint32), counters=None,
        m_gpu=np.zeros(m, np.uint8), m_level=lev, m_start=ms, m_end=me,
        m_label=np.arange(m, dtype=np.uint32), a_gpu=np.zeros(0, np.uint8),
        a_local=np.zeros(0, np.int64), a_ref=np.zeros(0, np.int64),
        name=f"tiny{n}")


def test_union_carry_over_many_chunks(ch):
    # The first record of the trace runs over everything after it, so the
    # second 2048-record tile of the union runs is corrected for that
    # carry item by item.  In that tile a long record (ending before the
    # carry) is followed by short ones: the running end of the tile's items
    # must keep the long record's end across every 64-item chunk after it.
    T = 2048
    s = np.concatenate([[0], 10 * np.arange(1, T), [30000],
                        30000 + 10 * np.arange(1, T)]).astype(np.int64)
    e = s + 5
    e[0] = 10 ** 9
    e[T] = 5 * 10 ** 8
    cs = (100 + 3000 * np.arange(8)).astype(np.int64)      # comm records
    n = 2 * T + 8
    start = np.concatenate([s, cs])
    end = np.concatenate([e, cs + 1000])
    cls = np.concatenate([np.zeros(2 * T, np.uint8), np.full(8, 5, np.uint8)])
    stream = np.concatenate([np.zeros(2 * T, np.uint8), np.ones(8, np.uint8)])
    tr = tg.Trace(
        n_gpus=1, depth=2, gpu=np.zeros(n, np.uint8), stream=stream,
        start=start, end=end, cls=cls, op_id=np.zeros(n, np.uint32),
        counters=None, m_gpu=np.zeros(3, np.uint8),
        m_level=np.array([0, 1, 1], np.uint8),
        m_start=np.array([0, 0, 25000], np.int64),
        m_end=np.array([2 * 10 ** 9, 25000, 2 * 10 ** 9], np.int64),
        m_label=np.arange(3, dtype=np.uint32), a_gpu=np.zeros(0, np.uint8),
        a_local=np.zeros(0, np.int64), a_ref=np.zeros(0, np.int64),
        name="carry over chunks")
    say("union carry over many chunks")
    assert_parity(run_gpu(ch, tr), oracle.run(tr), name=tr.name)


@pytest.mark.parametrize("seed", range(4))
def test_union_runs_heavy_tails(ch, seed):
    # several 2048-record tiles of two GPUs, starts dense, durations mostly
    # short with rare ones reaching thousands of records ahead: tiles whose
    # carry covers many chunks, with chunk maxima that go up and down
    rng = np.random.default_rng(4000 + seed)
    n = 7000 + 500 * seed
    gpu = np.sort(rng.integers(0, 2, size=n)).astype(np.uint8)
    start = np.zeros(n, np.int64)
    for g in (0, 1):
        k = int((gpu == g).sum())
        start[gpu == g] = np.sort(rng.integers(0, 20 * k, size=k))
    dur = rng.integers(0, 40, size=n).astype(np.int64)
    big = rng.random(n) < 0.004
    dur[big] = rng.integers(1000, 60000, size=int(big.sum()))
    cls = np.where(rng.random(n) < 0.1, 5, 0).astype(np.uint8)
    stream = np.where(cls == 5, 2, rng.integers(0, 2, size=n)).astype(np.uint8)
    ms = np.array([0, 0, 0, 0], np.int64)
    me = np.array([10 ** 7, 50000, 10 ** 7, 50000], np.int64)
    tr = tg.Trace(
        n_gpus=2, depth=2, gpu=gpu, stream=stream, start=start,
        end=start + dur, cls=cls, op_id=np.zeros(n, np.uint32),
        counters=None, m_gpu=np.array([0, 0, 1, 1], np.uint8),
        m_level=np.array([0, 1, 0, 1], np.uint8), m_start=ms, m_end=me,
        m_label=np.arange(4, dtype=np.uint32), a_gpu=np.zeros(0, np.uint8),
        a_local=np.zeros(0, np.int64), a_ref=np.zeros(0, np.int64),
        name=f"heavy tails {seed}")
    say("union runs heavy tails", seed, n)
    assert_parity(run_gpu(ch, tr), oracle.run(tr), name=tr.name)


@pytest.mark.parametrize("seed", range(3))
def test_attribution_skips_many_markers(ch, seed):
    # records in start order on one GPU with short level-1 markers between
    # them (a record often lies two or more markers past the previous
    # record's), and records inside, before and after them; about as many
    # markers as records, so that a tile's markers fit its window
    rng = np.random.default_rng(5000 + seed)
    n = 3000
    start = np.sort(rng.integers(0, 400 * n, size=n)).astype(np.int64)
    end = start + rng.integers(0, 30, size=n)
    m1 = (8 * n) // 10
    ms1 = np.sort(rng.integers(0, 400 * n, size=m1)).astype(np.int64)
    me1 = ms1 + rng.integers(1, 60, size=m1)
    # level-1 markers must not overlap each other: keep a non-overlapping
    # subsequence
    keep = np.ones(m1, bool)
    last = -1
    for i in range(m1):
        if ms1[i] < last:
            keep[i] = False
        else:
            last = me1[i]
    ms1, me1 = ms1[keep], me1[keep]
    ms = np.concatenate([[0, 200 * n], ms1]).astype(np.int64)
    me = np.concatenate([[200 * n, 400 * n + 100], me1]).astype(np.int64)
    m = ms.shape[0]
    tr = tg.Trace(
        n_gpus=1, depth=2, gpu=np.zeros(n, np.uint8),
        stream=np.zeros(n, np.uint8), start=start, end=end,
        cls=np.zeros(n, np.uint8), op_id=np.zeros(n, np.uint32),
        counters=None, m_gpu=np.zeros(m, np.uint8),
        m_level=np.concatenate([[0, 0], np.ones(m - 2)]).astype(np.uint8),
        m_start=ms, m_end=me, m_label=np.arange(m, dtype=np.uint32),
        a_gpu=np.zeros(0, np.uint8), a_local=np.zeros(0, np.int64),
        a_ref=np.zeros(0, np.int64), name=f"many markers {seed}")
    say("attribution skips many markers", seed, n, m)
    assert_parity(run_gpu(ch, tr), oracle.run(tr), name=tr.name)


@pytest.mark.parametrize("n", [0, 1, 2, 3, 2047, 2048, 2049, 4097])
def test_edge_sizes(ch, n):
    tr = _tiny(n, m=5)
    say("edge", n)
    ref = oracle.run(tr)
    assert ref["status"] == 0
    assert_parity(run_gpu(ch, tr), ref, name=tr.name)


def test_no_markers(ch):
    tr = _tiny(100, m=0)
    say("no markers")
    assert_parity(run_gpu(ch, tr), oracle.run(tr), name="nomarkers")


def test_overflowing_marker_sets_flag(ch):
    tr = _tiny(300, m=6, depth=2, overlapping=True)
    say("marker overlap")
    got, ref = run_gpu(ch, tr), oracle.run(tr)
    assert ref["status"] & oracle.MARKER_OVERLAP
    assert_parity(got, ref, name="overlap")


def test_bad_inputs_set_status(ch):
    tr = tg.make_micro(5, n_gpus=2, n_kernels=100, depth=2)
    tr.gpu[3] = 7          # beyond n_gpus
    tr.cls[4] = 9          # unknown class
    tr.end[5] = tr.start[5] - 10
    tr.m_level[0] = 5      # beyond depth
    say("bad inputs")
    got, ref = run_gpu(ch, tr), oracle.run(tr)
    for bit in (oracle.BAD_GPU, oracle.BAD_CLASS, oracle.NEG_DURATION,
                oracle.BAD_LEVEL):
        assert got["status"] & bit and ref["status"] & bit, bit


def test_repeated_steps_are_identical(ch):
    tr = tg.make_config(1)
    say("repeat")
    pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"))
    pipe.status.zero_()
    pipe.step()
    a = pipe.results()
    for _ in range(3):
        pipe.step()
    b = pipe.results()
    for k in REC_KEYS:
        assert np.array_equal(a[k], b[k]), k
    for k in ROW_KEYS:
        assert np.array_equal(a["rows"][k], b["rows"][k]), k
