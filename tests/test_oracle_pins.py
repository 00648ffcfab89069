"""Pins of the CPU oracle to things other than itself: a hand-worked example,
closed forms, exact rational least squares, per-nanosecond brute force,
linear scans, the paper's launch-overhead equations, and invariants."""
import json
import os
import random
from fractions import Fraction

import numpy as np
import pytest

import brute
import oracle
import tracegen as tg

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "worked_example.json")))


def golden_trace():
    r, m = GOLD["records"], GOLD["markers"]
    n = len(r["gpu"])
    return tg.Trace(
        n_gpus=GOLD["n_gpus"], depth=GOLD["depth"],
        gpu=np.array(r["gpu"], np.uint8), stream=np.array(r["stream"], np.uint8),
        start=np.array(r["start"], np.int64), end=np.array(r["end"], np.int64),
        cls=np.array(r["cls"], np.uint8), op_id=np.zeros(n, np.uint32),
        counters=None, m_gpu=np.array(m["gpu"], np.uint8),
        m_level=np.array(m["level"], np.uint8),
        m_start=np.array(m["start"], np.int64),
        m_end=np.array(m["end"], np.int64),
        m_label=np.array(m["label"], np.uint32),
        a_gpu=np.zeros(0, np.uint8), a_local=np.zeros(0, np.int64),
        a_ref=np.zeros(0, np.int64), name="golden")


# ----------------------------------------------------------------------------
# worked example
# ----------------------------------------------------------------------------
def test_golden_worked_example():
    tr = golden_trace()
    r = oracle.run(tr)
    ex = GOLD["expect"]
    assert r["status"] == 0
    assert r["order"].tolist() == ex["order"]
    assert r["korder"].tolist() == ex["korder"]
    assert r["idx"].tolist() == ex["idx"]
    assert r["ovl"].tolist() == ex["ovl"]
    assert r["gap"].tolist() == ex["gap"]
    assert r["mwin"].tolist() == ex["mwin"]
    assert r["gwin"].tolist() == ex["gwin"]
    rows, lo = r["rows"], r["rows"]["level_offset"]
    for lev, key in ((1, "rows_level1"), (0, "rows_level0")):
        got = []
        for i in range(lo[lev], lo[lev + 1]):
            got.append(dict(path=rows["path"][:, i].tolist(),
                            gpu=int(rows["gpu"][i]), kind=int(rows["kind"][i]),
                            n=int(rows["n"][i]), dur=int(rows["dur"][i]),
                            gap=int(rows["gap"][i]), ovl=int(rows["ovl"][i]),
                            tmin=int(rows["tmin"][i]), tmax=int(rows["tmax"][i]),
                            first=int(rows["first"][i])))
        assert got == ex[key]


@pytest.mark.parametrize("case", range(len(GOLD["clock_cases"])))
def test_golden_clock(case):
    cc = GOLD["clock_cases"][case]
    a = np.array([(g, x, x + w) for (g, x, w, cnt) in cc["anchor_groups"]
                  for _ in range(cnt)], np.int64)
    x0, c, d, rc = oracle.fit(a[:, 0], a[:, 1], a[:, 2], 1)
    assert rc == 0
    assert (int(x0[0]), int(c[0]), int(d[0])) == (cc["x0"], cc["c"], cc["d"])
    if not cc["transform"]:
        return
    t = np.array([p[0] for p in cc["transform"]], np.int64)
    out, st = oracle.transform(np.zeros(t.shape, np.uint8), t, 1, x0, c, d)
    assert out.tolist() == [p[1] for p in cc["transform"]]


# ----------------------------------------------------------------------------
# clock fit
# ----------------------------------------------------------------------------
def test_fit_no_anchors_is_identity():
    tr = tg.make_config(0)
    r = oracle.run(tr)
    assert (r["d"] == 0).all() and (r["c"] == 0).all()
    assert (r["start"] == tr.start).all() and (r["end"] == tr.end).all()
    assert (r["mstart"] == tr.m_start).all()


@pytest.mark.parametrize("seed", range(6))
def test_fit_exact_line_closed_form(seed):
    """Anchors exactly on w = c0 + p*k at local times x0 + k*2^38:
    D = p*2^10, C = c0 + p*k_first, and every anchor maps onto its
    reference time."""
    rnd = random.Random(seed)
    c0 = rnd.randint(-10**9, 10**9)
    p = rnd.randint(-2**20, 2**20)
    x0 = rnd.randint(-2**60, 2**60)
    ks = sorted(rnd.sample(range(0, 15), rnd.randint(2, 8)))
    xs = [x0 + k * 2**38 for k in ks]
    ys = [x + c0 + p * k for x, k in zip(xs, ks)]
    x0o, c, d, rc = oracle.fit(np.zeros(len(xs)), xs, ys, 1)
    assert rc == 0
    # the intercept is taken at the first anchor, k = ks[0]
    assert int(d[0]) == p * 2**10 and int(c[0]) == c0 + p * ks[0]
    assert int(x0o[0]) == xs[0]
    out, _ = oracle.transform(np.zeros(len(xs), np.uint8), np.array(xs), 1,
                              x0o, c, d)
    assert out.tolist() == ys
    # between anchors the aligned time is the floor of the exact line
    ts = [x0 + rnd.randint(-2**40, 2**41) for _ in range(50)]
    out, _ = oracle.transform(np.zeros(50, np.uint8), np.array(ts), 1, x0o, c,
                              d)
    for t, v in zip(ts, out.tolist()):
        exact = t + c0 + Fraction(p * (t - x0), 2**38)
        assert v == exact.numerator // exact.denominator


@pytest.mark.parametrize("seed", range(25))
def test_fit_matches_exact_rational_least_squares(seed):
    rnd = random.Random(100 + seed)
    G = rnd.randint(1, 4)
    gs, xs, ys = [], [], []
    for g in range(G):
        na = rnd.choice([0, 1, 2, 3, rnd.randint(4, 50)])
        off = rnd.randint(-10**7, 10**7)
        drift = rnd.uniform(-3e-4, 3e-4)
        base = rnd.randint(-2**61, 2**61)
        for q in range(na):
            x = base + rnd.randint(0, 2**41)
            if rnd.random() < 0.2 and q > 0:
                x = xs[-1]                      # duplicate local times
            ys.append(x + off + int(drift * (x - base)) + rnd.randint(-60, 60))
            xs.append(x)
            gs.append(g)
    x0, c, d, rc = oracle.fit(gs, xs, ys, G)
    assert rc == 0
    for g in range(G):
        sx = [x for x, q in zip(xs, gs) if q == g]
        sy = [y for y, q in zip(ys, gs) if q == g]
        assert (int(x0[g]), int(c[g]), int(d[g])) == brute.fit_fraction(sx, sy)


def test_fit_guards():
    # |w| >= 2^40 is refused
    x0, c, d, rc = oracle.fit([0, 0], [0, 10], [2**41, 2**41 + 10], 1)
    assert rc == oracle.EOVERFLOW
    # a slope of 1e-2 (D >= 2^38) is refused
    x0, c, d, rc = oracle.fit([0, 0], [0, 10**9], [0, 10**9 + 10**7], 1)
    assert rc == oracle.EOVERFLOW


def test_fit_agrees_with_float_least_squares():
    tr = tg.make_config(1)
    x0, c, d, rc = oracle.fit(tr.a_gpu, tr.a_local, tr.a_ref, tr.n_gpus)
    assert rc == 0
    for g in range(tr.n_gpus):
        sel = tr.a_gpu == g
        u = (tr.a_local[sel] - x0[g]).astype(np.float64)
        w = (tr.a_ref[sel] - tr.a_local[sel]).astype(np.float64)
        slope, icpt = np.polyfit(u, w, 1)
        assert abs(slope * 2**48 - d[g]) < 1e-6 * 2**48 * 1e-3
        assert abs(icpt - c[g]) < 1.0


@pytest.mark.parametrize("cid", [1, 2])
def test_align_recovers_reference_clock(cid):
    """With +-50 ns anchor jitter, aligned kernel times stay within 50 ns of
    the generator's reference-clock times."""
    tr = tg.make_config(cid)
    x0, c, d, rc = oracle.fit(tr.a_gpu, tr.a_local, tr.a_ref, tr.n_gpus)
    s, _ = oracle.transform(tr.gpu, tr.start, tr.n_gpus, x0, c, d)
    e, _ = oracle.transform(tr.gpu, tr.end, tr.n_gpus, x0, c, d)
    assert np.abs(s - tr.truth["ref_start"]).max() <= 50
    assert np.abs(e - tr.truth["ref_end"]).max() <= 50
    assert (e >= s).all()                      # monotone transform


# ----------------------------------------------------------------------------
# sort orders
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(8))
def test_orders_match_python_stable_sort(seed):
    tr = tg.make_micro(seed, n_kernels=300, n_streams=4)
    s = tr.start
    o = oracle.order(tr.gpu, tr.stream, tr.cls, s, False)
    ref = sorted(range(tr.n), key=lambda k: (tr.gpu[k], tr.stream[k], s[k]))
    assert o.tolist() == ref
    ko = oracle.order(tr.gpu, tr.stream, tr.cls, s, True)
    kind = np.isin(tr.cls, [5, 6]).astype(int)
    ref = sorted(range(tr.n), key=lambda k: (tr.gpu[k], kind[k], s[k]))
    assert ko.tolist() == ref


# ----------------------------------------------------------------------------
# attribution
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("nested", [True, False])
def test_attribute_matches_linear_scan(seed, nested):
    tr = tg.make_micro(seed, n_gpus=2, n_kernels=80, depth=4, nested=nested)
    idx, st = oracle.attribute(tr.gpu, tr.start, tr.m_gpu, tr.m_level,
                               tr.m_start, tr.m_end, tr.depth, tr.n_gpus)
    ref = brute.attribute_scan(tr.gpu, tr.start, tr.m_gpu, tr.m_level,
                               tr.m_start, tr.m_end, tr.depth)
    assert (idx == ref).all()
    # overlap flag: any two non-empty markers of one (gpu, level) intersect
    ov = False
    for j in range(tr.n_markers):
        for q in range(j + 1, tr.n_markers):
            if (tr.m_gpu[j] == tr.m_gpu[q] and tr.m_level[j] == tr.m_level[q]
                    and tr.m_end[j] > tr.m_start[j]
                    and tr.m_end[q] > tr.m_start[q]
                    and max(tr.m_start[j], tr.m_start[q]) <
                    min(tr.m_end[j], tr.m_end[q])):
                ov = True
    assert bool(st & oracle.MARKER_OVERLAP) == ov


@pytest.mark.parametrize("cid", [0, 1])
def test_attribute_op_marker_label_equals_op_id(cid):
    tr = tg.make_config(cid)
    r = oracle.run(tr)
    comp = ~np.isin(tr.cls, [5, 6])
    op = r["idx"][3][comp]
    assert (op != oracle.NONE).all()
    assert (tr.m_label[op] == tr.op_id[comp]).all()
    # iteration label of every compute kernel's level-0 marker is consistent
    it = tr.m_label[r["idx"][0][comp]]
    assert it.min() == 0 and it.max() == tg.CONFIGS[cid]["iters"] - 1


# ----------------------------------------------------------------------------
# overlap and bubbles
# ----------------------------------------------------------------------------
@pytest.mark.parametrize("seed", range(12))
@pytest.mark.parametrize("nested", [True, False])
def test_overlap_matches_per_ns_brute_force(seed, nested):
    tr = tg.make_micro(seed, n_gpus=2, n_kernels=70, n_streams=3, depth=3,
                       nested=nested)
    got = oracle.overlap(tr.gpu, tr.stream, tr.cls, tr.start, tr.end, tr.m_gpu,
                         tr.m_start, tr.m_end, tr.n_gpus)
    ref = brute.overlap_brute(tr.gpu, tr.stream, tr.cls, tr.start, tr.end,
                              tr.m_gpu, tr.m_start, tr.m_end, tr.n_gpus)
    for k in ("ovl", "gap", "mwin", "gwin"):
        assert (got[k] == ref[k]).all(), k


def test_overlap_config0_per_ns_brute_force():
    tr = tg.make_config(0)
    got = oracle.overlap(tr.gpu, tr.stream, tr.cls, tr.start, tr.end, tr.m_gpu,
                         tr.m_start, tr.m_end, tr.n_gpus)
    lo, c, m = brute.timelines(tr.gpu, tr.cls, tr.start, tr.end, tr.n_gpus)
    for j in range(tr.n_markers):
        w = brute.window_counts(lo, c, m, tr.m_gpu[j], tr.m_start[j],
                                tr.m_end[j])
        assert tuple(got["mwin"][j]) == w
    g = got["gwin"][0]
    assert tuple(g[2:]) == brute.window_counts(lo, c, m, 0, g[0], g[1])
    for k in range(0, tr.n, 7):
        if tr.end[k] > tr.start[k]:
            assert got["ovl"][k] == brute.window_counts(
                lo, c, m, 0, tr.start[k], tr.end[k])[2]


def _union_len(iv):
    iv = sorted((a, b) for a, b in iv if b > a)
    tot, cur_a, cur_b = 0, None, None
    for a, b in iv:
        if cur_b is None or a > cur_b:
            if cur_b is not None:
                tot += cur_b - cur_a
            cur_a, cur_b = a, b
        else:
            cur_b = max(cur_b, b)
    if cur_b is not None:
        tot += cur_b - cur_a
    return tot


def test_overlap_invariants_config1():
    tr = tg.make_config(1)
    r = oracle.run(tr)
    s, e = r["start"], r["end"]
    kind = np.isin(tr.cls, [5, 6])
    for g in range(tr.n_gpus):
        gw = r["gwin"][g]
        assert gw[2:].sum() == gw[1] - gw[0]
        sel = tr.gpu == g
        cu = _union_len(zip(s[sel & ~kind], e[sel & ~kind]))
        mu = _union_len(zip(s[sel & kind], e[sel & kind]))
        assert gw[2] + gw[4] == cu            # CO + OV = |union compute|
        assert gw[3] + gw[4] == mu            # MO + OV = |union comm|
        # one compute stream: overlapped ns of compute kernels add up to OV
        assert r["ovl"][sel & ~kind].sum() == gw[4]
        assert (e - s)[sel & ~kind].sum() == gw[2] + gw[4]
    w = r["mwin"]
    assert (w.sum(1) == np.maximum(r["mend"] - r["mstart"], 0)).all()


def test_overlap_special_cases():
    # no comm at all: MO = OV = 0; comm nested in one kernel: OV = comm dur
    gpu = np.zeros(3, np.uint8)
    stream = np.array([0, 0, 1], np.uint8)
    cls = np.array([0, 0, 5], np.uint8)
    s = np.array([0, 100, 20], np.int64)
    e = np.array([50, 200, 40], np.int64)
    r = oracle.overlap(gpu[:2], stream[:2], cls[:2], s[:2], e[:2],
                       np.zeros(0, np.uint8), np.zeros(0), np.zeros(0), 1)
    assert r["gwin"][0].tolist() == [0, 200, 150, 0, 0, 50]
    r = oracle.overlap(gpu, stream, cls, s, e, np.zeros(0, np.uint8),
                       np.zeros(0), np.zeros(0), 1)
    assert r["gwin"][0].tolist() == [0, 200, 130, 0, 20, 50]
    assert r["ovl"].tolist() == [20, 0, 20]


def test_gap_equals_launch_overhead_equations():
    """eqs. (1)-(3): O_prep + O_call = t_ks,i - t_ke,i-1 for any dispatch
    time t_l, so the summed launch overhead is the bubble the oracle reports
    whenever the next compute kernel starts after the previous one ended."""
    tr = tg.make_config(0)
    r = oracle.run(tr)
    rnd = random.Random(7)
    comp = np.nonzero(~np.isin(tr.cls, [5, 6]))[0]
    o = r["order"]
    pos = np.empty(tr.n, np.int64)
    pos[o] = np.arange(tr.n)
    checked = 0
    for k in comp:
        p = pos[k]
        q = p - 1
        while q >= 0 and tr.cls[o[q]] in (5, 6) and tr.stream[o[q]] == \
                tr.stream[k]:
            q -= 1
        if q < 0 or tr.stream[o[q]] != tr.stream[k]:
            assert r["gap"][k] == 0
            continue
        t_ke, t_ks = int(r["end"][o[q]]), int(r["start"][k])
        if t_ks < t_ke:
            assert r["gap"][k] == 0
            continue
        t_l = rnd.randint(t_ke - 10_000, t_ks + 10_000)
        o_prep = max(t_l - t_ke, 0)
        o_call = min(t_ks - t_l, t_ks - t_ke)
        assert o_prep + o_call == r["gap"][k]
        checked += 1
    assert checked > 1000


# ----------------------------------------------------------------------------
# aggregation
# ----------------------------------------------------------------------------
def _rows_of(rows, lo, hi, depth, nc):
    out = []
    for i in range(lo, hi):
        out.append(dict(path=rows["path"][:, i].tolist(), gpu=int(rows["gpu"][i]),
                        kind=int(rows["kind"][i]), n=int(rows["n"][i]),
                        dur=int(rows["dur"][i]), gap=int(rows["gap"][i]),
                        ovl=int(rows["ovl"][i]), tmin=int(rows["tmin"][i]),
                        tmax=int(rows["tmax"][i]), first=int(rows["first"][i]),
                        ctr=[int(x) for x in rows["ctr"][:, i]]))
    return out


@pytest.mark.parametrize("seed", range(10))
@pytest.mark.parametrize("nested", [True, False])
def test_aggregate_matches_dict_grouping(seed, nested):
    tr = tg.make_micro(seed, n_gpus=3, n_kernels=90, depth=3, n_counters=3,
                       nested=nested)
    r = oracle.run(tr)
    levels = list(range(tr.depth)) + [100, 101]
    ref = brute.aggregate_brute(tr.gpu, tr.cls, r["start"], r["end"], r["idx"],
                                r["gap"], r["ovl"], tr.counters, tr.depth,
                                levels)
    rows, lo = r["rows"], r["rows"]["level_offset"]
    for li, lev in enumerate(levels):
        got = _rows_of(rows, lo[li], lo[li + 1], tr.depth, tr.n_counters)
        want = [dict(path=w["path"], gpu=w["gpu"], kind=w["kind"], n=w["n"],
                     dur=w["dur"], gap=w["gap"], ovl=w["ovl"], tmin=w["tmin"],
                     tmax=w["tmax"], first=w["first"], ctr=w["ctr"])
                for w in ref[lev]]
        assert got == want, lev


@pytest.mark.parametrize("seed", range(6))
def test_aggregate_filter_matches_dict_grouping(seed):
    tr = tg.make_micro(seed, n_gpus=3, n_kernels=90, depth=3, n_counters=2)
    rnd = random.Random(seed)
    gpus = rnd.sample(range(3), 2)
    classes = rnd.sample(range(8), 5)
    base = oracle.run(tr)
    lab = tr.m_label
    it = (min(lab), max(lab) - 5)
    f = oracle.make_filter(gpus=gpus, classes=classes, iters=it)
    r = oracle.run(tr, filt=f)
    m0 = base["idx"][0]
    sel = [(tr.gpu[k] in gpus) and (tr.cls[k] in classes) and
           m0[k] != oracle.NONE and it[0] <= lab[m0[k]] <= it[1]
           for k in range(tr.n)]
    levels = list(range(tr.depth)) + [100, 101]
    ref = brute.aggregate_brute(tr.gpu, tr.cls, r["start"], r["end"], r["idx"],
                                r["gap"], r["ovl"], tr.counters, tr.depth,
                                levels, sel)
    rows, lo = r["rows"], r["rows"]["level_offset"]
    for li, lev in enumerate(levels):
        got = _rows_of(rows, lo[li], lo[li + 1], tr.depth, tr.n_counters)
        assert [g["n"] for g in got] == [w["n"] for w in ref[lev]]
        assert [g["first"] for g in got] == [w["first"] for w in ref[lev]]


def test_aggregate_single_level_requests():
    tr = tg.make_micro(3, n_gpus=2, n_kernels=60, depth=3, n_counters=1)
    full = oracle.run(tr)
    lo = full["rows"]["level_offset"]
    for li, lev in enumerate([0, 1, 2, 100, 101]):
        one = oracle.aggregate(tr.gpu, tr.cls, full["start"], full["end"],
                               full["idx"], full["gap"], full["ovl"],
                               tr.counters, tr.depth, lev)
        olo = one["level_offset"]
        assert olo[li + 1] - olo[li] == lo[li + 1] - lo[li]
        assert one["n_rows"] == lo[li + 1] - lo[li]
        sl = slice(lo[li], lo[li + 1])
        assert (one["n"] == full["rows"]["n"][sl]).all()
        assert (one["tmin"] == full["rows"]["tmin"][sl]).all()


@pytest.mark.parametrize("cid", [0, 1])
def test_aggregate_invariants(cid):
    tr = tg.make_config(cid)
    r = oracle.run(tr)
    rows, lo, D = r["rows"], r["rows"]["level_offset"], tr.depth
    N = tr.n
    for li in range(D + 2):
        assert int(rows["n"][lo[li]:lo[li + 1]].sum()) == N  # conservation
    # coarser rows are sums of their children
    for lev in range(D):
        fine = slice(lo[lev + 1], lo[lev + 2]) if lev + 1 < D else None
        if fine is None:
            continue
        parent = {}
        for i in range(lo[lev], lo[lev + 1]):
            key = (int(rows["gpu"][i]), tuple(rows["path"][:lev + 1, i]),
                   int(rows["kind"][i]))
            parent[key] = [0, 0, 0, 0]
        for i in range(fine.start, fine.stop):
            key = (int(rows["gpu"][i]), tuple(rows["path"][:lev + 1, i]),
                   int(rows["kind"][i]))
            acc = parent[key]
            acc[0] += int(rows["n"][i])
            acc[1] += int(rows["dur"][i])
            acc[2] += int(rows["gap"][i])
            acc[3] += int(rows["ovl"][i])
        for i in range(lo[lev], lo[lev + 1]):
            key = (int(rows["gpu"][i]), tuple(rows["path"][:lev + 1, i]),
                   int(rows["kind"][i]))
            assert parent[key] == [int(rows["n"][i]), int(rows["dur"][i]),
                                   int(rows["gap"][i]), int(rows["ovl"][i])]
    wl = slice(lo[D + 1], lo[D + 2])
    assert int(rows["dur"][wl].sum()) == int((r["end"] - r["start"]).sum())
    assert int(rows["ovl"][wl].sum()) == int(r["ovl"].sum())
    assert int(rows["gap"][wl].sum()) == int(r["gap"].sum())
    assert r["rows"]["status"] & oracle.PATH_CONFLICT == 0


def test_aggregate_counter_wraparound():
    tr = tg.make_micro(1, n_gpus=1, n_kernels=20, depth=2, n_counters=2)
    tr.counters[:] = np.uint64(2**64 - 3)
    r = oracle.run(tr)
    rows, lo = r["rows"], r["rows"]["level_offset"]
    for i in range(lo[2], lo[3]):                      # GPU rows
        assert int(rows["ctr"][0, i]) == (int(rows["n"][i]) * (2**64 - 3)) % 2**64


def test_path_conflict_flag():
    """Two records of one deepest marker but different parents: flagged."""
    gpu = np.zeros(2, np.uint8)
    cls = np.zeros(2, np.uint8)
    s = np.array([10, 30], np.int64)
    e = np.array([20, 40], np.int64)
    # level-1 marker [0, 50) spans two level-0 markers [0, 25) and [25, 50)
    idx = np.array([[0, 1], [2, 2]], np.uint32)
    z = np.zeros(2, np.int64)
    out = oracle.aggregate(gpu, cls, s, e, idx, z, z, None, 2)
    assert out["status"] & oracle.PATH_CONFLICT
    idx = np.array([[0, 0], [2, 2]], np.uint32)
    out = oracle.aggregate(gpu, cls, s, e, idx, z, z, None, 2)
    assert not out["status"] & oracle.PATH_CONFLICT


def test_ratios_are_single_ieee_divisions():
    tr = tg.make_config(0)
    tr2 = tg.make_micro(2, n_gpus=1, n_kernels=40, depth=2, n_counters=16)
    for t in (tr, tr2):
        r = oracle.run(t, freq_peak_mhz=2100.0)
        rows, rat = r["rows"], r["ratios"]
        for i in range(rows["n_rows"]):
            d = float(int(rows["dur"][i]))
            o = float(int(rows["ovl"][i]))
            want = o / d if d != 0 else (float("nan") if o == 0 else
                                         float("inf") * (1 if o > 0 else -1))
            got = rat[0, i]
            assert (np.isnan(got) and np.isnan(want)) or got == want
            if t.n_counters == 16:
                c = [int(x) for x in rows["ctr"][:, i]]
                cyc = float(c[0])
                if cyc > 0 and d > 0:
                    assert rat[3, i] == float(c[1]) / cyc
                    assert rat[4, i] == cyc * 1000.0 / 2100.0
                    assert rat[1, i] == float((c[4] + c[5]) % 2**64) / d
            else:
                assert np.isnan(rat[1:, i]).all()


@pytest.mark.parametrize("case", ["config1", "micro"])
def test_numpy_aggregation_matches_oracle(case):
    """The vectorized brute-force grouping used for full-size checks agrees
    with the oracle row for row."""
    if case == "config1":
        tr = tg.make_config(1)
    else:
        tr = tg.make_micro(9, n_gpus=3, n_kernels=400, depth=3, n_counters=5)
    r = oracle.run(tr)
    levels = list(range(tr.depth)) + [100, 101]
    ref = brute.aggregate_numpy(tr.gpu, tr.cls, r["start"], r["end"], r["idx"],
                                r["gap"], r["ovl"], tr.counters, tr.depth,
                                levels)
    rows, lo = r["rows"], r["rows"]["level_offset"]
    for li, lev in enumerate(levels):
        sl = slice(lo[li], lo[li + 1])
        for k in ("n", "dur", "gap", "ovl", "tmin", "tmax", "first", "gpu",
                  "kind"):
            assert np.array_equal(ref[lev][k], rows[k][sl]), (lev, k)
        assert np.array_equal(ref[lev]["path"], rows["path"][:, sl]), lev
        assert np.array_equal(ref[lev]["ctr"], rows["ctr"][:, sl]), lev
