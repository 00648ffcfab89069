"""Pins of the oracle's re-keyed views (Fig. end_to_end: duration and launch
overhead per phase and class, medians across iterations and GPUs,
throughput from the largest duration plus launch overhead across GPUs;
Section V-B / Fig. operation_time: operation duration summed across layers
with its bubbles; Section IV: warm-up iterations left out) to things other
than the oracle itself: a hand-worked example, a dictionary brute force over
the records, Python's statistics.median, and the aggregate rows."""
import math
import statistics

import numpy as np
import pytest

import oracle
import tracegen as tg

NONE = 0xFFFFFFFF


def _views(tr, r, **kw):
    return oracle.views(tr.cls, r["start"], r["end"], r["idx"], r["gap"],
                        r["ovl"], tr.m_level, tr.m_label, **kw)


# ----------------------------------------------------------------------------
# hand-worked example
# ----------------------------------------------------------------------------
def _hand_trace():
    """Two GPUs, three iterations [0,100), [100,200), [200,300) each, one
    phase marker (label 0) and one operation marker (label 5) per iteration,
    compute kernels on stream 0 and one all_gather on stream 1 (GPU 0,
    iteration 1)."""
    # a compute kernel's bubble reaches back to the previous compute kernel
    # of its stream, also across an iteration boundary
    recs = [  # gpu, stream, start, end, cls          busy of the iteration
        (0, 0, 10, 30, 0), (0, 0, 40, 50, 2),      # 20 + 10 + bubble 10 = 40
        (0, 0, 110, 120, 0), (0, 1, 115, 140, 5),  # 10 + bubble 60 = 70
        (0, 0, 200, 260, 1),                       # 60 + bubble 80 = 140
        (1, 0, 5, 25, 0), (1, 0, 25, 35, 0),       # 20 + 10 = 30
        (1, 0, 100, 150, 3), (1, 0, 170, 180, 2),  # 50 + 65 + 10 + 20 = 145
        (1, 0, 210, 220, 0),                       # 10 + bubble 30 = 40
    ]
    mks = []
    for g in range(2):
        for it in range(3):
            a, b = 100 * it, 100 * it + 100
            mks += [(g, 0, a, b, it), (g, 1, a, b, 0), (g, 2, a, b, 0),
                    (g, 3, a, b, 5)]
    r = np.array(recs, np.int64)
    m = np.array(mks, np.int64)
    n = len(recs)
    return tg.Trace(
        n_gpus=2, depth=4, gpu=r[:, 0].astype(np.uint8),
        stream=r[:, 1].astype(np.uint8), start=r[:, 2], end=r[:, 3],
        cls=r[:, 4].astype(np.uint8), op_id=np.zeros(n, np.uint32),
        counters=None, m_gpu=m[:, 0].astype(np.uint8),
        m_level=m[:, 1].astype(np.uint8), m_start=m[:, 2], m_end=m[:, 3],
        m_label=m[:, 4].astype(np.uint32), a_gpu=np.zeros(0, np.uint8),
        a_local=np.zeros(0, np.int64), a_ref=np.zeros(0, np.int64),
        name="views-hand")


def test_views_hand_example():
    tr = _hand_trace()
    r = oracle.run(tr)
    assert r["status"] == 0
    v = _views(tr, r, n_phases=1, n_ops=8, n_iters=3, warmup=0)
    assert v["n_units"] == 6
    # units are the iteration markers in input order: (gpu 0, it 0..2),
    # (gpu 1, it 0..2)
    assert v["unit_marker"].tolist() == [0, 4, 8, 12, 16, 20]
    # busy = kernel time + bubbles of the compute kernels of the unit
    assert v["busy"].tolist() == [40, 70, 140, 30, 145, 40]
    # the largest across GPUs per iteration, then the median over iterations
    assert v["iter_max"].tolist() == [40, 145, 140]
    assert v["iter_med"] == 140.0 and v["iter_cnt"] == 3
    # warm-up: iteration 0 left out -> median of {145, 140}
    w = _views(tr, r, n_phases=1, n_ops=8, n_iters=3, warmup=1)
    assert w["iter_med"] == 142.5 and w["iter_cnt"] == 2
    # class view, phase 0: GEMM (class 0) in units 0, 1, 3 (two kernels,
    # bubble 0), 5; attention in unit 2; RMSNorm in unit 4
    P, C = 1, 8
    # tables are [field][group][unit]; viewed here as [unit, phase, class]
    unit_major = lambda a, *g: np.moveaxis(a.reshape(*g, 6), -1, 0)
    n_tab = unit_major(v["cls_tab"][0], P, C)
    d_tab = unit_major(v["cls_tab"][1], P, C).astype(np.int64)
    g_tab = unit_major(v["cls_tab"][2], P, C).astype(np.int64)
    assert n_tab[:, 0, 0].tolist() == [1, 1, 0, 2, 0, 1]
    assert d_tab[:, 0, 0].tolist() == [20, 10, 0, 30, 0, 10]
    assert n_tab[:, 0, 2].tolist() == [1, 0, 0, 0, 1, 0]
    assert g_tab[:, 0, 2].tolist() == [10, 0, 0, 0, 20, 0]
    assert n_tab[:, 0, 5].tolist() == [0, 1, 0, 0, 0, 0]   # the all_gather
    assert d_tab[1, 0, 5] == 25
    # GEMM over units 0, 1, 3, 5: durations {20, 10, 30, 10}, bubbles
    # {0, 60, 0, 30}, sums {20, 70, 30, 40}
    assert v["cls_cnt"][0] == 4
    assert v["cls_med"][0][0] == 15.0
    assert v["cls_med"][1][0] == 15.0
    assert v["cls_med"][2][0] == 35.0
    # operation view: op 5, compute: dur + gap per unit = busy
    O = 8
    o_n = unit_major(v["op_tab"][0], P, O, 2)
    o_d = unit_major(v["op_tab"][1], P, O, 2).astype(np.int64)
    o_g = unit_major(v["op_tab"][2], P, O, 2).astype(np.int64)
    assert (o_d[:, 0, 5, 0] + o_g[:, 0, 5, 0]).tolist() == v["busy"].tolist()
    assert o_n[:, 0, 5, 1].tolist() == [0, 1, 0, 0, 0, 0]
    # the all_gather [115, 140) overlaps the GEMM [110, 120) for 5 ns
    assert int(unit_major(v["op_tab"][3], P, O, 2)[1, 0, 5, 1]) == 5
    g = (0 * O + 5) * 2
    assert v["op_cnt"][g] == 6
    assert v["op_med"][2][g] == 55.0      # {30, 40, 40, 70, 140, 145}
    assert math.isnan(v["op_med"][0][(0 * O + 4) * 2])      # empty group


# ----------------------------------------------------------------------------
# brute force over the records (dictionaries, no index arithmetic)
# ----------------------------------------------------------------------------
def _brute(tr, r, P, O, NI, warmup, iter_level=0, phase_level=1, op_level=2):
    n = tr.start.shape[0]
    idx = r["idx"].reshape(-1, n)
    units = [m for m in range(tr.m_level.shape[0])
             if tr.m_level[m] == iter_level]
    cls_d, op_d, busy = {}, {}, {m: 0 for m in units}
    for k in range(n):
        mi = int(idx[iter_level][k])
        if mi == NONE:
            continue
        dur = int(r["end"][k]) - int(r["start"][k])
        gp, ov = int(r["gap"][k]), int(r["ovl"][k])
        comm = int(tr.cls[k]) in (5, 6)
        if not comm:
            busy[mi] += dur + gp
        mp = int(idx[phase_level][k])
        if mp == NONE or int(tr.m_label[mp]) >= P:
            continue
        p = int(tr.m_label[mp])
        if int(tr.cls[k]) < 8:
            e = cls_d.setdefault((mi, p, int(tr.cls[k])), [0, 0, 0])
            e[0] += 1
            e[1] += dur
            e[2] += gp
        mo = int(idx[op_level][k])
        if mo == NONE or int(tr.m_label[mo]) >= O:
            continue
        e = op_d.setdefault((mi, p, int(tr.m_label[mo]), int(comm)),
                            [0, 0, 0, 0])
        e[0] += 1
        e[1] += dur
        e[2] += gp
        e[3] += ov
    it_max = {}
    for m in units:
        lab = int(tr.m_label[m])
        if lab < NI:
            it_max[lab] = max(it_max.get(lab, -1), busy[m])
    return units, cls_d, op_d, busy, it_max


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_views_brute_force(seed):
    tr = tg.make_micro(seed, n_gpus=3, n_kernels=300, depth=3, span=6000)
    r = oracle.run(tr)
    P, O, NI, W = 50, 50, 50, 7
    v = _views(tr, r, iter_level=0, phase_level=1, op_level=2, n_phases=P,
               n_ops=O, n_iters=NI, warmup=W)
    units, cls_d, op_d, busy, it_max = _brute(tr, r, P, O, NI, W)
    U = len(units)
    assert v["n_units"] == U and v["unit_marker"].tolist() == units
    ui = {m: u for u, m in enumerate(units)}
    ct = np.moveaxis(v["cls_tab"].astype(np.int64).reshape(3, P, 8, U), 3, 1)
    got = {}
    for u, p, c in zip(*np.nonzero(ct[0])):
        got[(units[u], int(p), int(c))] = [int(ct[f, u, p, c])
                                           for f in range(3)]
    assert got == cls_d
    ot = np.moveaxis(v["op_tab"].astype(np.int64).reshape(4, P, O, 2, U), 4,
                     1)
    got = {}
    for u, p, o, k in zip(*np.nonzero(ot[0])):
        got[(units[u], int(p), int(o), int(k))] = [int(ot[f, u, p, o, k])
                                                   for f in range(4)]
    assert got == op_d
    assert v["busy"].tolist() == [busy[m] for m in units]
    assert v["iter_max"].tolist() == [it_max.get(i, -1) for i in range(NI)]
    # medians: statistics.median over the kept units of each group
    kept = [m for m in units if int(tr.m_label[m]) >= W]
    for p in range(P):
        for c in range(8):
            for st in range(3):
                vals = []
                for m in kept:
                    e = cls_d.get((m, p, c))
                    if e:
                        vals.append([e[1], e[2], e[1] + e[2]][st])
                g = p * 8 + c
                assert v["cls_cnt"][g] == len(vals)
                got = v["cls_med"][st][g]
                if vals:
                    assert got == statistics.median(vals)
                else:
                    assert math.isnan(got)
    for (m, p, o, k) in {(m, p, o, k) for (m, p, o, k) in op_d}:
        g = (p * O + o) * 2 + k
        vals = [op_d[(q, p, o, k)][1] + op_d[(q, p, o, k)][2] for q in kept
                if (q, p, o, k) in op_d]
        assert v["op_cnt"][g] == len(vals)
        if vals:
            assert v["op_med"][2][g] == statistics.median(vals)
    its = [it_max[i] for i in range(W, NI) if it_max.get(i, -1) >= 0]
    assert v["iter_cnt"] == len(its)
    if its:
        assert v["iter_med"] == statistics.median(its)


# ----------------------------------------------------------------------------
# invariants against the aggregate rows (an independent grouping)
# ----------------------------------------------------------------------------
def test_views_against_rows_config0():
    tr = tg.make_config(0)
    r = oracle.run(tr)
    P, O = 3, 64
    v = _views(tr, r, n_phases=P, n_ops=O, n_iters=4, warmup=0)
    rows, lo = r["rows"], r["rows"]["level_offset"]
    U = v["n_units"]
    ui = {int(m): u for u, m in enumerate(v["unit_marker"])}
    # busy: level-0 rows of kind 0 (path0 = the unit's iteration marker)
    b = np.zeros(U, np.int64)
    for i in range(lo[0], lo[1]):
        if rows["kind"][i] == 0 and rows["path"][0, i] != NONE:
            b[ui[int(rows["path"][0, i])]] += rows["dur"][i] + rows["gap"][i]
    assert v["busy"].tolist() == b.tolist()
    # operation view: level-3 rows re-keyed by (unit, phase label, operation
    # label, kind) and summed across layers
    ot = np.moveaxis(v["op_tab"].astype(np.int64).reshape(4, P, O, 2, U), 4,
                     1)
    acc = np.zeros_like(ot)
    for i in range(lo[3], lo[4]):
        p0, p1, p3 = (int(rows["path"][l, i]) for l in (0, 1, 3))
        if NONE in (p0, p1, p3):
            continue
        ph, op = int(tr.m_label[p1]), int(tr.m_label[p3])
        if ph >= P or op >= O:
            continue
        k = int(rows["kind"][i])
        for f, key in enumerate(("n", "dur", "gap", "ovl")):
            acc[f, ui[p0], ph, op, k] += int(rows[key][i])
    assert np.array_equal(acc, ot)
    # class view summed over classes = level-1 rows (phase) summed over kind
    ct = np.moveaxis(v["cls_tab"].astype(np.int64).reshape(3, P, 8, U), 3, 1)
    acc = np.zeros((3, U, P), np.int64)
    for i in range(lo[1], lo[2]):
        p0, p1 = int(rows["path"][0, i]), int(rows["path"][1, i])
        if NONE in (p0, p1) or int(tr.m_label[p1]) >= P:
            continue
        for f, key in enumerate(("n", "dur", "gap")):
            acc[f, ui[p0], int(tr.m_label[p1])] += int(rows[key][i])
    assert np.array_equal(acc, ct.sum(axis=3))
    # every compute record of config 0 lies in an operation (label below
    # 64), phase and iteration; a communication record can start before the
    # first marker (the first all_gather of the pipeline fill)
    comp = ~np.isin(tr.cls, [5, 6])
    dur = (r["end"] - r["start"]).astype(np.int64)
    assert int(ot[1, :, :, :, 0].sum()) == int(dur[comp].sum())
    idx = r["idx"].reshape(-1, tr.start.shape[0])
    inside = (idx[0] != NONE) & (idx[1] != NONE)
    assert int(ct[0].sum()) == int(inside.sum()) >= tr.start.shape[0] - 1
