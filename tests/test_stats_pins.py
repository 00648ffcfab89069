"""Pins of the oracle's overlap statistics and overhead breakdown (Fig.
gemm_overlap: overlap ratio against operation duration, correlation,
quantile fills; Section VI eqs. 6-10): numpy's corrcoef and polyfit on the
same instances, exact lines, constant overlap (NaN correlation, as the paper
notes), order statistics, and the breakdown equations evaluated here."""
import math

import numpy as np
import pytest

import oracle

NONE = 0xFFFFFFFF


def _rows(ovl, dur, gap, kind=None, ctr=None, phase=0, op=1):
    """Operation-level rows of one (phase, operation): marker 0 is the phase
    marker (label phase), marker 1 the operation marker (label op)."""
    n = len(dur)
    path = np.zeros((4, n), np.uint32)
    path[1], path[3] = 0, 1
    return dict(level_offset=np.array([0, 0, 0, 0, n, n, n], np.int64),
                path=path, kind=np.zeros(n, np.uint8) if kind is None
                else np.asarray(kind, np.uint8),
                n=np.ones(n, np.uint64), dur=np.asarray(dur, np.int64),
                gap=np.asarray(gap, np.int64), ovl=np.asarray(ovl, np.int64),
                ctr=ctr), np.array([phase, op], np.uint32)


def _stat(out, name, g=0):
    return out[oracle.OP_STATS.index(name)][g]


def test_stats_against_numpy():
    rng = np.random.default_rng(1)
    m = 500
    dur = rng.integers(1000, 100000, m)
    ovl = (dur * rng.random(m)).astype(np.int64)
    gap = rng.integers(0, 5000, m)
    rows, lab = _rows(ovl, dur, gap)
    out, cnt = oracle.op_stats(rows, lab, 4, n_phases=1, n_ops=2)
    g = 1                                  # phase 0, operation 1
    assert cnt[g] == m
    x = np.floor(ovl * 2.0**30 / dur)      # exact here: below 2^53
    y = (dur + gap).astype(np.float64)
    assert abs(_stat(out, "pearson", g) - np.corrcoef(x, y)[0, 1]) < 1e-12
    b, a = np.polyfit(x, y, 1)
    assert math.isclose(_stat(out, "slope", g), b, rel_tol=1e-9)
    assert math.isclose(_stat(out, "intercept", g), a, rel_tol=1e-9)
    assert _stat(out, "d50", g) == _stat(out, "intercept", g) + \
        _stat(out, "slope", g) * 2.0**29
    xs = np.sort(x) / 2.0**30
    assert _stat(out, "q0", g) == xs[0] and _stat(out, "q100", g) == xs[-1]
    assert _stat(out, "q25", g) == xs[(m - 1) // 4]
    assert _stat(out, "q75", g) == xs[3 * (m - 1) // 4]
    assert _stat(out, "q50", g) == np.median(x) / 2.0**30
    assert _stat(out, "d_act", g) == y.sum() / m
    assert math.isnan(_stat(out, "pearson", 0)) and cnt[0] == 0


def test_stats_exact_line_and_constant_overlap():
    # dur = 2^20: x = ovl * 2^10 exactly; y = 1000 + 3 ovl = 1000 + 3 x / 2^10
    # on every instance -> correlation 1, slope 3 / 2^10, duration 1000 at
    # no overlap
    dur = np.full(64, 1 << 20, np.int64)
    ovl = np.arange(64, dtype=np.int64) * 1000
    gap = 1000 + 3 * ovl - dur
    rows, lab = _rows(ovl, dur, gap)
    out, _ = oracle.op_stats(rows, lab, 4, n_phases=1, n_ops=2)
    assert abs(_stat(out, "pearson", 1) - 1.0) < 1e-15
    assert math.isclose(_stat(out, "slope", 1), 3 / 2**10, rel_tol=1e-12)
    assert math.isclose(_stat(out, "d0", 1), 1000, rel_tol=1e-12)
    # constant overlap ratio: no correlation defined (NaN), as for b_mlp_n
    rows, lab = _rows(np.zeros(10, np.int64), np.arange(10, 20),
                      np.zeros(10, np.int64))
    out, cnt = oracle.op_stats(rows, lab, 4, n_phases=1, n_ops=2)
    assert cnt[1] == 10 and math.isnan(_stat(out, "pearson", 1))
    assert math.isnan(_stat(out, "slope", 1))
    assert _stat(out, "q0", 1) == _stat(out, "q100", 1) == 0.0


def test_stats_breakdown_equations():
    rng = np.random.default_rng(2)
    m = 200
    dur = rng.integers(1000, 50000, m)
    ovl = (dur * rng.random(m)).astype(np.int64)
    gap = rng.integers(0, 500, m)
    ctr = np.zeros((16, m), np.uint64)
    ctr[0] = rng.integers(1000, 100000, m)          # GPU cycles
    ctr[1] = (ctr[0] * rng.random(m)).astype(np.uint64)   # MFMA busy
    ctr[11] = rng.integers(1 << 20, 1 << 30, m)     # MFMA flops
    rows, lab = _rows(ovl, dur, gap, ctr=ctr)
    fg = np.full(2, 7.5e8)
    out, _ = oracle.op_stats(rows, lab, 4, n_phases=1, n_ops=2,
                             freq_peak_mhz=2100.0, tpt_peak=1.3e6, f_gemm=fg)
    g = 1
    d_act = float((dur + gap).sum()) / m
    d_peak = float(ctr[0].sum()) * 1000.0 / 2100.0 / m        # eq. 10
    util = float(ctr[1].sum()) / float(ctr[0].sum())
    assert _stat(out, "d_peak", g) == d_peak
    assert _stat(out, "ovr_util", g) == 1.0 / util              # eq. 8
    assert _stat(out, "ovr_inst", g) == (float(ctr[11].sum()) / m) / 7.5e8
    assert _stat(out, "d_thr", g) == 7.5e8 / 1.3e6             # eq. 6
    # eq. 9 from the per-GPU CDF (one GPU here): its D_50% / D_0%
    _, _, gout, gcnt = oracle.op_stats(rows, lab, 4, n_phases=1, n_ops=2,
                                       freq_peak_mhz=2100.0, tpt_peak=1.3e6,
                                       f_gemm=fg, per_gpu=True)
    ovr_ov = gout[oracle.OP_CDF.index("ovr"), g]
    assert gcnt[g] == m
    assert ovr_ov == gout[oracle.OP_CDF.index("d50"), g] / \
        gout[oracle.OP_CDF.index("d0"), g]
    assert _stat(out, "ovr_overlap", g) == ovr_ov
    assert _stat(out, "ovr_freq", g) == d_act / d_peak / ovr_ov  # eq. 10
    # communication rows and rows of zero duration are not instances
    kind = np.zeros(m, np.uint8)
    kind[:50] = 1
    rows2, _ = _rows(ovl, dur, gap, kind=kind, ctr=ctr)
    _, cnt = oracle.op_stats(rows2, lab, 4, n_phases=1, n_ops=2)
    assert cnt[g] == m - 50


# ---------------------------------------------------------------- per-GPU CDF
import json
import os
from fractions import Fraction

GOLD_CDF = json.load(open(os.path.join(os.path.dirname(__file__), "golden",
                                       "overlap_cdf.json")))


def _rows_gpu(gpu, ovl, dur, gap, phase=0, op=1):
    rows, lab = _rows(ovl, dur, gap, phase=phase, op=op)
    rows["gpu"] = np.asarray(gpu, np.uint8)
    return rows, lab


def _cdf(gout, name, i):
    return gout[oracle.OP_CDF.index(name), i]


def test_cdf_hand_worked():
    r = np.array(GOLD_CDF["rows"], np.int64)
    rows, lab = _rows_gpu(r[:, 0], r[:, 1], r[:, 2], r[:, 3])
    out, cnt, gout, gcnt = oracle.op_stats(rows, lab, 4, n_phases=1, n_ops=2,
                                           n_gpus=2, per_gpu=True)
    g = 1                                  # phase 0, operation 1
    for h, want in enumerate(GOLD_CDF["gpu"]):
        i = g * 2 + h
        assert gcnt[i] == want["m"], (h, want["why"])
        for k, q in zip(("q0", "q25", "q50", "q75", "q100"), want["q"]):
            assert _cdf(gout, k, i) == float(q), (h, k)
        assert _cdf(gout, "y_min", i) == want["y_min"]
        for k in ("d0", "d50", "ovr"):
            assert _cdf(gout, k, i) == float(want[k]), (h, k, want["why"])
    assert _stat(out, "ovr_overlap", g) == float(GOLD_CDF["ovr_overlap"])
    # empty groups: count 0, NaN
    assert gcnt[0] == gcnt[1] == 0 and np.isnan(gout[:, 0]).all()


def _random_gpus(seed, m=400, G=5):
    rng = np.random.default_rng(seed)
    gpu = rng.integers(0, G, m)
    dur = rng.integers(1000, 100000, m)
    ovl = (dur * rng.random(m)).astype(np.int64)
    ovl[rng.random(m) < 0.3] = 0               # ties at no overlap
    gap = rng.integers(0, 5000, m)
    return gpu, ovl, dur, gap


@pytest.mark.parametrize("seed", [3, 4, 5])
def test_cdf_invariants(seed):
    """Per-GPU counts add up to the operation's; quantiles are ordered and
    the per-GPU extremes are the operation's extremes (pinned above against
    numpy); normalised durations are at least 1; eq. 9 is the median of the
    per-GPU ratios (statistics.median)."""
    import statistics
    G = 5
    gpu, ovl, dur, gap = _random_gpus(seed, G=G)
    rows, lab = _rows_gpu(gpu, ovl, dur, gap)
    out, cnt, gout, gcnt = oracle.op_stats(rows, lab, 4, n_phases=1, n_ops=2,
                                           n_gpus=G, per_gpu=True)
    g = 1
    sl = slice(g * G, (g + 1) * G)
    assert gcnt[sl].sum() == cnt[g] == len(dur)
    q = np.stack([gout[oracle.OP_CDF.index(k), sl]
                  for k in ("q0", "q25", "q50", "q75", "q100")])
    assert (np.diff(q, axis=0) >= 0).all()
    assert q[0].min() == _stat(out, "q0", g)
    assert q[4].max() == _stat(out, "q100", g)
    assert (gout[oracle.OP_CDF.index("d0"), sl] >= 1.0).all()
    assert (gout[oracle.OP_CDF.index("d50"), sl] >= 1.0).all()
    for h in range(G):
        sel = gpu == h
        assert _cdf(gout, "y_min", g * G + h) == (dur + gap)[sel].min()
    ratios = list(gout[oracle.OP_CDF.index("ovr"), sl])
    assert _stat(out, "ovr_overlap", g) == statistics.median(ratios)


def test_cdf_single_gpu_quantiles_are_the_operation_quantiles():
    gpu, ovl, dur, gap = _random_gpus(7, G=1)
    rows, lab = _rows_gpu(gpu, ovl, dur, gap)
    out, cnt, gout, gcnt = oracle.op_stats(rows, lab, 4, n_phases=1, n_ops=2,
                                           n_gpus=1, per_gpu=True)
    for k in ("q0", "q25", "q50", "q75", "q100"):
        assert _cdf(gout, k, 1) == _stat(out, k, 1), k


def test_cdf_closed_forms():
    # constant duration: every normalised duration is 1, eq. 9 gives 1
    G = 3
    gpu = np.arange(60) % G
    dur = np.full(60, 5000, np.int64)
    ovl = (np.arange(60) * 83) % 5000
    rows, lab = _rows_gpu(gpu, ovl, dur, np.zeros(60, np.int64))
    out, _, gout, _ = oracle.op_stats(rows, lab, 4, n_phases=1, n_ops=2,
                                      n_gpus=G, per_gpu=True)
    for h in range(G):
        assert _cdf(gout, "d0", G + h) == _cdf(gout, "d50", G + h) == 1.0
    assert _stat(out, "ovr_overlap", 1) == 1.0
    # duration growing with overlap, distinct ratios: the CDF order is the
    # duration order, so D_0% = 1 and D_50% = median / minimum
    m = 41
    dur = np.full(m, 1 << 20, np.int64)
    ovl = np.arange(m, dtype=np.int64)[::-1] * 1000   # rows not in x order
    gap = 2000 + 7 * ovl
    rows, lab = _rows_gpu(np.zeros(m), ovl, dur, gap)
    out, _, gout, _ = oracle.op_stats(rows, lab, 4, n_phases=1, n_ops=2,
                                      n_gpus=1, per_gpu=True)
    y = dur + gap
    assert _cdf(gout, "d0", 1) == 1.0
    want = Fraction(int(np.sort(y)[m // 2]), int(y.min()))
    assert _cdf(gout, "d50", 1) == float(want)
    assert _stat(out, "ovr_overlap", 1) == float(want)
