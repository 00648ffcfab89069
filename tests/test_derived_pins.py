"""Pins of the oracle's derived metrics (Section III-C derived metrics such as
bandwidth; eq. 10 duration at the peak clock; Section V-C overlap windows).

* a hand-worked fixture (tests/golden/derived_metrics.json) whose counter
  columns all hold distinct values, so that reading a wrong column, a wrong
  numerator or a wrong denominator changes an expected value;
* the meaning of the counter columns taken from the generator's counter
  table (cycles from duration and SCLK, SCLK samples in 1300..2100 MHz):
  mean SCLK of every row lies in that range and the actual over peak-clock
  duration in [1, 2100/1300];
* window fractions equal the exact rationals w / (window length), rounded
  once to the nearest double, with the window length taken from the aligned
  marker times (so CO + MO + OV + ID = length is pinned too).
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
import tracegen as tg

HERE = os.path.dirname(os.path.abspath(__file__))
GOLD = json.load(open(os.path.join(HERE, "golden", "derived_metrics.json")))


def _same(got, want):
    return (np.isnan(got) and np.isnan(want)) or got == want


def _rows_from_fixture():
    rs = GOLD["rows"]
    return dict(n_rows=len(rs),
                n=np.array([r["n"] for r in rs], np.uint64),
                dur=np.array([r["dur"] for r in rs], np.int64),
                ovl=np.array([r["ovl"] for r in rs], np.int64),
                ctr=np.array([r["ctr"] for r in rs], np.uint64).T.copy())


def test_ratios_hand_worked():
    rows = _rows_from_fixture()
    rat = oracle.ratios(rows, GOLD["freq_peak_mhz"])
    assert rat.shape == (6, rows["n_rows"])
    for i, r in enumerate(GOLD["rows"]):
        for col, w in enumerate(r["want"]):
            assert _same(rat[col, i], float(w)), (i, col, rat[col, i], w,
                                                   r["why"])


def test_ratios_every_counter_column_matters():
    """Changing any counter column that a metric reads changes that metric,
    and changing any other column changes nothing."""
    rows = _rows_from_fixture()
    base = oracle.ratios(rows, GOLD["freq_peak_mhz"])
    reads = {0: {3, 4, 5}, 1: {3}, 4: {1}, 5: {1}, 13: {2}}
    for c in range(16):
        mod = dict(rows)
        mod["ctr"] = rows["ctr"].copy()
        mod["ctr"][c, 0] += np.uint64(7)
        got = oracle.ratios(mod, GOLD["freq_peak_mhz"])
        changed = {z for z in range(6) if not _same(got[z, 0], base[z, 0])}
        assert changed == reads.get(c, set()), (c, changed)


def test_ratios_follow_counter_table():
    """Rows of a trace whose counters come from the generator's table: SCLK
    samples lie in 1300..2100 MHz, so the mean SCLK column does; cycles are
    duration x SCLK / 1000 per record, so the duration over the duration at
    the 2100 MHz peak lies in [1, 2100/1300] (up to the drift of the clock
    alignment and the floor of the cycle count)."""
    tr = tg.make_config(2, iters=2)
    r = oracle.run(tr, freq_peak_mhz=2100.0)
    rows, rat = r["rows"], r["ratios"]
    n = rows["n"].astype(np.float64)
    live = (rows["dur"] > 0) & (n > 0)
    assert live.sum() > 1000
    assert ((rat[2][n > 0] >= 1300.0) & (rat[2][n > 0] <= 2100.0)).all()
    q = rat[5][live]
    assert (q >= 1.0 - 1e-4).all() and (q <= 2100.0 / 1300.0 + 1e-3).all()
    # bandwidth from the two byte counters only
    bw = (rows["ctr"][4].astype(np.float64) + rows["ctr"][5]) / rows["dur"]
    np.testing.assert_allclose(rat[1][live], bw[live], rtol=1e-15)


def test_window_fractions_hand_worked():
    w = np.array([x["w"] for x in GOLD["windows"]], np.int64)
    got = oracle.window_fractions(w)
    for i, x in enumerate(GOLD["windows"]):
        for z, want in enumerate(x["want"]):
            assert _same(got[i, z], float(want)), (i, z, got[i, z], x["why"])


@pytest.mark.parametrize("case", ["config0", "micro", "unnested"])
def test_window_fractions_are_exact_rationals(case):
    if case == "config0":
        tr = tg.make_config(0)
    elif case == "micro":
        tr = tg.make_micro(31, n_gpus=3, n_kernels=500, n_streams=3, depth=3,
                           anchors=4)
    else:
        tr = tg.make_micro(32, n_gpus=2, n_kernels=300, n_streams=2, depth=3,
                           nested=False)
    r = oracle.run(tr)
    length = r["mend"] - r["mstart"]
    mwin, wf = r["mwin"].reshape(-1, 4), r["wfrac"].reshape(-1, 4)
    assert mwin.shape[0] == tr.n_markers
    for j in range(mwin.shape[0]):
        L = int(max(length[j], 0))
        assert int(mwin[j].sum()) == L, j
        for z in range(4):
            if L == 0:
                assert np.isnan(wf[j, z])
            else:
                assert wf[j, z] == float(Fraction(int(mwin[j, z]), L)), (j, z)
