"""Parity of chopper_views (re-keyed views and their medians) with the CPU
oracle through the C ABI: tables, busy times, iteration maxima and counts
bit-exact; medians equal as doubles (NaN matching NaN) since both sides take
the same two order statistics and the same IEEE operations."""
import sys

import numpy as np
import pytest

import oracle
import tracegen as tg
from test_views_pins import _hand_trace

pytestmark = pytest.mark.gpu

INT_KEYS = ("unit_marker", "cls_tab", "op_tab", "busy", "iter_max", "cls_cnt",
            "op_cnt")


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


def run_both(ch, tr, **spec):
    pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"))
    pipe.status.zero_()
    pipe.step()
    v = ch.Views(pipe, **spec)
    v.run()
    got = v.results()
    st = int(pipe.status.item()) & 0xFFFFFFFF
    r = pipe.results()
    ref = oracle.views(tr.cls, r["start"], r["end"], r["idx"], r["gap"],
                       r["ovl"], tr.m_level, tr.m_label, **spec)
    return got, ref, st


def assert_views(got, ref, name):
    assert got["n_units"] == ref["n_units"], name
    for k in INT_KEYS:
        g, r = np.asarray(got[k]), np.asarray(ref[k])
        assert g.shape == r.shape, (name, k, g.shape, r.shape)
        if not np.array_equal(g, r):
            d = np.nonzero((g != r).reshape(-1))[0]
            raise AssertionError(f"{name}: {k}: {d.size} differences, first "
                                 f"at {d[0]}: {g.reshape(-1)[d[0]]} vs "
                                 f"{r.reshape(-1)[d[0]]}")
    for k in ("cls_med", "op_med"):
        g, r = np.asarray(got[k]), np.asarray(ref[k])
        same = (g == r) | (np.isnan(g) & np.isnan(r))
        if not same.all():
            i = np.nonzero(~same.reshape(-1))[0][0]
            raise AssertionError(f"{name}: {k}: first difference at {i}: "
                                 f"{g.reshape(-1)[i]!r} vs {r.reshape(-1)[i]!r}")
    assert got["iter_cnt"] == ref["iter_cnt"], name
    gm, rm = got["iter_med"], ref["iter_med"]
    assert gm == rm or (np.isnan(gm) and np.isnan(rm)), (name, gm, rm)


def test_views_hand_example(ch):
    say("views: hand example")
    tr = _hand_trace()
    for w in (0, 1, 3):
        got, ref, st = run_both(ch, tr, n_phases=1, n_ops=8, n_iters=3,
                                warmup=w)
        assert st == 0
        assert_views(got, ref, f"hand warmup={w}")
    assert got["iter_cnt"] == 0 and np.isnan(got["iter_med"])


@pytest.mark.parametrize("seed", [0, 1, 2, 3, 4, 5])
def test_views_micro(ch, seed):
    say(f"views: micro seed {seed}")
    tr = tg.make_micro(seed, n_gpus=3, n_kernels=300 + 97 * seed, depth=3,
                       span=6000)
    got, ref, _ = run_both(ch, tr, iter_level=0, phase_level=1, op_level=2,
                           n_phases=16, n_ops=50, n_iters=50, warmup=7)
    assert_views(got, ref, f"micro {seed}")


def test_views_micro_levels_swapped(ch):
    say("views: micro, other level choice")
    tr = tg.make_micro(11, n_gpus=2, n_kernels=900, depth=4, span=9000)
    got, ref, _ = run_both(ch, tr, iter_level=1, phase_level=0, op_level=3,
                           n_phases=16, n_ops=128, n_iters=40, warmup=0)
    assert_views(got, ref, "micro levels 1/0/3")


# (config, its iterations, n_iters, warm-up)
@pytest.mark.parametrize("cid,iters,ni,w", [(0, 2, 4, 0), (0, 2, 4, 1),
                                            (1, 10, 10, 2), (2, 100, 100, 10)])
def test_views_configs(ch, cid, iters, ni, w):
    say(f"views: config {cid} warmup {w}")
    tr = tg.make_config(cid)
    got, ref, st = run_both(ch, tr, n_phases=3, n_ops=64, n_iters=ni,
                            warmup=w)
    assert st == 0
    assert_views(got, ref, f"config {cid}")
    assert got["n_units"] == tr.n_gpus * iters
    assert got["iter_cnt"] == iters - w


def test_views_no_units(ch):
    say("views: no marker at the unit level")
    tr = tg.make_micro(3, n_gpus=2, n_kernels=200, depth=3, span=5000)
    tr.m_level = np.where(tr.m_level == 0, 1, tr.m_level).astype(np.uint8)
    got, ref, _ = run_both(ch, tr, iter_level=0, phase_level=1, op_level=2,
                           n_phases=16, n_ops=50, n_iters=50, warmup=0)
    assert got["n_units"] == 0
    assert_views(got, ref, "no units")


def test_views_shuffled_records(ch):
    """Records in shuffled order (the adversarial trace's shape, six
    iterations): a 512-record tile meets far more (iteration, phase) pairs
    than the class view sums per group, so most records take the item by
    item path; tables and medians exact."""
    say("views: shuffled records")
    tr = tg.make_config(4, iters=6)
    got, ref, st = run_both(ch, tr, n_phases=3, n_ops=64, n_iters=6,
                            warmup=1)
    # distinct (iteration marker, phase marker) pairs per 512-record tile
    r = oracle.run(tr)
    idx = r["idx"].reshape(-1, tr.n)
    key = idx[0].astype(np.uint64) << np.uint64(32) | idx[1].astype(np.uint64)
    tiles = [np.unique(key[i:i + 512]).size for i in range(0, tr.n, 512)]
    assert np.mean(tiles) > 16, np.mean(tiles)
    assert_views(got, ref, "shuffled")
    # (the trace drops a few markers, iteration markers among them)
    assert 0 < got["n_units"] <= tr.n_gpus * 6
