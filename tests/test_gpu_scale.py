"""Full-size parity (the 20M-record headline trace and the 50M-record
adversarial trace), in the launch configuration bench.py times.

Clocks, alignment, attribution, overlap and bubbles are compared with the C
oracle over every record and marker; the two orders with numpy's stable
lexsort; the aggregated rows of every level with the vectorized brute-force
grouping of tests/brute.py (pinned to the oracle on CPU); the derived ratios
by recomputing the same IEEE divisions in numpy."""
import sys
import time

import numpy as np
import pytest

import brute
import oracle
import tracegen as tg

pytestmark = pytest.mark.gpu


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


def same(a, b, what):
    a, b = np.asarray(a), np.asarray(b)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    if not np.array_equal(a, b):
        d = np.nonzero((a != b).reshape(-1))[0]
        raise AssertionError(f"{what}: {d.size} differences, first at {d[0]}")


ITERS = {3: 800, 4: 2035}     # iterations of the two traces


@pytest.mark.parametrize("cid", [3, 4])
def test_full_size_parity(ch, cid):
    t0 = time.time()
    tr = tg.make_config(cid, with_truth=False)
    say(f"config {cid}: {tr.n} records {tr.n_markers} markers "
        f"({time.time() - t0:.0f}s)")
    pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"))
    pipe.status.zero_()
    pipe.step()
    got = pipe.results()
    assert got["status"] == 0, got["status"]
    say(f"gpu done ({time.time() - t0:.0f}s)")
    G = tr.n_gpus
    x0, c, d, rc = oracle.fit(tr.a_gpu, tr.a_local, tr.a_ref, G)
    assert rc == 0
    same(got["x0"], x0, "x0")
    same(got["c"], c, "c")
    same(got["d"], d, "d")
    s, _ = oracle.transform(tr.gpu, tr.start, G, x0, c, d)
    e, _ = oracle.transform(tr.gpu, tr.end, G, x0, c, d)
    ms, _ = oracle.transform(tr.m_gpu, tr.m_start, G, x0, c, d)
    me, _ = oracle.transform(tr.m_gpu, tr.m_end, G, x0, c, d)
    same(got["start"], s, "start")
    same(got["end"], e, "end")
    same(got["mstart"], ms, "mstart")
    same(got["mend"], me, "mend")
    n = tr.n
    ar = np.arange(n)
    kind = np.isin(tr.cls, [5, 6]).astype(np.int64)
    same(got["order"], np.lexsort((ar, s, tr.stream.astype(np.int64),
                                   tr.gpu.astype(np.int64))), "order")
    same(got["korder"], np.lexsort((ar, s, kind, tr.gpu.astype(np.int64))),
         "korder")
    say(f"align ok ({time.time() - t0:.0f}s)")
    idx, st = oracle.attribute(tr.gpu, s, tr.m_gpu, tr.m_level, ms, me,
                               tr.depth, G)
    assert st == 0
    same(got["idx"], idx, "idx")
    say(f"attribute ok ({time.time() - t0:.0f}s)")
    ov = oracle.overlap(tr.gpu, tr.stream, tr.cls, s, e, tr.m_gpu, ms, me, G)
    for k in ("ovl", "gap", "mwin", "gwin"):
        same(got[k], ov[k], k)
    say(f"overlap ok ({time.time() - t0:.0f}s)")
    levels = list(range(tr.depth)) + [100, 101]
    ref = brute.aggregate_numpy(tr.gpu, tr.cls, s, e, idx, ov["gap"],
                                ov["ovl"], tr.counters, tr.depth, levels)
    rows, lo = got["rows"], got["rows"]["level_offset"]
    for li, lev in enumerate(levels):
        sl = slice(lo[li], lo[li + 1])
        for k in ("gpu", "kind", "n", "dur", "gap", "ovl", "tmin", "tmax",
                  "first"):
            same(rows[k][sl], ref[lev][k], f"level {lev} {k}")
        same(rows["path"][:, sl], ref[lev]["path"], f"level {lev} path")
        same(rows["ctr"][:, sl], ref[lev]["ctr"], f"level {lev} ctr")
    say(f"aggregate ok ({time.time() - t0:.0f}s)")
    # derived ratios: the same IEEE operations in numpy
    f = lambda a: np.asarray(a).astype(np.float64)
    with np.errstate(divide="ignore", invalid="ignore"):
        dur = f(rows["dur"])
        cyc = f(rows["ctr"][0])
        dpeak = cyc * 1000.0 / 2100.0
        want = np.stack([f(rows["ovl"]) / dur,
                         f(rows["ctr"][4] + rows["ctr"][5]) / dur,
                         f(rows["ctr"][13]) / f(rows["n"]),
                         f(rows["ctr"][1]) / cyc, dpeak, dur / dpeak])
    gotr = got["ratios"]
    ok = (gotr == want) | (np.isnan(gotr) & np.isnan(want))
    assert ok.all(), "ratios"
    say(f"ratios ok ({time.time() - t0:.0f}s)")
    # re-keyed views over (iteration, phase, class / operation) and medians
    # over iterations and GPUs, the first ten iterations as warm-up
    spec = dict(n_phases=3, n_ops=64, n_iters=ITERS[cid], warmup=10)
    v = ch.Views(pipe, **spec)
    v.run()
    gv = v.results()
    rv = oracle.views(tr.cls, s, e, idx, ov["gap"], ov["ovl"], tr.m_level,
                      tr.m_label, **spec)
    assert gv["n_units"] == rv["n_units"]
    if cid == 3:      # no marker dropped there
        assert rv["n_units"] == G * ITERS[cid]
        assert rv["iter_cnt"] == ITERS[cid] - 10
    for k in ("unit_marker", "cls_tab", "op_tab", "busy", "iter_max",
              "cls_cnt", "op_cnt"):
        same(gv[k], rv[k], f"views {k}")
    for k in ("cls_med", "op_med"):
        a, b = gv[k], rv[k]
        assert ((a == b) | (np.isnan(a) & np.isnan(b))).all(), f"views {k}"
    assert gv["iter_cnt"] == rv["iter_cnt"]
    assert gv["iter_med"] == rv["iter_med"]
    say(f"views ok ({time.time() - t0:.0f}s)")
    # overlap statistics and overhead breakdown per (phase, operation), the
    # oracle run on the brute-force rows of the operation level
    fg = np.linspace(2e9, 9e10, 64)
    pipe.status.zero_()
    so, sc = pipe.op_stats(freq_peak_mhz=2100.0, tpt_peak=1.3e6, f_gemm=fg)
    assert int(pipe.status.item()) & 0xFFFFFFFF == 0
    r3 = ref[3]
    lofs = np.zeros(tr.depth + 3, np.int64)
    lofs[4:] = r3["n"].shape[0]
    ro, rcnt = oracle.op_stats(dict(r3, level_offset=lofs), tr.m_label,
                               tr.depth, freq_peak_mhz=2100.0, tpt_peak=1.3e6,
                               f_gemm=fg)
    same(sc.cpu().numpy(), rcnt, "op stats counts")
    so = so.cpu().numpy()
    assert ((so == ro) | (np.isnan(so) & np.isnan(ro))).all(), "op stats"
    assert rcnt.sum() > 0
    say(f"op stats ok ({time.time() - t0:.0f}s)")
    # launch overhead split from seeded dispatch times
    import torch
    tl = tg.make_launch(tr, 11, max_lead=20000)
    prep, call = pipe.launch_split(torch.from_numpy(tl).cuda())
    tla, _ = oracle.transform(tr.gpu, tl, G, x0, c, d)
    rp, rc2 = oracle.launch_split(tr.gpu, tr.stream, tr.cls, s, e, tla)
    same(prep.cpu().numpy(), rp, "prep")
    same(call.cpu().numpy(), rc2, "call")
    say(f"launch split ok ({time.time() - t0:.0f}s)")
    if cid == 3:
        # counters of seven serialized passes attached back to the records
        lab = np.full(n, 0xFFFFFFFF, np.uint32)
        ok = idx[0] != 0xFFFFFFFF
        lab[ok] = tr.m_label[idx[0][ok]]
        passes = tg.make_counter_passes(tr, lab, 5, drop_frac=0.001,
                                        mismatch_frac=0.001, extra=2)
        t = lambda a, dt: torch.from_numpy(
            np.ascontiguousarray(a).view(dt)).cuda()
        dp = [dict(gpu=t(q["gpu"], np.uint8), stream=t(q["stream"], np.uint8),
                   cls=t(q["cls"], np.uint8), label=t(q["lab"], np.int32),
                   values=t(q["values"], np.int64), dst=q["dst"])
              for q in passes]
        pipe.status.zero_()
        ctr, matched = pipe.join_counters(dp)
        st = int(pipe.status.item()) & 0xFFFFFFFF
        rc3, rm3, rs3 = oracle.join(tr.gpu, tr.stream, tr.cls, s, lab, passes)
        assert st == rs3 == oracle.JOIN_MISS
        same(matched.cpu().numpy(), rm3, "join matched")
        same(ctr.cpu().numpy().view(np.uint64), rc3, "join counters")
    say(f"done ({time.time() - t0:.0f}s)")
