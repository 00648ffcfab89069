"""Full-size parity (the 20M-record headline trace and the 50M-record
adversarial trace), in the launch configuration bench.py times.

Clocks, alignment, attribution, overlap and bubbles are compared with the C
oracle over every record and marker; the two orders with numpy's stable
lexsort; the aggregated rows of every level with the oracle's own grouping
on the 20M-record trace and with the vectorized brute-force grouping of
tests/brute.py (pinned to the oracle on CPU) on the 50M-record one; the derived ratios
by recomputing the same IEEE divisions in numpy; the views, the overlap
statistics, the launch split and (on the 20M-record trace) the counter-pass
join with the oracle.  One module-scoped run per trace feeds short tests, so
that none of them is silent for long."""
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


class Full:
    """The trace, the GPU run and the oracle's results of one full-size
    configuration, computed once per module and in pieces, so that each
    test ends (and reports) within about a minute."""

    def __init__(self, ch, cid):
        self.ch, self.cid, self.t0 = ch, cid, time.time()
        tr = tg.make_config(cid, with_truth=False)
        self.tr = tr
        say(f"config {cid}: {tr.n} records {tr.n_markers} markers "
            f"({self.el()}s)")
        self.pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"))
        self.pipe.status.zero_()
        self.pipe.step()
        self.got = self.pipe.results()
        say(f"gpu done ({self.el()}s)")
        self._memo = {}

    def el(self):
        return f"{time.time() - self.t0:.0f}"

    def need(self, what):
        if what not in self._memo:
            self._memo[what] = getattr(self, "_" + what)()
        return self._memo[what]

    def _aligned(self):
        tr, G = self.tr, self.tr.n_gpus
        x0, c, d, rc = oracle.fit(tr.a_gpu, tr.a_local, tr.a_ref, G)
        s, _ = oracle.transform(tr.gpu, tr.start, G, x0, c, d)
        e, _ = oracle.transform(tr.gpu, tr.end, G, x0, c, d)
        ms, _ = oracle.transform(tr.m_gpu, tr.m_start, G, x0, c, d)
        me, _ = oracle.transform(tr.m_gpu, tr.m_end, G, x0, c, d)
        return dict(x0=x0, c=c, d=d, rc=rc, s=s, e=e, ms=ms, me=me)

    def _idx(self):
        tr, a = self.tr, self.need("aligned")
        return oracle.attribute(tr.gpu, a["s"], tr.m_gpu, tr.m_level, a["ms"],
                                a["me"], tr.depth, tr.n_gpus)

    def _ov(self):
        tr, a = self.tr, self.need("aligned")
        return oracle.overlap(tr.gpu, tr.stream, tr.cls, a["s"], a["e"],
                              tr.m_gpu, a["ms"], a["me"], tr.n_gpus)

    def _rows(self):
        """Rows of every level: the oracle's own aggregation on the 20M-record
        trace; on the 50M-record shuffled trace (where the oracle's
        sort-based grouping takes minutes) the vectorized grouping of
        tests/brute.py, pinned to the oracle on CPU."""
        tr, a = self.tr, self.need("aligned")
        idx, ov = self.need("idx")[0], self.need("ov")
        levels = list(range(tr.depth)) + [100, 101]
        if self.cid == 3:
            r = oracle.aggregate(tr.gpu, tr.cls, a["s"], a["e"], idx,
                                 ov["gap"], ov["ovl"], tr.counters, tr.depth)
            lo, out = r["level_offset"], {}
            for li, lev in enumerate(levels):
                sl = slice(int(lo[li]), int(lo[li + 1]))
                out[lev] = {k: r[k][sl] for k in ("gpu", "kind", "n", "dur",
                                                  "gap", "ovl", "tmin",
                                                  "tmax", "first")}
                out[lev]["path"] = r["path"][:, sl]
                out[lev]["ctr"] = r["ctr"][:, sl]
            return levels, out
        return levels, brute.aggregate_numpy(
            tr.gpu, tr.cls, a["s"], a["e"], idx, ov["gap"], ov["ovl"],
            tr.counters, tr.depth, levels)


@pytest.fixture(scope="module", params=[3, 4])
def full(ch, request):
    return Full(ch, request.param)


def test_full_align(full):
    tr, got, a = full.tr, full.got, full.need("aligned")
    assert got["status"] == 0, got["status"]
    assert a["rc"] == 0
    for k in ("x0", "c", "d"):
        same(got[k], a[k], k)
    same(got["start"], a["s"], "start")
    same(got["end"], a["e"], "end")
    same(got["mstart"], a["ms"], "mstart")
    same(got["mend"], a["me"], "mend")
    ar = np.arange(tr.n)
    kind = np.isin(tr.cls, [5, 6]).astype(np.int64)
    same(got["order"], np.lexsort((ar, a["s"], tr.stream.astype(np.int64),
                                   tr.gpu.astype(np.int64))), "order")
    same(got["korder"], np.lexsort((ar, a["s"], kind,
                                    tr.gpu.astype(np.int64))), "korder")
    say(f"align ok ({full.el()}s)")


def test_full_attribute(full):
    idx, st = full.need("idx")
    assert st == 0
    same(full.got["idx"], idx, "idx")
    say(f"attribute ok ({full.el()}s)")


def test_full_overlap(full):
    ov = full.need("ov")
    for k in ("ovl", "gap", "mwin", "gwin"):
        same(full.got[k], ov[k], k)
    say(f"overlap ok ({full.el()}s)")


def test_full_aggregate_and_ratios(full):
    levels, ref = full.need("rows")
    rows, lo = full.got["rows"], full.got["rows"]["level_offset"]
    for li, lev in enumerate(levels):
        sl = slice(lo[li], lo[li + 1])
        for k in ("gpu", "kind", "n", "dur", "gap", "ovl", "tmin", "tmax",
                  "first"):
            same(rows[k][sl], ref[lev][k], f"level {lev} {k}")
        same(rows["path"][:, sl], ref[lev]["path"], f"level {lev} path")
        same(rows["ctr"][:, sl], ref[lev]["ctr"], f"level {lev} ctr")
    say(f"aggregate ok ({full.el()}s)")
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
    gotr = full.got["ratios"]
    ok = (gotr == want) | (np.isnan(gotr) & np.isnan(want))
    assert ok.all(), "ratios"
    say(f"ratios ok ({full.el()}s)")


def test_full_views(full):
    # re-keyed views over (iteration, phase, class / operation) and medians
    # over iterations and GPUs, the first ten iterations as warm-up
    tr, cid, G = full.tr, full.cid, full.tr.n_gpus
    a, idx, ov = full.need("aligned"), full.need("idx")[0], full.need("ov")
    spec = dict(n_phases=3, n_ops=64, n_iters=ITERS[cid], warmup=10)
    v = full.ch.Views(full.pipe, **spec)
    v.run()
    gv = v.results()
    rv = oracle.views(tr.cls, a["s"], a["e"], idx, ov["gap"], ov["ovl"],
                      tr.m_level, tr.m_label, **spec)
    assert gv["n_units"] == rv["n_units"]
    if cid == 3:      # no marker dropped there
        assert rv["n_units"] == G * ITERS[cid]
        assert rv["iter_cnt"] == ITERS[cid] - 10
    for k in ("unit_marker", "cls_tab", "op_tab", "busy", "iter_max",
              "cls_cnt", "op_cnt"):
        same(gv[k], rv[k], f"views {k}")
    for k in ("cls_med", "op_med"):
        x, y = gv[k], rv[k]
        assert ((x == y) | (np.isnan(x) & np.isnan(y))).all(), f"views {k}"
    assert gv["iter_cnt"] == rv["iter_cnt"]
    assert gv["iter_med"] == rv["iter_med"]
    say(f"views ok ({full.el()}s)")


def test_full_op_stats(full):
    # overlap statistics and overhead breakdown per (phase, operation), the
    # oracle run on the brute-force rows of the operation level
    tr, pipe = full.tr, full.pipe
    _, ref = full.need("rows")
    fg = np.linspace(2e9, 9e10, 64)
    pipe.status.zero_()
    so, sc, sg, sgc = pipe.op_stats(freq_peak_mhz=2100.0, tpt_peak=1.3e6,
                                    f_gemm=fg, per_gpu=True)
    assert int(pipe.status.item()) & 0xFFFFFFFF == 0
    r3 = ref[3]
    lofs = np.zeros(tr.depth + 3, np.int64)
    lofs[4:] = r3["n"].shape[0]
    ro, rcnt, rg, rgc = oracle.op_stats(
        dict(r3, level_offset=lofs), tr.m_label, tr.depth,
        freq_peak_mhz=2100.0, tpt_peak=1.3e6, f_gemm=fg, n_gpus=tr.n_gpus,
        per_gpu=True)
    same(sc.cpu().numpy(), rcnt, "op stats counts")
    so = so.cpu().numpy()
    assert ((so == ro) | (np.isnan(so) & np.isnan(ro))).all(), "op stats"
    assert rcnt.sum() > 0
    # the per-GPU overlap CDFs that eq. 9 is read from
    same(sgc.cpu().numpy(), rgc, "per-GPU CDF counts")
    sg = sg.cpu().numpy()
    assert ((sg == rg) | (np.isnan(sg) & np.isnan(rg))).all(), "per-GPU CDF"
    assert rgc.sum() == rcnt.sum()
    say(f"op stats ok ({full.el()}s)")


def test_full_launch_split(full):
    # launch overhead split from seeded dispatch times
    import torch
    tr, a, G = full.tr, full.need("aligned"), full.tr.n_gpus
    tl = tg.make_launch(tr, 11, max_lead=20000)
    prep, call = full.pipe.launch_split(torch.from_numpy(tl).cuda())
    tla, _ = oracle.transform(tr.gpu, tl, G, a["x0"], a["c"], a["d"])
    rp, rc2 = oracle.launch_split(tr.gpu, tr.stream, tr.cls, a["s"], a["e"],
                                  tla)
    same(prep.cpu().numpy(), rp, "prep")
    same(call.cpu().numpy(), rc2, "call")
    say(f"launch split ok ({full.el()}s)")


def test_full_join(full):
    # counters of seven serialized passes attached back to the records (both
    # traces carry the 16 counters that the passes split)
    import torch
    tr, pipe, n = full.tr, full.pipe, full.tr.n
    a, idx = full.need("aligned"), full.need("idx")[0]
    lab = np.full(n, 0xFFFFFFFF, np.uint32)
    ok = idx[0] != 0xFFFFFFFF
    lab[ok] = tr.m_label[idx[0][ok]]
    passes = tg.make_counter_passes(tr, lab, 5, drop_frac=0.001,
                                    mismatch_frac=0.001, extra=2)
    t = lambda x, dt: torch.from_numpy(np.ascontiguousarray(x).view(dt)).cuda()
    dp = [dict(gpu=t(q["gpu"], np.uint8), stream=t(q["stream"], np.uint8),
               cls=t(q["cls"], np.uint8), label=t(q["lab"], np.int32),
               values=t(q["values"], np.int64), dst=q["dst"])
          for q in passes]
    pipe.status.zero_()
    ctr, matched = pipe.join_counters(dp)
    st = int(pipe.status.item()) & 0xFFFFFFFF
    say(f"join: gpu done, oracle ({full.el()}s)")
    rc3, rm3, rs3 = oracle.join(tr.gpu, tr.stream, tr.cls, a["s"], lab,
                                passes)
    assert st == rs3
    assert rs3 & oracle.JOIN_MISS
    same(matched.cpu().numpy(), rm3, "join matched")
    same(ctr.cpu().numpy().view(np.uint64), rc3, "join counters")
    say(f"join ok ({full.el()}s)")
