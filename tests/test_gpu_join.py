"""Parity of chopper_join_counters (Section III-A counter passes attached to
the runtime trace, III-B) with the CPU oracle through the C ABI: counters and
matched bits bit-exact, status bits equal; the round trip of unperturbed
passes gives back the generator's counters."""
import sys

import numpy as np
import pytest

import oracle
import tracegen as tg

pytestmark = pytest.mark.gpu
NONE = 0xFFFFFFFF


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


def join_both(ch, tr, passes):
    import torch
    pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"))
    pipe.status.zero_()
    pipe.step()
    pipe.status.zero_()
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a).view(dt)).cuda()
    dp = [dict(gpu=t(q["gpu"], np.uint8), stream=t(q["stream"], np.uint8),
               cls=t(q["cls"], np.uint8), label=t(q["lab"], np.int32),
               values=t(q["values"], np.int64), dst=q["dst"]) for q in passes]
    ctr, m = pipe.join_counters(dp)
    got = (ctr.cpu().numpy().view(np.uint64), m.cpu().numpy(),
           int(pipe.status.item()) & 0xFFFFFFFF)
    r = pipe.results()
    idx = r["idx"][0]
    lab = np.full(tr.n, NONE, np.uint32)
    ok = idx != NONE
    lab[ok] = tr.m_label[idx[ok]]
    ref = oracle.join(tr.gpu, tr.stream, tr.cls, r["start"], lab, passes)
    return got, ref, lab


def check(got, ref, name):
    gc, gm, gs = got
    rc, rm, rs = ref
    assert gs == rs, (name, gs, rs)
    assert np.array_equal(gm, rm), name
    if not np.array_equal(gc, rc):
        d = np.nonzero((gc != rc).reshape(-1))[0]
        raise AssertionError(f"{name}: {d.size} counter differences, first "
                             f"at {d[0]}")


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_join_micro(ch, seed):
    say(f"join: micro seed {seed}")
    tr = tg.make_micro(seed, n_gpus=2 + seed % 2, n_kernels=500 + 100 * seed,
                       n_streams=1 + seed % 3, depth=2, span=9000,
                       n_counters=16)
    for variant in range(3):
        r0 = oracle.run(tr)
        idx = r0["idx"].reshape(-1, tr.n)[0]
        lab = np.full(tr.n, NONE, np.uint32)
        lab[idx != NONE] = tr.m_label[idx[idx != NONE]]
        passes = tg.make_counter_passes(
            tr, lab, seed + 100 * variant,
            drop_frac=[0, 0.02, 0][variant],
            mismatch_frac=[0, 0.03, 0][variant], extra=[0, 2, 5][variant])
        got, ref, lab = join_both(ch, tr, passes)
        check(got, ref, f"micro {seed} variant {variant}")
        if variant == 0:
            has = lab != NONE
            assert np.array_equal(got[0][:, has], tr.counters[:, has])


@pytest.mark.parametrize("cid", [0, 1, 2])
def test_join_configs(ch, cid):
    say(f"join: config {cid}")
    tr = tg.make_config(cid)
    if tr.counters is None:
        rng = np.random.default_rng(cid)
        tr.counters = rng.integers(0, 1 << 40, size=(16, tr.n),
                                   dtype=np.uint64)
    r0 = oracle.run(tr)
    idx = r0["idx"].reshape(-1, tr.n)[0]
    lab = np.full(tr.n, NONE, np.uint32)
    lab[idx != NONE] = tr.m_label[idx[idx != NONE]]
    for variant in range(2):
        passes = tg.make_counter_passes(
            tr, lab, 7 + variant, drop_frac=0.01 * variant,
            mismatch_frac=0.01 * variant, extra=variant)
        got, ref, lab2 = join_both(ch, tr, passes)
        assert not ref[2] & oracle.JOIN_ORDER
        check(got, ref, f"config {cid} variant {variant}")
        if variant == 0:
            has = lab2 != NONE
            assert np.array_equal(got[0][:, has], tr.counters[:, has])
            assert (got[1][has] == 127).all()


def test_join_labels_out_of_order(ch):
    """Random iteration labels: labels split into several runs and
    decreasing along a stream (JOIN_ORDER, a warning); values exact."""
    say("join: labels out of order")
    tr = tg.make_micro(9, n_gpus=2, n_kernels=400, n_streams=2, depth=2,
                       span=6000, n_counters=16)
    r0 = oracle.run(tr)
    idx = r0["idx"].reshape(-1, tr.n)[0]
    lab = np.full(tr.n, NONE, np.uint32)
    lab[idx != NONE] = tr.m_label[idx[idx != NONE]]
    passes = tg.make_counter_passes(tr, lab, 1, cols=(4, 4))
    got, ref, _ = join_both(ch, tr, passes)
    assert ref[2] & oracle.JOIN_ORDER
    check(got, ref, "random labels")
    bad = tg.make_counter_passes(tr, lab, 3, cols=(4, 4), drop_frac=0.05,
                                 mismatch_frac=0.05, extra=4)
    got, ref, _ = join_both(ch, tr, bad)
    check(got, ref, "random labels, perturbed passes")


def test_join_label_split_by_unlabelled_kernels(ch):
    """Every iteration label increasing in time, but some kernels inside an
    iteration have no iteration marker: a label is then two runs on the
    record side only."""
    say("join: labels split by kernels without an iteration")
    tr = tg.make_config(0)
    rng = np.random.default_rng(5)
    tr.counters = rng.integers(0, 1 << 40, size=(16, tr.n), dtype=np.uint64)
    r0 = oracle.run(tr)
    idx = r0["idx"].reshape(-1, tr.n)[0]
    lab = np.full(tr.n, NONE, np.uint32)
    lab[idx != NONE] = tr.m_label[idx[idx != NONE]]
    passes = tg.make_counter_passes(tr, lab, 4)
    # the records lose their iteration here and there (the passes keep it)
    lab2 = lab.copy()
    holes = rng.choice(tr.n, size=40, replace=False)
    lab2[holes] = NONE
    import torch
    pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"))
    pipe.status.zero_()
    pipe.step()
    # drop the level-0 attribution of the hole records on the device
    r = pipe.results()
    idx_dev = pipe.idx.view(-1)[:tr.n]
    hole_t = torch.from_numpy(holes.astype(np.int64)).cuda()
    idx_dev.index_fill_(0, hole_t, -1)
    pipe.status.zero_()
    t = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a).view(dt)).cuda()
    dp = [dict(gpu=t(q["gpu"], np.uint8), stream=t(q["stream"], np.uint8),
               cls=t(q["cls"], np.uint8), label=t(q["lab"], np.int32),
               values=t(q["values"], np.int64), dst=q["dst"]) for q in passes]
    ctr, m = pipe.join_counters(dp)
    got = (ctr.cpu().numpy().view(np.uint64), m.cpu().numpy(),
           int(pipe.status.item()) & 0xFFFFFFFF)
    ref = oracle.join(tr.gpu, tr.stream, tr.cls, r["start"], lab2, passes)
    assert not ref[2] & oracle.JOIN_ORDER
    check(got, ref, "split labels")


def test_join_empty_pass(ch):
    say("join: a pass without entries")
    tr = tg.make_micro(4, n_gpus=2, n_kernels=300, depth=2, n_counters=16)
    r0 = oracle.run(tr)
    idx = r0["idx"].reshape(-1, tr.n)[0]
    lab = np.full(tr.n, NONE, np.uint32)
    lab[idx != NONE] = tr.m_label[idx[idx != NONE]]
    passes = tg.make_counter_passes(tr, lab, 2, cols=(3, 2))
    empty = dict(gpu=np.zeros(0, np.uint8), stream=np.zeros(0, np.uint8),
                 cls=np.zeros(0, np.uint8), lab=np.zeros(0, np.uint32),
                 values=np.zeros((2, 0), np.uint64), dst=[10, 11])
    got, ref, _ = join_both(ch, tr, passes + [empty])
    check(got, ref, "empty pass")


@pytest.mark.parametrize("variant", [0, 1])
def test_join_shuffled_records(ch, variant):
    """Records in shuffled input order (the adversarial trace's shape, five
    iterations): far from their sorted order, so the join gathers in sorted
    order through its stage; values, matched bits and status exact."""
    say(f"join: shuffled records, variant {variant}")
    tr = tg.make_config(4, iters=5)
    # the sorted order jumps far at most steps (what sends the join to its
    # sorted-order gather)
    order = np.lexsort((np.arange(tr.n), tr.start, tr.stream.astype(np.int64),
                        tr.gpu.astype(np.int64)))
    far = np.abs(np.diff(order.astype(np.int64))) > 4096
    assert far.mean() > 0.5, far.mean()
    r0 = oracle.run(tr)
    idx = r0["idx"].reshape(-1, tr.n)[0]
    lab = np.full(tr.n, NONE, np.uint32)
    lab[idx != NONE] = tr.m_label[idx[idx != NONE]]
    passes = tg.make_counter_passes(
        tr, lab, 11 + variant, drop_frac=0.01 * variant,
        mismatch_frac=0.01 * variant, extra=2 * variant)
    got, ref, lab2 = join_both(ch, tr, passes)
    check(got, ref, f"shuffled variant {variant}")
    if variant == 0:
        has = lab2 != NONE
        assert np.array_equal(got[0][:, has], tr.counters[:, has])


def test_join_shuffled_records_odd_width(ch):
    """The sorted-order gather with an odd number of value columns in all
    (rows of the stage not 16-byte aligned, copied back one value at a
    time), a pass with no entries among them."""
    say("join: shuffled records, five columns")
    tr = tg.make_config(4, iters=3)
    r0 = oracle.run(tr)
    idx = r0["idx"].reshape(-1, tr.n)[0]
    lab = np.full(tr.n, NONE, np.uint32)
    lab[idx != NONE] = tr.m_label[idx[idx != NONE]]
    passes = tg.make_counter_passes(tr, lab, 21, cols=(3, 2),
                                    drop_frac=0.02, mismatch_frac=0.01)
    empty = dict(gpu=np.zeros(0, np.uint8), stream=np.zeros(0, np.uint8),
                 cls=np.zeros(0, np.uint8), lab=np.zeros(0, np.uint32),
                 values=np.zeros((2, 0), np.uint64), dst=[9, 10])
    assert sum(q["values"].shape[0] for q in passes + [empty]) % 2 == 1
    got, ref, _ = join_both(ch, tr, passes + [empty])
    check(got, ref, "shuffled, seven columns")
