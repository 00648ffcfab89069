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


def monotone_iterations(tr):
    """Level-0 labels increasing with start on every GPU."""
    lab = tr.m_label.copy()
    for g in range(tr.n_gpus):
        sel = np.nonzero((tr.m_gpu == g) & (tr.m_level == 0))[0]
        sel = sel[np.argsort(tr.m_start[sel], kind="stable")]
        lab[sel] = np.arange(sel.shape[0], dtype=np.uint32) * 3 + 5
    tr.m_label = lab
    return tr


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
    if rs & oracle.JOIN_ORDER:
        # the result (misses included) is unspecified then; the flag is not
        assert gs & oracle.JOIN_ORDER, (name, gs, rs)
        return
    assert gs == rs, (name, gs, rs)
    assert np.array_equal(gm, rm), name
    if not np.array_equal(gc, rc):
        d = np.nonzero((gc != rc).reshape(-1))[0]
        raise AssertionError(f"{name}: {d.size} counter differences, first "
                             f"at {d[0]}")


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_join_micro(ch, seed):
    say(f"join: micro seed {seed}")
    tr = monotone_iterations(tg.make_micro(
        seed, n_gpus=2 + seed % 2, n_kernels=500 + 100 * seed,
        n_streams=1 + seed % 3, depth=2, span=9000, n_counters=16,
        drop_frac=0.0))
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
        if variant == 0 and not ref[2] & oracle.JOIN_ORDER:
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


def test_join_order_flag(ch):
    say("join: labels out of order")
    tr = tg.make_micro(9, n_gpus=2, n_kernels=400, n_streams=2, depth=2,
                       span=6000, n_counters=16)
    r0 = oracle.run(tr)
    idx = r0["idx"].reshape(-1, tr.n)[0]
    lab = np.full(tr.n, NONE, np.uint32)
    lab[idx != NONE] = tr.m_label[idx[idx != NONE]]
    passes = tg.make_counter_passes(tr, lab, 1, cols=(4, 4))
    got, ref, _ = join_both(ch, tr, passes)
    check(got, ref, "random labels")


def test_join_empty_pass(ch):
    say("join: a pass without entries")
    tr = monotone_iterations(tg.make_micro(4, n_gpus=2, n_kernels=300,
                                           depth=2, n_counters=16))
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
