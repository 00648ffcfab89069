"""Parity of chopper_launch_split (Section V-D eqs. 1-3) with the CPU oracle
through the C ABI, bit-exact: dispatch times aligned with the fitted clocks,
preparation and call overhead per record, and their per-row sums through
chopper_aggregate's counter columns."""
import sys

import numpy as np
import pytest

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


def split_both(ch, tr, tl):
    import torch
    pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"))
    pipe.status.zero_()
    pipe.step()
    prep, call = pipe.launch_split(torch.from_numpy(tl).cuda())
    got = (prep.cpu().numpy(), call.cpu().numpy())
    st = int(pipe.status.item()) & 0xFFFFFFFF
    r = pipe.results()
    x0, c, d, rc = oracle.fit(tr.a_gpu, tr.a_local, tr.a_ref, tr.n_gpus)
    tla, _ = oracle.transform(tr.gpu, tl, tr.n_gpus, x0, c, d)
    ref = oracle.launch_split(tr.gpu, tr.stream, tr.cls, r["start"], r["end"],
                              tla)
    return got, ref, st, r


CASES = [("micro", dict(seed=s, n_gpus=2, n_kernels=300 + 50 * s,
                        n_streams=1 + s % 3, depth=2, span=6000), 60)
         for s in range(4)] + [("config", 0, 20000), ("config", 1, 20000),
                               ("config", 2, 20000)]


@pytest.mark.parametrize("kind,arg,lead", CASES)
def test_launch_split_parity(ch, kind, arg, lead):
    say(f"launch split: {kind} {arg}")
    tr = tg.make_micro(**arg) if kind == "micro" else tg.make_config(arg)
    tl = tg.make_launch(tr, 7, max_lead=lead)
    (gp, gc), (rp, rc), st, r = split_both(ch, tr, tl)
    assert np.array_equal(gp, rp), "prep"
    assert np.array_equal(gc, rc), "call"
    assert np.array_equal(gp + gc, r["gap"]), "prep + call = bubble"
    assert st == r["status"]


def test_launch_split_sums_through_aggregate(ch):
    say("launch split: per-row sums as counter columns")
    import dataclasses
    tr = tg.make_config(1)
    tl = tg.make_launch(tr, 3, max_lead=20000)
    (gp, gc), (rp, rc), _, _ = split_both(ch, tr, tl)
    assert np.array_equal(gp, rp) and np.array_equal(gc, rc)
    ctr = np.stack([gp, gc]).astype(np.int64).view(np.uint64)
    tr2 = dataclasses.replace(tr, counters=ctr)
    pipe = ch.Pipeline(ch.DeviceTrace(tr2, "cuda"))
    pipe.status.zero_()
    pipe.step()
    got = pipe.results()["rows"]
    ref = oracle.run(tr2)["rows"]
    assert np.array_equal(got["level_offset"], ref["level_offset"])
    assert np.array_equal(got["ctr"], ref["ctr"])
    assert np.array_equal(got["ctr"][0] + got["ctr"][1],
                          got["gap"].view(np.uint64))


def test_launch_split_range(ch):
    say("launch split: out-of-range dispatch time")
    tr = tg.make_micro(5, n_gpus=2, n_kernels=100, depth=2)
    tl = tg.make_launch(tr, 1, max_lead=30)
    tl[7] = 1 << 62
    (gp, gc), (rp, rc), st, r = split_both(ch, tr, tl)
    assert st & 16
    assert np.array_equal(gp + gc, r["gap"])
