"""chopper_launch_split_noalloc (no scratch argument, the library's static
device table) against chopper_launch_split through the C ABI: bit-exact on
two calls in a row, the second with a smaller input (fewer records and fewer
GPUs), so that what the first call left in the static table must not leak
into the second."""
import sys

import numpy as np
import pytest

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


def both(ch, tr, lead):
    import torch
    pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"))
    pipe.status.zero_()
    pipe.step()
    tl = torch.from_numpy(tg.make_launch(tr, 11, max_lead=lead)).cuda()
    p0, c0 = pipe.launch_split(tl)
    p1, c1 = pipe.launch_split_noalloc(tl)
    torch.cuda.synchronize()
    return ((p0.cpu().numpy(), c0.cpu().numpy()),
            (p1.cpu().numpy(), c1.cpu().numpy()), pipe)


def test_noalloc_matches_scratch_variant_twice(ch):
    first = tg.make_config(1)                       # 8 GPUs, 245,760 records
    second = tg.make_micro(5, n_gpus=2, n_kernels=700, n_streams=2, depth=2,
                           anchors=4, span=8000)    # 2 GPUs, 700 records
    assert second.n < first.n and second.n_gpus < first.n_gpus
    for tr, lead in ((first, 20000), (second, 60)):
        say("noalloc launch split:", tr.name, tr.n, tr.n_gpus)
        (rp, rc), (gp, gc), pipe = both(ch, tr, lead)
        assert gp.shape == (tr.n,) and gc.shape == (tr.n,)
        assert np.array_equal(gp, rp), "prep"
        assert np.array_equal(gc, rc), "call"
        assert int(pipe.status.item()) & 0xFFFFFFFF == 0
