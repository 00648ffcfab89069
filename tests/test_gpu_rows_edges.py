"""Edge sizes of the rows' consumers: the overlap statistics and the launch
split on traces of 0, 1, 2 and 2049 records (one GPU, two marker levels,
two streams), checked against the oracle through the C ABI."""
import sys

import numpy as np
import pytest

import oracle
import tracegen as tg
from test_gpu_parity import _tiny

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


@pytest.mark.parametrize("n", [0, 1, 2, 2049])
def test_op_stats_edge_sizes(ch, n):
    say(f"op stats: {n} records")
    tr = _tiny(n, m=5)
    tr.m_label = (np.arange(tr.m_label.shape[0]) % 3).astype(np.uint32)
    pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"))
    pipe.status.zero_()
    pipe.step()
    out, cnt = pipe.op_stats(phase_level=0, op_level=1, n_phases=2, n_ops=4)
    go, gc = out.cpu().numpy(), cnt.cpu().numpy()
    ro, rc = oracle.op_stats(oracle.run(tr)["rows"], tr.m_label, tr.depth,
                             phase_level=0, op_level=1, n_phases=2, n_ops=4)
    assert np.array_equal(gc, rc)
    assert ((go == ro) | (np.isnan(go) & np.isnan(ro))).all()
    if n == 0:
        assert gc.sum() == 0


@pytest.mark.parametrize("n", [0, 1, 2, 2049])
def test_launch_split_edge_sizes(ch, n):
    import torch
    say(f"launch split: {n} records")
    tr = _tiny(n, m=5)
    pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"))
    pipe.step()
    tl = tg.make_launch(tr, 3, max_lead=100)
    prep, call = pipe.launch_split(torch.from_numpy(tl).cuda())
    r = oracle.run(tr)
    rp, rcall = oracle.launch_split(tr.gpu, tr.stream, tr.cls, r["start"],
                                    r["end"], tl)
    assert np.array_equal(prep.cpu().numpy(), rp)
    assert np.array_equal(call.cpu().numpy(), rcall)
