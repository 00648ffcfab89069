"""Pins of the oracle's launch-overhead split (Section V-D eqs. 1-3) to the
equations themselves, evaluated here record by record with a linear search
for the previous compute kernel, and to the bubble of the overlap oracle."""
import numpy as np
import pytest

import oracle
import tracegen as tg


def _eqs(tr, s, e, tl):
    """eqs. 1-2 literally, the previous compute kernel of the same (gpu,
    stream) found by scanning all records (largest (start', index) before)."""
    n = s.shape[0]
    prep = np.zeros(n, np.int64)
    call = np.zeros(n, np.int64)
    comp = ~np.isin(tr.cls, [5, 6])
    for i in range(n):
        if not comp[i]:
            continue
        best = None
        for p in range(n):
            if (p != i and comp[p] and tr.gpu[p] == tr.gpu[i]
                    and tr.stream[p] == tr.stream[i]
                    and (s[p], p) < (s[i], i)
                    and (best is None or (s[p], p) > (s[best], best))):
                best = p
        if best is None or s[i] - e[best] <= 0:
            continue
        o_prep = max(int(tl[i]) - int(e[best]), 0)
        o_call = min(int(s[i]) - int(tl[i]), int(s[i]) - int(e[best]))
        if tl[i] > s[i]:                  # dispatched after the start
            o_prep, o_call = int(s[i]) - int(e[best]), 0
        prep[i], call[i] = o_prep, o_call
    return prep, call


def test_launch_hand_example():
    # one stream: kernels [0,10), [15,20), [20,30), [50,60); dispatches at
    # -5 (first kernel), 12 (bubble 5: 2 ns of preparation, 3 of call), 14
    # (abutting: no bubble), 35 (bubble 20 after the communication kernel is
    # skipped: 5 of preparation, 15 of call)
    gpu = np.zeros(5, np.uint8)
    stream = np.array([0, 0, 0, 1, 0], np.uint8)
    cls = np.array([0, 2, 0, 5, 1], np.uint8)
    s = np.array([0, 15, 20, 22, 50], np.int64)
    e = np.array([10, 20, 30, 40, 60], np.int64)
    tl = np.array([-5, 12, 14, 0, 35], np.int64)
    prep, call = oracle.launch_split(gpu, stream, cls, s, e, tl)
    assert prep.tolist() == [0, 2, 0, 0, 5]
    assert call.tolist() == [0, 3, 0, 0, 15]
    # dispatched after its start (clock noise): the whole bubble is
    # preparation
    tl2 = tl.copy()
    tl2[4] = 52
    prep, call = oracle.launch_split(gpu, stream, cls, s, e, tl2)
    assert prep[4] == 20 and call[4] == 0


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_launch_equations_and_bubble(seed):
    tr = tg.make_micro(seed, n_gpus=2, n_kernels=160, n_streams=2, depth=2,
                       span=3000)
    r = oracle.run(tr)
    tl = tg.make_launch(tr, seed, max_lead=80, late_frac=0.05)
    prep, call = oracle.launch_split(tr.gpu, tr.stream, tr.cls, r["start"],
                                     r["end"], tl)
    want_p, want_c = _eqs(tr, r["start"], r["end"], tl)
    assert prep.tolist() == want_p.tolist()
    assert call.tolist() == want_c.tolist()
    # eq. 3: the two parts add up to the bubble of the overlap oracle
    assert (prep + call).tolist() == r["gap"].tolist()
    assert (prep >= 0).all() and (call >= 0).all()
    # both cases occur: dispatched before and after the previous end
    assert (prep > 0).any() and ((call > 0) & (prep == 0)).any()
