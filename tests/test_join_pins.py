"""Pins of the oracle's counter-pass join (Section III-A: counters from
serialized passes of two or three counters without valid timestamps;
Section III-B: alignment attaches them to the runtime trace) to a
hand-worked example, a dictionary join over (gpu, stream, iteration label,
ordinal), and the round trip: unperturbed passes give back the counters the
generator split into them."""
import numpy as np
import pytest

import oracle
import tracegen as tg

NONE = 0xFFFFFFFF


def _labels(tr, r, level=0):
    idx = r["idx"].reshape(-1, tr.n)[level]
    lab = np.full(tr.n, NONE, np.uint32)
    ok = idx != NONE
    lab[ok] = tr.m_label[idx[ok]]
    return lab


def test_join_hand_example():
    # GPU 0, streams 0 and 1, iterations 7 and 8; records (index: stream,
    # start, class, label): 0: (0, 10, GEMM, 7) 1: (1, 12, AG, 7)
    # 2: (0, 20, NORM, 7) 3: (0, 30, GEMM, 8) 4: (1, 31, RS, 8)
    gpu = np.zeros(5, np.uint8)
    stream = np.array([0, 1, 0, 0, 1], np.uint8)
    cls = np.array([0, 5, 3, 0, 6], np.uint8)
    s = np.array([10, 12, 20, 30, 31], np.int64)
    lab = np.array([7, 7, 7, 8, 8], np.uint32)
    # the pass lists stream 1 first, then stream 0, and has no entry for
    # record 3; record 2's entry carries another class
    p = dict(gpu=np.zeros(4, np.uint8), stream=np.array([1, 1, 0, 0], np.uint8),
             cls=np.array([5, 6, 0, 2], np.uint8),
             lab=np.array([7, 8, 7, 7], np.uint32),
             values=np.array([[101, 104, 100, 102], [201, 204, 200, 202]],
                             np.uint64), dst=[4, 9])
    ctr, m, st = oracle.join(gpu, stream, cls, s, lab, [p])
    assert ctr[4].tolist() == [100, 101, 0, 0, 104]
    assert ctr[9].tolist() == [200, 201, 0, 0, 204]
    assert m.tolist() == [1, 1, 0, 0, 1]
    assert st == oracle.JOIN_MISS
    assert int(ctr.sum()) == 100 + 101 + 104 + 200 + 201 + 204
    # a pass whose labels decrease along a stream: JOIN_ORDER (a warning)
    q = dict(p, lab=np.array([8, 7, 7, 7], np.uint32))
    assert oracle.join(gpu, stream, cls, s, lab, [q])[2] & oracle.JOIN_ORDER
    # records of one label split by a record without an iteration: labels
    # never decrease, no warning
    lab2 = np.array([7, 7, NONE, 7, 8], np.uint32)
    assert not oracle.join(gpu, stream, cls, s, lab2, [p])[2] & \
        oracle.JOIN_ORDER
    # a record without an iteration at the start of a stream is fine
    lab3 = np.array([NONE, 7, 7, 8, 8], np.uint32)
    assert not oracle.join(gpu, stream, cls, s, lab3, [p])[2] & \
        oracle.JOIN_ORDER


def test_join_hand_example_labels_out_of_order():
    # GPU 0, stream 0, records in time order with labels 7, 9, 7, 9, 7 and
    # classes GEMM, NORM, GEMM, GEMM, ELEM: the ordinals count earlier
    # records of the same label, whatever lies between them:
    #   record 0 (7, #0), 1 (9, #0), 2 (7, #1), 3 (9, #1), 4 (7, #2)
    gpu = np.zeros(5, np.uint8)
    stream = np.zeros(5, np.uint8)
    cls = np.array([0, 3, 0, 0, 2], np.uint8)
    s = np.array([10, 20, 30, 40, 50], np.int64)
    lab = np.array([7, 9, 7, 9, 7], np.uint32)
    # the pass lists label 9 first, then label 7 (entries in the pass's own
    # order: 9 #0, 9 #1, 7 #0, 7 #1, 7 #2); the entry 7 #1 has another class
    p = dict(gpu=np.zeros(5, np.uint8), stream=np.zeros(5, np.uint8),
             cls=np.array([3, 0, 0, 3, 2], np.uint8),
             lab=np.array([9, 9, 7, 7, 7], np.uint32),
             values=np.array([[901, 902, 701, 702, 703]], np.uint64), dst=[2])
    ctr, m, st = oracle.join(gpu, stream, cls, s, lab, [p])
    assert ctr[2].tolist() == [701, 901, 0, 902, 703]
    assert m.tolist() == [1, 1, 0, 1, 1]
    # labels decrease on both sides (9 -> 7): the warning, and one miss
    assert st == oracle.JOIN_ORDER | oracle.JOIN_MISS


def _dict_join(tr, s, lab, passes):
    n = tr.n
    ords, seen = {}, {}
    for k in sorted(range(n), key=lambda k: (int(s[k]), k)):
        if int(lab[k]) == NONE:
            continue
        key = (int(tr.gpu[k]), int(tr.stream[k]), int(lab[k]))
        ords[k] = key + (seen.get(key, 0),)
        seen[key] = seen.get(key, 0) + 1
    ctr = np.zeros((16, n), np.uint64)
    matched = np.zeros(n, np.uint8)
    for pi, p in enumerate(passes):
        table, seen = {}, {}
        for i in range(p["gpu"].shape[0]):
            key = (int(p["gpu"][i]), int(p["stream"][i]), int(p["lab"][i]))
            table[key + (seen.get(key, 0),)] = i
            seen[key] = seen.get(key, 0) + 1
        for k in range(n):
            if k not in ords:
                continue
            i = table.get(ords[k])
            if i is not None and int(p["cls"][i]) == int(tr.cls[k]):
                for c, d in enumerate(p["dst"]):
                    ctr[d, k] = p["values"][c, i]
                matched[k] |= 1 << pi
    return ctr, matched


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_join_round_trip_and_dict(seed):
    tr = tg.make_micro(seed, n_gpus=2, n_kernels=400, n_streams=3, depth=2,
                       span=8000, n_counters=16)
    r = oracle.run(tr)
    lab = _labels(tr, r)
    passes = tg.make_counter_passes(tr, lab, seed)
    ctr, m, st = oracle.join(tr.gpu, tr.stream, tr.cls, r["start"], lab,
                             passes)
    # unperturbed passes: every record with an iteration matched in every
    # pass, and the join gives back the counters that were split into the
    # passes, whatever the order of the random labels of these traces
    has = lab != NONE
    assert st & oracle.JOIN_MISS == 0
    assert (m[has] == (1 << len(passes)) - 1).all() and (m[~has] == 0).all()
    assert np.array_equal(ctr[:, has], tr.counters[:, has])
    # perturbed passes: the oracle equals a dictionary join
    bad = tg.make_counter_passes(tr, lab, seed + 10, drop_frac=0.02,
                                 mismatch_frac=0.02, extra=3)
    ctr, m, st = oracle.join(tr.gpu, tr.stream, tr.cls, r["start"], lab, bad)
    want_c, want_m = _dict_join(tr, r["start"], lab, bad)
    assert np.array_equal(ctr, want_c)
    assert np.array_equal(m, want_m)
    assert st & oracle.JOIN_MISS


def test_join_round_trip_config2():
    tr = tg.make_config(2)
    r = oracle.run(tr)
    lab = _labels(tr, r)
    passes = tg.make_counter_passes(tr, lab, 5)
    ctr, m, st = oracle.join(tr.gpu, tr.stream, tr.cls, r["start"], lab,
                             passes)
    assert st == 0                 # iteration labels increase with time
    # records before a GPU's first iteration marker (its first all_gather of
    # the pipeline fill) have no iteration and are not joined
    has = lab != NONE
    assert (~has).sum() <= tr.n_gpus
    assert (m[has] == 127).all() and (m[~has] == 0).all()
    assert np.array_equal(ctr[:, has], tr.counters[:, has])
    assert (ctr[:, ~has] == 0).all()
