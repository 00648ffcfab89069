"""Parity of chopper_op_stats (overlap statistics and overhead breakdown of
operations: Fig. gemm_overlap, Section VI eqs. 6-10) with the CPU oracle
through the C ABI: instance counts bit-exact and every statistic equal as a
double (NaN matching NaN) -- both sides take the same IEEE operations on
the same exact integer moments and order statistics."""
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


def stats_both(ch, tr, **spec):
    pipe = ch.Pipeline(ch.DeviceTrace(tr, "cuda"))
    pipe.status.zero_()
    pipe.step()
    out, cnt, gout, gcnt = pipe.op_stats(per_gpu=True, **spec)
    got = (out.cpu().numpy(), cnt.cpu().numpy(),
           int(pipe.status.item()) & 0xFFFFFFFF, gout.cpu().numpy(),
           gcnt.cpu().numpy())
    ref = oracle.op_stats(oracle.run(tr)["rows"], tr.m_label, tr.depth,
                          n_gpus=tr.n_gpus, per_gpu=True, **spec)
    return got, ref


def _same_doubles(a, b, names, name):
    same = (a == b) | (np.isnan(a) & np.isnan(b))
    if not same.all():
        k, g = np.argwhere(~same)[0]
        raise AssertionError(f"{name}: {names[k]} of group {g}: "
                             f"{a[k, g]!r} vs {b[k, g]!r}")


def check(got, ref, name):
    go, gc, _, gg, ggc = got
    ro, rc, rg, rgc = ref
    assert np.array_equal(gc, rc), name
    _same_doubles(go, ro, oracle.OP_STATS, name)
    # the per-GPU overlap CDFs behind eq. 9
    assert np.array_equal(ggc, rgc), name + " per-GPU counts"
    _same_doubles(gg, rg, oracle.OP_CDF, name + " per GPU")
    assert ggc.sum() <= gc.sum()


@pytest.mark.parametrize("cid", [0, 1, 2])
def test_stats_configs(ch, cid):
    say(f"op stats: config {cid}")
    tr = tg.make_config(cid)
    fg = np.linspace(1e8, 9e9, 64)
    got, ref = stats_both(ch, tr, n_phases=3, n_ops=64, freq_peak_mhz=2100.0,
                          tpt_peak=1.3e6, f_gemm=fg)
    check(got, ref, f"config {cid}")
    assert got[1].sum() > 0 and np.isfinite(got[0][0]).any()


def test_stats_no_gemm_flops(ch):
    say("op stats: config 2 without per-operation FLOPs")
    got, ref = stats_both(ch, tg.make_config(2))
    check(got, ref, "config 2, f_gemm NULL")
    assert np.isnan(got[0][13]).all() and np.isnan(got[0][16]).all()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_stats_micro(ch, seed):
    say(f"op stats: micro seed {seed}")
    tr = tg.make_micro(seed, n_gpus=3, n_kernels=900, n_streams=3, depth=3,
                       span=12000, n_counters=16 if seed != 1 else 0)
    # few labels, so that groups hold several instances
    tr.m_label = (tr.m_label % (3 + seed)).astype(tr.m_label.dtype)
    got, ref = stats_both(ch, tr, phase_level=1, op_level=2, n_phases=16,
                          n_ops=50)
    check(got, ref, f"micro {seed}")
    assert got[1].max() >= 2


def test_stats_max_groups(ch):
    say("op stats: 16 phases x 128 operations, labels past both limits")
    tr = tg.make_micro(7, n_gpus=4, n_kernels=3000, n_streams=2, depth=3,
                       span=30000, n_counters=16)
    rng = np.random.default_rng(7)
    top = np.where(tr.m_level == 0, 18, 135)
    tr.m_label = (rng.random(tr.m_label.shape[0]) * top).astype(
        tr.m_label.dtype)
    got, ref = stats_both(ch, tr, phase_level=0, op_level=2, n_phases=16,
                          n_ops=128, f_gemm=np.arange(1, 129) * 1e9)
    check(got, ref, "16 x 128")
    assert got[1].sum() > 0


def test_stats_no_instances(ch):
    say("op stats: every operation label out of range")
    tr = tg.make_micro(8, n_gpus=2, n_kernels=400, depth=3, span=5000)
    tr.m_label = np.full_like(tr.m_label, 200)
    got, ref = stats_both(ch, tr, phase_level=1, op_level=2, n_phases=2,
                          n_ops=8)
    check(got, ref, "no instances")
    assert got[1].sum() == 0 and np.isnan(got[0]).all()
