"""Seeded synthetic inputs for the trace pipeline: kernel records, annotation
markers and clock anchors.

The traces imitate what runtime and hardware profiling collect from an
eight-GPU FSDP training run of Llama 3 8B (paper: Section III-A for what a
trace holds; Table "llm_config" for 32 layers; caption of Fig. "transformer"
for the operation names; Section II-B for the all-gather / reduce-scatter
pattern).  The paper's own traces are not available, so these stand in for
them.

This module only *creates* inputs.  It holds none of the analysis: no clock
fit, no attribution, no overlap sweep, no aggregation.  Both the CPU oracle and
the HIP library consume exactly the arrays produced here.

Layout (structure of arrays, one entry per record / marker / anchor):

records  gpu u8, stream u8, start i64, end i64 (ns, the GPU's local clock),
         cls u8 (0 GEMM, 1 attention, 2 elementwise, 3 RMSNorm, 4 RoPE,
         5 all_gather, 6 reduce_scatter, 7 optimizer), op_id u32,
         counters u64[n_counters][n] (counter-major)
markers  gpu u8, level u8 (0 iteration, 1 phase, 2 layer, 3 op, 4-5 sub-op),
         start i64, end i64 (local clock), label u32
anchors  gpu u8, local i64, ref i64 (host-side pairs of the same instant)
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional

import numpy as np

# ----------------------------------------------------------------------------
# Vocabulary
# ----------------------------------------------------------------------------
GEMM, ATTN, ELEM, NORM, ROPE, ALL_GATHER, REDUCE_SCATTER, OPTIM = range(8)
CLASS_NAMES = ["gemm", "attention", "elementwise", "rmsnorm", "rope",
               "all_gather", "reduce_scatter", "optimizer"]
COMM_CLASSES = (ALL_GATHER, REDUCE_SCATTER)

# Per-layer operations of the forward pass in execution order:
# (name, class, kernels).  6 GEMM kernels, 1 attention, 2 norms, 1 RoPE and
# 4 elementwise kernels per layer.
FWD_OPS = [
    ("attn_n", NORM, 1), ("qkv_ip", GEMM, 2), ("qkv_re", ROPE, 1),
    ("attn_fa", ATTN, 1), ("attn_op", GEMM, 1), ("attn_ra", ELEM, 1),
    ("mlp_n", NORM, 1), ("mlp_gp", GEMM, 1), ("mlp_gs", ELEM, 1),
    ("mlp_up", GEMM, 1), ("mlp_gu", ELEM, 1), ("mlp_dp", GEMM, 1),
    ("mlp_ra", ELEM, 1),
]
# Operation labels (op_id of a compute record == label of its op marker).
FWD_LABEL0, BWD_LABEL0 = 0, 16
LABEL_B_GA, LABEL_OPT_STEP = 32, 33
LABEL_ALL_GATHER, LABEL_REDUCE_SCATTER = 40, 41


def op_label_name(label: int) -> str:
    if FWD_LABEL0 <= label < FWD_LABEL0 + len(FWD_OPS):
        return "f_" + FWD_OPS[label - FWD_LABEL0][0]
    if BWD_LABEL0 <= label < BWD_LABEL0 + len(FWD_OPS):
        return "b_" + FWD_OPS[label - BWD_LABEL0][0]
    return {LABEL_B_GA: "b_ga", LABEL_OPT_STEP: "opt_step",
            LABEL_ALL_GATHER: "all_gather",
            LABEL_REDUCE_SCATTER: "reduce_scatter"}.get(label, "?")


# Arithmetic mean kernel durations in ns; backward compute is twice as long.
MEAN_NS = {GEMM: 400_000, ATTN: 300_000, ELEM: 20_000, NORM: 30_000,
           ROPE: 20_000, OPTIM: 5_000}
DUR_SIGMA = 0.3
GAP_MEAN_NS = 5_000.0
BWD_SCALE = 2.0

N_COUNTERS = 16
COUNTER_NAMES = ["GPU_CYCLES", "MFMA_BUSY", "VALU_BUSY", "SALU_BUSY",
                 "HBM_RD_BYTES", "HBM_WR_BYTES", "L2_HIT", "L2_MISS",
                 "LDS_BANK_CONFLICT", "LDS_INSTS", "VMEM_INSTS", "MFMA_FLOPS",
                 "WAVES", "SCLK_MHZ", "MCLK_MHZ", "POWER_W"]
# Per-class rate (events per microsecond of kernel time) of counters 1..12.
_RATE = np.array([
    # MFMA  VALU  SALU  RD      WR      L2H   L2M   LDSC  LDSI  VMEM  FLOP     WAVES
    [1500,  300,  50,   2.0e6,  6.0e5,  4e3,  1e3,  20,   600,  300,  1.0e9,   40],   # GEMM
    [900,   900,  80,   1.5e6,  4.0e5,  3e3,  8e2,  60,   900,  400,  6.0e8,   30],   # attention
    [0,     1500, 60,   3.5e6,  3.5e6,  1e3,  3e3,  0,    10,   900,  0.0,     60],   # elementwise
    [0,     1400, 70,   3.0e6,  2.5e6,  1e3,  2e3,  5,    200,  800,  0.0,     50],   # RMSNorm
    [0,     1300, 60,   3.0e6,  3.0e6,  1e3,  2e3,  0,    50,   800,  0.0,     50],   # RoPE
    [0,     200,  40,   4.0e6,  4.0e6,  5e2,  4e3,  0,    0,    700,  0.0,     20],   # all_gather
    [0,     600,  40,   4.0e6,  4.0e6,  5e2,  4e3,  0,    0,    700,  0.0,     20],   # reduce_scatter
    [0,     1200, 90,   2.5e6,  2.5e6,  1e3,  2e3,  0,    0,    600,  0.0,     30],   # optimizer
], dtype=np.float64)

BASE_REF_NS = 1_700_000_000_000_000_000  # epoch-scale timestamps


@dataclasses.dataclass
class Trace:
    n_gpus: int
    depth: int
    # records
    gpu: np.ndarray
    stream: np.ndarray
    start: np.ndarray
    end: np.ndarray
    cls: np.ndarray
    op_id: np.ndarray
    counters: Optional[np.ndarray]          # u64 [C, N] or None
    # markers
    m_gpu: np.ndarray
    m_level: np.ndarray
    m_start: np.ndarray
    m_end: np.ndarray
    m_label: np.ndarray
    # anchors
    a_gpu: np.ndarray
    a_local: np.ndarray
    a_ref: np.ndarray
    # generator ground truth (reference-clock record times), not a method input
    truth: Dict[str, np.ndarray] = dataclasses.field(default_factory=dict)
    name: str = ""

    @property
    def n(self) -> int:
        return int(self.gpu.shape[0])

    @property
    def n_markers(self) -> int:
        return int(self.m_gpu.shape[0])

    @property
    def n_counters(self) -> int:
        return 0 if self.counters is None else int(self.counters.shape[0])

    def nbytes(self) -> int:
        tot = 0
        for f in dataclasses.fields(self):
            v = getattr(self, f.name)
            if isinstance(v, np.ndarray):
                tot += v.nbytes
        return tot


CONFIGS = {
    0: dict(seed=0, n_gpus=1, iters=2, layers=4, k_opt=220, compute_streams=1,
            split_comm=False, offset_ns=0, drift_ppm=0.0, anchors_per_iter=0,
            counters=0, zero_frac=0.0, abut_frac=0.0, u_lo=0.3, u_hi=0.7,
            depth_lo=4, depth_hi=4, drop_frac=0.0, shuffle=False),
    1: dict(seed=1, n_gpus=8, iters=10, layers=32, k_opt=66, compute_streams=1,
            split_comm=False, offset_ns=50_000, drift_ppm=20.0,
            anchors_per_iter=4, counters=0, zero_frac=0.0, abut_frac=0.0,
            u_lo=0.3, u_hi=0.7, depth_lo=4, depth_hi=4, drop_frac=0.0,
            shuffle=False),
    2: dict(seed=2, n_gpus=8, iters=100, layers=32, k_opt=66,
            compute_streams=1, split_comm=False, offset_ns=50_000,
            drift_ppm=20.0, anchors_per_iter=4, counters=16, zero_frac=0.0,
            abut_frac=0.0, u_lo=0.3, u_hi=0.7, depth_lo=4, depth_hi=4,
            drop_frac=0.0, shuffle=False),
    3: dict(seed=3, n_gpus=8, iters=800, layers=32, k_opt=66,
            compute_streams=1, split_comm=False, offset_ns=50_000,
            drift_ppm=20.0, anchors_per_iter=4, counters=16, zero_frac=0.0,
            abut_frac=0.0, u_lo=0.3, u_hi=0.7, depth_lo=4, depth_hi=4,
            drop_frac=0.0, shuffle=False),
    4: dict(seed=4, n_gpus=8, iters=2035, layers=32, k_opt=66,
            compute_streams=2, split_comm=True, offset_ns=5_000_000,
            drift_ppm=200.0, anchors_per_iter=4, counters=16, zero_frac=0.05,
            abut_frac=0.05, u_lo=0.3, u_hi=1.0, depth_lo=3, depth_hi=6,
            drop_frac=0.01, shuffle=True),
}

CONFIG_NAMES = {
    0: "tiny: 1 GPU x 2 iterations x 4 layers, no skew, no counters",
    1: "8 GPUs x 10 iterations x 32 layers, clock skew, no counters",
    2: "8 GPUs x 100 iterations x 32 layers, 16 counters",
    3: "8 GPUs x 800 iterations x 32 layers, 16 counters (headline)",
    4: "adversarial: 8 GPUs x 2035 iterations x 32 layers, 4 streams, "
       "shuffled, depth 3-6",
}


def expected_size(cid: int, iters: Optional[int] = None) -> int:
    c = CONFIGS[cid]
    it = c["iters"] if iters is None else iters
    return c["n_gpus"] * it * c["layers"] * (30 + c["k_opt"])


# ----------------------------------------------------------------------------
# Per-iteration kernel template
# ----------------------------------------------------------------------------
def _iteration_template(layers: int, k_opt: int):
    """Compute kernels of one iteration, grouped in layer blocks.

    Returns a list of blocks in execution order; each block is a dict with
    arrays over its kernels: cls, label, mean_ns, op (op index inside the
    block), and scalars phase, layer.
    """
    blocks = []
    fwd_cls, fwd_lab, fwd_op = [], [], []
    for j, (_, c, nk) in enumerate(FWD_OPS):
        for _ in range(nk):
            fwd_cls.append(c)
            fwd_lab.append(FWD_LABEL0 + j)
            fwd_op.append(j)
    bwd_cls, bwd_lab, bwd_op = [], [], []
    for jj, j in enumerate(reversed(range(len(FWD_OPS)))):
        _, c, nk = FWD_OPS[j]
        for _ in range(nk):
            bwd_cls.append(c)
            bwd_lab.append(BWD_LABEL0 + j)
            bwd_op.append(jj)
    opt_cls = [OPTIM] * k_opt
    opt_lab = [LABEL_B_GA] * 3 + [LABEL_OPT_STEP] * (k_opt - 3)
    opt_op = [0] * 3 + [1] * (k_opt - 3)

    def mk(cls, lab, op, phase, scale):
        cls = np.asarray(cls, np.uint8)
        mean = np.array([MEAN_NS[int(c)] for c in cls], np.float64) * scale
        return dict(cls=cls, label=np.asarray(lab, np.uint32),
                    op=np.asarray(op, np.int64), mean=mean, phase=phase)

    fwd = mk(fwd_cls, fwd_lab, fwd_op, 0, 1.0)
    bwd = mk(bwd_cls, bwd_lab, bwd_op, 1, BWD_SCALE)
    opt = mk(opt_cls, opt_lab, opt_op, 2, 1.0)
    for phase, tpl in ((0, fwd), (1, bwd), (2, opt)):
        for b in range(layers):
            layer = (layers - 1 - b) if phase == 1 else b
            blocks.append((phase, layer, tpl))
    return blocks, (fwd, bwd, opt)


def _lognormal_int(rng, mean, sigma, size):
    mu = np.log(mean) - 0.5 * sigma * sigma
    return np.rint(rng.lognormal(mu, sigma, size=size)).astype(np.int64)


def _block_times(rng, tpl, n_blocks, n_streams, zero_frac, abut_frac):
    """Kernel offsets inside n_blocks repetitions of one block template.

    Kernel j of a block runs on compute stream j % n_streams; each stream is a
    sequential timeline starting at the block base.  Returns (start_off,
    end_off, stream, span) with shapes (n_blocks, k) and (n_blocks,).
    """
    k = tpl["cls"].shape[0]
    dur = _lognormal_int(rng, tpl["mean"][None, :].repeat(n_blocks, 0),
                         DUR_SIGMA, (n_blocks, k))
    gap = np.rint(rng.exponential(GAP_MEAN_NS, size=(n_blocks, k))
                  ).astype(np.int64)
    if zero_frac > 0:
        dur[rng.random((n_blocks, k)) < zero_frac] = 0
    if abut_frac > 0:
        gap[rng.random((n_blocks, k)) < abut_frac] = 0
    s_off = np.empty_like(dur)
    e_off = np.empty_like(dur)
    span = np.zeros(n_blocks, np.int64)
    stream = (np.arange(k) % n_streams).astype(np.uint8)
    for s in range(n_streams):
        cols = np.arange(s, k, n_streams)
        if cols.size == 0:
            continue
        e = np.cumsum(gap[:, cols] + dur[:, cols], axis=1)
        e_off[:, cols] = e
        s_off[:, cols] = e - dur[:, cols]
        span = np.maximum(span, e[:, -1])
    return s_off, e_off, stream, span


def _gpu_timeline(rng, cfg, base_ref):
    """All kernels and markers of one GPU in the reference clock."""
    L, I = cfg["layers"], cfg["iters"]
    S = cfg["compute_streams"]
    blocks, (fwd, bwd, opt) = _iteration_template(L, cfg["k_opt"])
    tpls = (fwd, bwd, opt)
    # times per phase type: arrays (I, L, k)
    per = []
    for tpl in tpls:
        s_off, e_off, stream, span = _block_times(
            rng, tpl, I * L, S, cfg["zero_frac"], cfg["abut_frac"])
        k = tpl["cls"].shape[0]
        per.append((s_off.reshape(I, L, k), e_off.reshape(I, L, k), stream,
                    span.reshape(I, L)))
    # block bases: execution order per iteration is fwd L, bwd L, opt L
    spans = np.concatenate([per[0][3], per[1][3], per[2][3]], axis=1)  # (I,3L)
    lead_gap = np.rint(rng.exponential(GAP_MEAN_NS, size=spans.shape)
                       ).astype(np.int64)
    flat = (spans + lead_gap).reshape(-1)
    bases = base_ref + np.concatenate([[0], np.cumsum(flat)[:-1]]) \
        + lead_gap.reshape(-1)
    bases = bases.reshape(I, 3, L)

    comp = dict(start=[], end=[], stream=[], cls=[], label=[])
    # op boundaries per (iteration, phase, layer-block, op)
    op_first = []      # list per phase of (I, L, n_ops) min starts
    for p, tpl in enumerate(tpls):
        s_off, e_off, stream, _ = per[p]
        b = bases[:, p, :][:, :, None]
        st = b + s_off
        en = b + e_off
        k = tpl["cls"].shape[0]
        comp["start"].append(st.reshape(-1))
        comp["end"].append(en.reshape(-1))
        comp["stream"].append(np.broadcast_to(stream, (I, L, k)).reshape(-1))
        comp["cls"].append(np.broadcast_to(tpl["cls"], (I, L, k)).reshape(-1))
        comp["label"].append(np.broadcast_to(tpl["label"], (I, L, k)
                                             ).reshape(-1))
        n_ops = int(tpl["op"].max()) + 1
        first = np.full((I, L, n_ops), np.iinfo(np.int64).max, np.int64)
        for o in range(n_ops):
            cols = np.nonzero(tpl["op"] == o)[0]
            first[:, :, o] = st[:, :, cols].min(axis=2)
        op_first.append(first)
    for key in comp:
        comp[key] = np.concatenate(comp[key])
    comp_end_max = int(comp["end"].max())

    # ---------------- communication kernels -------------------------------
    # One all-gather per layer in the forward phase and one reduce-scatter per
    # layer in the backward phase.  The k-th comm kernel of a phase starts
    # uniformly inside the compute window of block k-1 (block 0: at the phase
    # start) and lasts u * that window; kernels on one stream serialize.
    win_s = np.stack([bases[:, p, :] for p in range(3)], axis=1)  # (I,3,L)
    win_len = np.stack([per[p][3] for p in range(3)], axis=1)
    u = rng.uniform(cfg["u_lo"], cfg["u_hi"], size=(I, 2, L))
    pos = rng.random(size=(I, 2, L))
    c_start, c_end, c_stream, c_cls, c_lab = [], [], [], [], []
    if cfg["split_comm"]:
        stream_of = {0: 2, 1: 3}
    else:
        stream_of = {0: 1, 1: 1}
    free = {1: -(1 << 62), 2: -(1 << 62), 3: -(1 << 62)}
    ws = win_s.tolist()
    wl = win_len.tolist()
    ul = u.tolist()
    pl = pos.tolist()
    for i in range(I):
        for p in range(2):
            st_id = stream_of[p]
            for k in range(L):
                kk = max(k - 1, 0)
                w0 = ws[i][p][kk]
                wlen = wl[i][p][kk]
                s = w0 if k == 0 else w0 + int(pl[i][p][k] * wlen)
                s = max(s, free[st_id])
                d = int(round(ul[i][p][k] * wlen))
                c_start.append(s)
                c_end.append(s + d)
                free[st_id] = s + d
                c_stream.append(st_id)
                c_cls.append(ALL_GATHER if p == 0 else REDUCE_SCATTER)
                c_lab.append(LABEL_ALL_GATHER if p == 0
                             else LABEL_REDUCE_SCATTER)
    comm = dict(start=np.asarray(c_start, np.int64),
                end=np.asarray(c_end, np.int64),
                stream=np.asarray(c_stream, np.uint8),
                cls=np.asarray(c_cls, np.uint8),
                label=np.asarray(c_lab, np.uint32))

    # ---------------- markers (tiling, nested) -----------------------------
    # Op boundaries in execution order: running maximum of each op's first
    # kernel start; an op marker runs to the next op's boundary.
    per_iter_ops = []
    op_phase, op_layer, op_lab = [], [], []
    for p, tpl in enumerate(tpls):
        n_ops = op_first[p].shape[2]
        per_iter_ops.append(op_first[p].reshape(I, L * n_ops))
        labs = []
        for o in range(n_ops):
            cols = np.nonzero(tpl["op"] == o)[0]
            labs.append(int(tpl["label"][cols[0]]))
        for b in range(L):
            layer = (L - 1 - b) if p == 1 else b
            for o in range(n_ops):
                op_phase.append(p)
                op_layer.append(layer)
                op_lab.append(labs[o])
    ops_per_iter = sum(x.shape[1] for x in per_iter_ops)
    first_all = np.concatenate(per_iter_ops, axis=1).reshape(-1)
    bnd = np.maximum.accumulate(first_all)
    bnd_next = np.concatenate([bnd[1:], [max(comp_end_max, int(bnd[-1]))]])
    op_phase = np.asarray(op_phase, np.int64)
    op_layer = np.asarray(op_layer, np.int64)
    op_lab = np.asarray(op_lab, np.uint32)
    B = bnd.reshape(I, ops_per_iter)
    Bn = bnd_next.reshape(I, ops_per_iter)
    # index of the first op of each phase / layer block within an iteration
    n_ops_ph = [per_iter_ops[p].shape[1] for p in range(3)]
    ph_first = np.cumsum([0] + n_ops_ph[:-1])
    ph_last = ph_first + np.asarray(n_ops_ph) - 1
    mk = dict(level=[], start=[], end=[], label=[], it=[])

    def add(level, s, e, lab, it):
        mk["level"].append(np.full(s.shape, level, np.uint8))
        mk["start"].append(s)
        mk["end"].append(e)
        mk["label"].append(np.asarray(lab, np.uint32))
        mk["it"].append(it)

    its = np.arange(I)
    # iteration markers
    add(0, B[:, 0], Bn[:, -1], its.astype(np.uint32), its)
    for p in range(3):
        add(1, B[:, ph_first[p]], Bn[:, ph_last[p]],
            np.full(I, p, np.uint32), its)
    for p in range(3):
        n_ops = n_ops_ph[p] // L
        for b in range(L):
            f = ph_first[p] + b * n_ops
            layer = (L - 1 - b) if p == 1 else b
            add(2, B[:, f], Bn[:, f + n_ops - 1],
                np.full(I, layer, np.uint32), its)
    add(3, B.reshape(-1), Bn.reshape(-1),
        np.tile(op_lab, I), np.repeat(its, ops_per_iter))
    markers = {k: np.concatenate(v) for k, v in mk.items()}
    iter_bounds = (B[:, 0].copy(), Bn[:, -1].copy())
    return comp, comm, markers, iter_bounds


def _sub_splits(rng, level, s, e, pieces_max, it):
    """Split each marker [s, e) into 1..pieces_max consecutive pieces."""
    n = s.shape[0]
    k = rng.integers(1, pieces_max + 1, size=n)
    length = e - s
    cuts = np.sort(rng.random((n, pieces_max - 1)), axis=1)
    cut_pts = s[:, None] + np.floor(cuts * length[:, None]).astype(np.int64)
    out_s, out_e, out_l, out_it = [], [], [], []
    for kk in range(1, pieces_max + 1):
        sel = np.nonzero(k == kk)[0]
        if sel.size == 0:
            continue
        # use the first kk-1 cuts of the sorted set
        pts = np.concatenate([s[sel, None], cut_pts[sel, :kk - 1],
                              e[sel, None]], axis=1)
        pts = np.sort(pts, axis=1)
        for q in range(kk):
            out_s.append(pts[:, q])
            out_e.append(pts[:, q + 1])
            out_l.append(np.full(sel.size, q, np.uint32))
            out_it.append(it[sel])
    if not out_s:
        z = np.zeros(0, np.int64)
        return z, z, np.zeros(0, np.uint32), z
    return (np.concatenate(out_s), np.concatenate(out_e),
            np.concatenate(out_l), np.concatenate(out_it))


def _to_local(t, off, drift_ppm, t0):
    """Reference clock -> a GPU's local clock: offset plus linear drift."""
    if drift_ppm == 0.0 and off == 0:
        return t.copy()
    rel = (t - t0).astype(np.float64)
    return t + off + np.rint(rel * (drift_ppm * 1e-6)).astype(np.int64)


def _counters(rng, cls, dur, n_counters):
    """16 hardware counters per record: cycles from duration and SCLK, clock
    and power samples, and class-dependent lognormal event counts."""
    n = cls.shape[0]
    out = np.empty((n_counters, n), np.uint64)
    sclk = rng.integers(1300, 2101, size=n, dtype=np.int64)
    mclk = rng.integers(900, 1301, size=n, dtype=np.int64)
    power = rng.integers(300, 751, size=n, dtype=np.int64)
    cols = {0: (dur * sclk // 1000), 13: sclk, 14: mclk, 15: power}
    dur_us = (dur.astype(np.float32) * np.float32(1e-3))
    rate = _RATE.astype(np.float32)
    for j in range(min(n_counters, 16)):
        if j in cols:
            out[j] = cols[j].view(np.uint64)
            continue
        z = rng.standard_normal(n, dtype=np.float32)
        z *= np.float32(0.5)
        z -= np.float32(0.125)
        np.exp(z, out=z)
        z *= dur_us
        z *= rate[cls, j - 1]
        np.floor(z, out=z)
        out[j] = z.astype(np.int64).view(np.uint64)
    return out


def make_config(cid: int, iters: Optional[int] = None,
                with_truth: bool = True, seed: Optional[int] = None) -> Trace:
    """Build the synthetic trace of configuration `cid` (0..4).

    `iters` overrides the iteration count (same per-iteration shape) to make
    bounded samples of a configuration; `seed` overrides its seed.
    """
    cfg = dict(CONFIGS[cid])
    if iters is not None:
        cfg["iters"] = int(iters)
    sd = cfg["seed"] if seed is None else seed
    rng = np.random.default_rng(np.random.PCG64(sd))
    G = cfg["n_gpus"]
    recs = dict(gpu=[], stream=[], start=[], end=[], cls=[], op_id=[],
                ref_start=[], ref_end=[])
    mks = dict(gpu=[], level=[], start=[], end=[], label=[])
    anc = dict(gpu=[], local=[], ref=[])
    depth = cfg["depth_hi"]
    t0 = BASE_REF_NS
    for g in range(G):
        base = t0 + int(rng.integers(0, 1_000_000))
        comp, comm, markers, (it_s, it_e) = _gpu_timeline(rng, cfg, base)
        if cfg["offset_ns"]:
            off = int(rng.integers(-cfg["offset_ns"], cfg["offset_ns"] + 1))
            drift = float(rng.uniform(-cfg["drift_ppm"], cfg["drift_ppm"]))
        else:
            off, drift = 0, 0.0
        # ---- records of this GPU in profiler order (local start, stream)
        r_start = np.concatenate([comp["start"], comm["start"]])
        r_end = np.concatenate([comp["end"], comm["end"]])
        r_stream = np.concatenate([comp["stream"], comm["stream"]])
        r_cls = np.concatenate([comp["cls"], comm["cls"]])
        r_lab = np.concatenate([comp["label"], comm["label"]])
        l_start = _to_local(r_start, off, drift, t0)
        l_end = _to_local(r_end, off, drift, t0)
        o = np.lexsort((r_stream, l_start))
        recs["gpu"].append(np.full(o.shape, g, np.uint8))
        recs["stream"].append(r_stream[o])
        recs["start"].append(l_start[o])
        recs["end"].append(l_end[o])
        recs["cls"].append(r_cls[o])
        recs["op_id"].append(r_lab[o])
        recs["ref_start"].append(r_start[o])
        recs["ref_end"].append(r_end[o])
        # ---- markers
        lv, ms, me, ml, mit = (markers["level"], markers["start"],
                               markers["end"], markers["label"], markers["it"])
        if cfg["depth_hi"] > 4 or cfg["depth_lo"] < 4:
            d_it = rng.integers(cfg["depth_lo"], cfg["depth_hi"] + 1,
                                size=cfg["iters"])
            keep = (lv < 3) | (d_it[mit] >= 4)
            extra = []
            ops = np.nonzero((lv == 3) & (d_it[mit] >= 5))[0]
            if ops.size:
                s4, e4, l4, i4 = _sub_splits(rng, 4, ms[ops], me[ops], 3,
                                             mit[ops])
                extra.append((4, s4, e4, l4, i4))
                sel5 = d_it[i4] >= 6
                if sel5.any():
                    s5, e5, l5, i5 = _sub_splits(rng, 5, s4[sel5], e4[sel5],
                                                 2, i4[sel5])
                    extra.append((5, s5, e5, l5, i5))
            lv, ms, me, ml = lv[keep], ms[keep], me[keep], ml[keep]
            for (lev, s_, e_, l_, _i) in extra:
                lv = np.concatenate([lv, np.full(s_.shape, lev, np.uint8)])
                ms = np.concatenate([ms, s_])
                me = np.concatenate([me, e_])
                ml = np.concatenate([ml, l_])
        if cfg["drop_frac"] > 0:
            keep = rng.random(lv.shape[0]) >= cfg["drop_frac"]
            lv, ms, me, ml = lv[keep], ms[keep], me[keep], ml[keep]
        # profiler order: ranges in the order they open (start, outer first)
        mo = np.lexsort((lv, ms))
        lv, ms, me, ml = lv[mo], ms[mo], me[mo], ml[mo]
        mks["gpu"].append(np.full(lv.shape, g, np.uint8))
        mks["level"].append(lv)
        mks["start"].append(_to_local(ms, off, drift, t0))
        mks["end"].append(_to_local(me, off, drift, t0))
        mks["label"].append(ml)
        # ---- anchors: same instant read on the local and reference clocks
        A = cfg["anchors_per_iter"]
        if A:
            span = np.maximum(it_e - it_s, 1)
            q = np.arange(A)[None, :]
            y = (it_s[:, None] + (q * span[:, None]) // A +
                 rng.integers(0, np.maximum(span // A, 1)[:, None],
                              size=(span.shape[0], A)))
            y = y.reshape(-1)
            x = _to_local(y, off, drift, t0) + rng.integers(-50, 51,
                                                            size=y.shape)
            anc["gpu"].append(np.full(y.shape, g, np.uint8))
            anc["local"].append(x.astype(np.int64))
            anc["ref"].append(y.astype(np.int64))

    cat = lambda lst, dt: (np.concatenate(lst).astype(dt, copy=False)
                           if lst else np.zeros(0, dt))
    gpu = cat(recs["gpu"], np.uint8)
    stream = cat(recs["stream"], np.uint8)
    start = cat(recs["start"], np.int64)
    end = cat(recs["end"], np.int64)
    cls = cat(recs["cls"], np.uint8)
    op_id = cat(recs["op_id"], np.uint32)
    ref_start = cat(recs["ref_start"], np.int64)
    ref_end = cat(recs["ref_end"], np.int64)
    m_gpu = cat(mks["gpu"], np.uint8)
    m_level = cat(mks["level"], np.uint8)
    m_start = cat(mks["start"], np.int64)
    m_end = cat(mks["end"], np.int64)
    m_label = cat(mks["label"], np.uint32)
    if cfg["shuffle"]:
        p = rng.permutation(gpu.shape[0])
        gpu, stream, start, end, cls, op_id = (gpu[p], stream[p], start[p],
                                               end[p], cls[p], op_id[p])
        ref_start, ref_end = ref_start[p], ref_end[p]
        q = rng.permutation(m_gpu.shape[0])
        m_gpu, m_level, m_start, m_end, m_label = (
            m_gpu[q], m_level[q], m_start[q], m_end[q], m_label[q])
    counters = None
    if cfg["counters"]:
        counters = _counters(rng, cls, end - start, cfg["counters"])
    truth = dict(ref_start=ref_start, ref_end=ref_end) if with_truth else {}
    return Trace(n_gpus=G, depth=depth, gpu=gpu, stream=stream, start=start,
                 end=end, cls=cls, op_id=op_id, counters=counters,
                 m_gpu=m_gpu, m_level=m_level, m_start=m_start, m_end=m_end,
                 m_label=m_label, a_gpu=cat(anc["gpu"], np.uint8),
                 a_local=cat(anc["local"], np.int64),
                 a_ref=cat(anc["ref"], np.int64), truth=truth,
                 name=f"config{cid}" + ("" if iters is None
                                        else f"[iters={iters}]"))


# ----------------------------------------------------------------------------
# Micro traces for property tests (small spans so per-ns timelines fit)
# ----------------------------------------------------------------------------
def make_micro(seed: int, n_gpus: int = 2, n_kernels: int = 48,
               n_streams: int = 3, depth: int = 3, span: int = 4000,
               n_counters: int = 0, anchors: int = 0, nested: bool = True,
               mixed_stream_kinds: bool = True, max_dur: int = 200,
               drop_frac: float = 0.1, base: int = 0) -> Trace:
    """A small random trace.

    Kernels: random streams, classes and integer times in [base, base+span)
    including zero-length and abutting kernels (per stream sequential when
    `nested` is True, else arbitrary overlaps).  Markers: a random tiling
    hierarchy of `depth` levels per GPU with random drops (nested=True), or
    arbitrary random intervals (nested=False).  Anchors: random pairs from a
    random offset+drift line with jitter.
    """
    rng = np.random.default_rng(np.random.PCG64(10_000 + seed))
    G = n_gpus
    gpu = rng.integers(0, G, size=n_kernels).astype(np.uint8)
    stream = rng.integers(0, n_streams, size=n_kernels).astype(np.uint8)
    # class: per (gpu, stream) a preferred kind, sometimes mixed
    cls = rng.integers(0, 8, size=n_kernels).astype(np.uint8)
    if not mixed_stream_kinds:
        comm_stream = (stream % 2 == 1)
        cls = np.where(comm_stream, rng.integers(5, 7, size=n_kernels),
                       rng.choice([0, 1, 2, 3, 4, 7], size=n_kernels)
                       ).astype(np.uint8)
    start = np.empty(n_kernels, np.int64)
    end = np.empty(n_kernels, np.int64)
    if nested:
        for g in range(G):
            for s in range(n_streams):
                idx = np.nonzero((gpu == g) & (stream == s))[0]
                t = base + int(rng.integers(0, max(1, span // 8)))
                for k in idx:
                    gap = 0 if rng.random() < 0.2 else int(
                        rng.integers(0, max(2, span // (2 * max(1, idx.size)))))
                    d = 0 if rng.random() < 0.15 else int(
                        rng.integers(1, max_dur))
                    start[k] = t + gap
                    end[k] = t + gap + d
                    t = end[k]
    else:
        start[:] = base + rng.integers(0, span, size=n_kernels)
        d = rng.integers(0, max_dur, size=n_kernels)
        d[rng.random(n_kernels) < 0.15] = 0
        end[:] = start + d
    op_id = rng.integers(0, 64, size=n_kernels).astype(np.uint32)
    # markers
    mg, ml, ms, me, mlab = [], [], [], [], []
    lo = int(start.min()) - 5 if n_kernels else base
    hi = int(end.max()) + 5 if n_kernels else base + span
    for g in range(G):
        if nested:
            # recursive tiling: each level splits the parent into pieces
            parents = [(lo + int(rng.integers(0, 20)),
                        hi - int(rng.integers(0, 20)))]
            for lev in range(depth):
                nxt = []
                for (a, b) in parents:
                    k = int(rng.integers(1, 5))
                    pts = sorted(set([a, b] + [int(x) for x in
                                 rng.integers(a, max(a + 1, b), size=k - 1)]))
                    for q in range(len(pts) - 1):
                        nxt.append((pts[q], pts[q + 1]))
                # random gaps: shrink some pieces (their children then tile
                # the shrunken piece, so the hierarchy stays nested); dropped
                # pieces still shape their children
                kept = []
                for (a, b) in nxt:
                    if rng.random() < 0.1 and b - a > 2:
                        b = b - int(rng.integers(1, (b - a) // 2 + 1))
                    kept.append((a, b))
                    if rng.random() < drop_frac:
                        continue
                    mg.append(g)
                    ml.append(lev)
                    ms.append(a)
                    me.append(b)
                    mlab.append(int(rng.integers(0, 50)))
                parents = kept
        else:
            for lev in range(depth):
                k = int(rng.integers(1, 8))
                for _ in range(k):
                    a = int(rng.integers(lo, hi))
                    b = a + int(rng.integers(0, max(2, (hi - lo) // 3)))
                    mg.append(g)
                    ml.append(lev)
                    ms.append(a)
                    me.append(b)
                    mlab.append(int(rng.integers(0, 50)))
    perm = rng.permutation(len(mg))
    m_gpu = np.asarray(mg, np.uint8)[perm] if mg else np.zeros(0, np.uint8)
    m_level = np.asarray(ml, np.uint8)[perm] if ml else np.zeros(0, np.uint8)
    m_start = np.asarray(ms, np.int64)[perm] if ms else np.zeros(0, np.int64)
    m_end = np.asarray(me, np.int64)[perm] if me else np.zeros(0, np.int64)
    m_label = np.asarray(mlab, np.uint32)[perm] if mlab else np.zeros(
        0, np.uint32)
    # anchors
    a_gpu, a_local, a_ref = [], [], []
    for g in range(G):
        # tiny spans: small drift and no jitter keep the fitted slope well
        # inside the Q48 range the fit accepts (|slope| < 2^-10)
        off = int(rng.integers(-300, 301))
        drift = float(rng.uniform(-2e-4, 2e-4))
        for _ in range(anchors):
            y = base + int(rng.integers(0, span))
            x = y + off + int(round(drift * (y - base)))
            a_gpu.append(g)
            a_local.append(x)
            a_ref.append(y)
    counters = None
    if n_counters:
        counters = rng.integers(0, 1 << 40, size=(n_counters, n_kernels),
                                dtype=np.uint64)
    p = rng.permutation(n_kernels)
    return Trace(n_gpus=G, depth=depth, gpu=gpu[p], stream=stream[p],
                 start=start[p], end=end[p], cls=cls[p], op_id=op_id[p],
                 counters=None if counters is None else counters[:, p],
                 m_gpu=m_gpu, m_level=m_level, m_start=m_start, m_end=m_end,
                 m_label=m_label, a_gpu=np.asarray(a_gpu, np.uint8),
                 a_local=np.asarray(a_local, np.int64),
                 a_ref=np.asarray(a_ref, np.int64), name=f"micro{seed}")


def make_launch(tr: Trace, seed: int, max_lead: int,
                late_frac: float = 0.01) -> np.ndarray:
    """Host dispatch times of the records of `tr` on each GPU's local clock:
    start minus a uniform lead in [0, max_lead] ns, a fraction `late_frac`
    dispatched up to max_lead / 4 ns after the start (clock noise)."""
    rng = np.random.default_rng(seed)
    n = tr.n
    lead = rng.integers(0, max_lead + 1, size=n).astype(np.int64)
    late = rng.random(n) < late_frac
    lead[late] = -rng.integers(1, max(2, max_lead // 4), size=int(late.sum()))
    return tr.start - lead


def make_counter_passes(tr: Trace, rec_label: np.ndarray, seed: int,
                        cols=(3, 3, 2, 2, 2, 2, 2), drop_frac: float = 0.0,
                        mismatch_frac: float = 0.0,
                        extra: int = 0) -> List[dict]:
    """Serialized hardware-counter passes of the records of `tr` (paper
    III-A: two or three counters per pass, no valid timestamps): pass p
    lists every record once, grouped by GPU in dispatch (local start) order,
    with its iteration label rec_label[k] and the values of the counter
    columns it covers.  Perturbations: a fraction of entries dropped, a
    fraction given another class, `extra` entries per GPU appended with an
    iteration label past the last one."""
    rng = np.random.default_rng(seed)
    assert tr.counters is not None and sum(cols) <= tr.counters.shape[0]
    order = np.lexsort((np.arange(tr.n), tr.start, tr.gpu.astype(np.int64)))
    passes, c0 = [], 0
    for p, nc in enumerate(cols):
        k = order.copy()
        if drop_frac > 0:
            k = k[rng.random(k.shape[0]) >= drop_frac]
        cls = tr.cls[k].copy()
        if mismatch_frac > 0:
            flip = rng.random(k.shape[0]) < mismatch_frac
            cls[flip] = (cls[flip] + 1) % 8
        gpu, stream = tr.gpu[k].copy(), tr.stream[k].copy()
        lab = np.asarray(rec_label, np.uint32)[k].copy()
        vals = tr.counters[c0:c0 + nc][:, k].copy()
        if extra:
            pos = np.searchsorted(gpu, np.arange(tr.n_gpus), side="right")
            ins_g = np.repeat(np.arange(tr.n_gpus), extra)
            at = np.repeat(pos, extra)
            gpu = np.insert(gpu, at, ins_g.astype(np.uint8))
            stream = np.insert(stream, at, np.zeros(at.shape, np.uint8))
            cls = np.insert(cls, at, np.zeros(at.shape, np.uint8))
            top = np.uint32(lab[lab != 0xFFFFFFFF].max() + 1 if
                            (lab != 0xFFFFFFFF).any() else 0)
            lab = np.insert(lab, at, np.full(at.shape, top, np.uint32))
            vals = np.insert(vals, at, np.zeros((nc, at.shape[0]), np.uint64),
                             axis=1)
        passes.append(dict(gpu=gpu, stream=stream, cls=cls, lab=lab,
                           values=np.ascontiguousarray(vals, np.uint64),
                           dst=list(range(c0, c0 + nc))))
        c0 += nc
    return passes
