"""Throughput of the trace pipeline on one MI355X.

One step = chopper_align + chopper_attribute + chopper_overlap +
chopper_aggregate(all levels) + derived ratios over the whole synthetic trace
of 8 GPUs x 800 iterations x 32 layers with 16 counters per record (the
Llama-3-8B FSDP trace shape), inputs resident in HBM.  After the timed steps
chopper_views (per-phase/class and per-operation views with their medians),
chopper_op_stats (overlap statistics and overhead breakdown per operation),
chopper_launch_split (preparation / call overhead from seeded dispatch
times) and chopper_join_counters (the counters split into seven serialized
passes and attached back) are timed on their own over the same run
("views", "op_stats", "launch_split", "join_counters").
Prints one JSON line.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--config 3]
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("kernel records/sec end-to-end (align+attribute+overlap+aggregate);"
          " % HBM peak")
HBM_PEAK_GBS = 8000.0
# the kernel whose roofline is reported: the records reduction, which reads
# every record's counters -- the fast path's (groups are runs of the
# (gpu, kind, start') order) or, where that does not hold (e.g. shuffled
# input with markers numbered out of order), the general path's
ROOF_KERNELS = ("agg_fast_reduce_records", "agg_reduce_records")


def algorithmic_bytes(n, nm, rows, depth, nc, n_rows_finest):
    """Bytes that must cross HBM once: every input read once, every output
    written once (records, markers, aggregated rows, derived ratios)."""
    rec_in = n * (1 + 1 + 8 + 8 + 1 + 8 * nc)          # gpu stream start end cls ctr
    rec_out = n * (8 + 8 + 4 + 4 + 4 * depth + 8 + 8)  # start' end' order korder idx gap ovl
    mk = nm * (1 + 1 + 8 + 8) + nm * (8 + 8 + 32 + 32)  # in; start' end' CO..ID fractions
    row = 4 * depth + 1 + 1 + 8 + 5 * 8 + 4 + 8 * nc + 6 * 8
    return rec_in + rec_out + mk + rows * row


def roof_kernel_bytes(kernel, n, depth, nc, rows_written, input_order):
    """Algorithmic bytes of one launch of the records reduction: per record
    gpu, cls, path, start, end, gap, ovl and counters read once (and korder
    when the input is not grouped by GPU in start order, so that the
    reduction reads through it; the general path reads the gathered path
    and gpu/kind items, 4 per level + 2 bytes, in place of gpu, cls and
    path); per row it produces (the two finest levels on the fast path, the
    finest on the general one) its header (path, gpu, kind, first record)
    and its sums and counters written once."""
    if kernel == "agg_reduce_records":
        per_rec = 4 + 2 + 4 * depth + 8 * 4 + 8 * nc
    else:
        per_rec = (0 if input_order else 4) + 1 + 1 + 4 * depth + 8 * 4 + 8 * nc
    per_row = 4 * depth + 1 + 1 + 4 + 8 * (6 + nc)
    return n * per_rec + rows_written * per_row


def views_bytes(n, nm, rows_op, units, P, O):
    """Algorithmic bytes of chopper_views: per record cls, start', end', gap
    and its iteration and phase markers read once; per marker its level read
    and its unit number written; per row of the operation level its three
    path entries, kind and n / dur / gap / ovl read; the tables, busy times
    and unit markers written once."""
    return (n * (1 + 8 + 8 + 8 + 4 + 4) + nm * (1 + 4) + rows_op * (12 + 1 + 32)
            + units * (8 * (3 * P * 8 + 4 * P * O * 2 + 1) + 4))


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed counter record
    (FETCH_SIZE and WRITE_SIZE scaled by a plain copy of known size), or
    None when there is none or the kernel's sources changed since."""
    import glob
    import hashlib
    for path in glob.glob(os.path.join(ROOT, "profiles", "*_traffic.json")):
        try:
            rec = json.load(open(path))
        except (OSError, ValueError):
            continue
        if rec.get("kernel") != kernel:
            continue
        h = hashlib.sha256()
        try:
            for f in rec["source_files"]:
                h.update(open(os.path.join(ROOT, f), "rb").read())
        except OSError:
            return None
        if h.hexdigest() != rec.get("source_sha256"):
            return None
        return float(rec["traffic_bytes_per_dispatch"])
    return None


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cid, iters, tr=None):
    """The CPU oracle, as it stands (single-threaded C), over the whole
    pipeline: on the benchmark's own trace when `tr` is given, else on a
    trace of the same shape with `iters` iterations."""
    import oracle
    import tracegen as tg
    whole = tr is not None
    if tr is None:
        tr = tg.make_config(cid, iters=iters, with_truth=False)
    t0 = time.perf_counter()
    oracle.run(tr)
    dt = time.perf_counter() - t0
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count()
    what = (f"the whole benchmark trace ({tr.n} records, {tr.n_markers} "
            "markers)" if whole else
            f"a trace of the benchmark's shape ({tg.CONFIG_NAMES[cid]}) "
            f"with {iters} iterations ({tr.n} records, {tr.n_markers} "
            "markers)")
    return {"value": tr.n / dt, "unit": "records/s", "cores": 1,
            "host_cores_available": cores, "cpu_model": cpu_model(),
            "kind": "oracle", "seconds": dt,
            "sample": what + ", single-threaded C oracle: align, sort, "
                      "attribute, overlap, aggregate, ratios"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-iters", type=int, default=0,
                    help="time the oracle on a trace of this many iterations "
                         "instead of the benchmark's own (0: the whole "
                         "benchmark trace up to 25M records, else 500)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run plain device copies of this many MiB (the "
                         "reference kernel for scaling HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py runs on one GPU only: the traces of all ranks are "
              "input data to a single device (the path would shard by source "
              "GPU, each device taking the traces of its ranks).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    if args.copy_calibration > 0:
        nb = args.copy_calibration << 20
        a = torch.ones(nb, dtype=torch.uint8, device="cuda:0")
        b = torch.empty_like(a)
        for _ in range(3):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": nb, "copies": 3}), flush=True)
        return
    import tracegen as tg
    import paper_2512_08242_amd as ch

    def log(*a):
        print(*a, file=sys.stderr, flush=True)

    cid = args.config
    t0 = time.perf_counter()
    tr = tg.make_config(cid, with_truth=False)
    log(f"[bench] generated config {cid}: {tr.n} records, {tr.n_markers} "
        f"markers in {time.perf_counter() - t0:.1f}s")
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    dt = ch.DeviceTrace(tr, dev)
    n, nm, depth, nc = tr.n, tr.n_markers, tr.depth, tr.n_counters
    # records grouped by GPU and in start order inside each GPU: the
    # reduction then reads them in input order
    g = tr.gpu.astype(np.int64)
    input_order = bool(np.all(np.diff(g) >= 0) and np.all(
        (np.diff(g) != 0) | (np.diff(tr.start) >= 0)))
    # seeded dispatch times (local clocks) for the launch-overhead split
    launch_host = tg.make_launch(tr, 11, max_lead=20000)
    trace_host = tr
    del g
    torch.cuda.synchronize()
    pipe = ch.Pipeline(dt)
    for _ in range(max(args.warmup, 1)):
        pipe.step()
    torch.cuda.synchronize()
    lo = pipe.rows.level_offset.cpu().numpy()
    rows_total = int(lo[-1])
    rows_finest = int(lo[depth] - lo[depth - 1])
    log(f"[bench] warmup done; rows: {rows_total} (finest level "
        f"{rows_finest})")
    # which records reduction this trace takes: one probe step per candidate
    # (events recorded first, the stop before the start, so that a kernel
    # that does not run reads at most 0 even beside one that takes a few us)
    probe = {}
    for name in ROOF_KERNELS:
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        b.record()
        a.record()
        ch.time_kernel(name, a, b)
        pipe.step()
        torch.cuda.synchronize()
        ch.time_kernel(None)
        probe[name] = a.elapsed_time(b)
    ROOF_KERNEL = max(ROOF_KERNELS, key=lambda k: probe[k])
    # the fast path writes the two finest levels, the general one the finest
    rows_records = (int(lo[depth] - lo[max(depth - 2, 0)])
                    if ROOF_KERNEL == "agg_fast_reduce_records"
                    else rows_finest)

    K = args.steps
    kev = [(torch.cuda.Event(enable_timing=True),
            torch.cuda.Event(enable_timing=True)) for _ in range(K)]
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for k in range(K):
        ch.time_kernel(ROOF_KERNEL, kev[k][0], kev[k][1])
        pipe.step()
    e1.record()
    torch.cuda.synchronize()
    ch.time_kernel(None)
    ms = e0.elapsed_time(e1) / K
    kms = float(np.mean([a.elapsed_time(b) for a, b in kev]))
    status = int(pipe.status.item()) & 0xFFFFFFFF
    log(f"[bench] {ms:.3f} ms/step, {ROOF_KERNEL} {kms:.3f} ms, "
        f"status {status}")

    value = n / (ms * 1e-3)
    bmin = algorithmic_bytes(n, nm, rows_total, depth, nc, rows_finest)
    kb = roof_kernel_bytes(ROOF_KERNEL, n, depth, nc, rows_records,
                           input_order)
    achieved = kb / (kms * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "records/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {
            "workload": tg.CONFIG_NAMES[cid],
            "records": n, "markers": nm, "depth": depth, "counters": nc,
            "rows": rows_total,
        },
        "hbm_frac_end_to_end": bmin / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "algorithmic_bytes_per_step": bmin,
        "roofline": {
            "kernel": ROOF_KERNEL,
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": measured_traffic(ROOF_KERNEL),
            "kernel_ms": kms,
            "bytes_per_launch": kb,
            "input_order": input_order,
        },
        "status": status,
    }
    # the re-keyed views of the same run, timed on their own after the steps
    iters = tg.CONFIGS[cid]["iters"]
    P, O = 3, 64
    views = ch.Views(pipe, n_phases=P, n_ops=O, n_iters=iters,
                     warmup=10 if iters > 10 else 0)
    views.run()
    torch.cuda.synchronize()
    v0 = torch.cuda.Event(enable_timing=True)
    v1 = torch.cuda.Event(enable_timing=True)
    v0.record()
    for _ in range(K):
        views.run()
    v1.record()
    torch.cuda.synchronize()
    vms = v0.elapsed_time(v1) / K
    vb = views_bytes(n, nm, int(lo[min(3, depth - 1) + 1] -
                                lo[min(3, depth - 1)]), views.U, P, O)
    out["views"] = {
        "ms": vms, "units": views.U, "bytes": vb,
        "achieved": vb / (vms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
        "unit": "GB/s", "frac": vb / (vms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "spec": {"n_phases": P, "n_ops": O, "n_iters": iters,
                 "warmup": 10 if iters > 10 else 0}}
    log(f"[bench] views {vms:.3f} ms")
    # overlap statistics and overhead breakdown per (phase, operation)
    fg = np.linspace(2e9, 9e10, O)
    pipe.op_stats(n_phases=P, n_ops=O, tpt_peak=1.3e6, f_gemm=fg)
    torch.cuda.synchronize()
    v0.record()
    for _ in range(K):
        pipe.op_stats(n_phases=P, n_ops=O, tpt_peak=1.3e6, f_gemm=fg)
    v1.record()
    torch.cuda.synchronize()
    sms = v0.elapsed_time(v1) / K
    # per operation-level row: kind, duration, gap, overlap, the phase and
    # operation path entries, three counters
    lop = min(3, depth - 1)
    rows_op = int(lo[lop + 1] - lo[lop])
    sb = rows_op * (1 + 8 + 8 + 8 + 4 + 4 + (24 if nc >= 16 else 0))
    out["op_stats"] = {
        "ms": sms, "rows": rows_op, "bytes": sb,
        "achieved": sb / (sms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
        "unit": "GB/s", "frac": sb / (sms * 1e-3) / 1e9 / HBM_PEAK_GBS}
    log(f"[bench] op stats {sms:.3f} ms")
    # the launch-overhead split from seeded dispatch times, timed on its own
    tl = torch.from_numpy(launch_host).to(dev)
    pipe.launch_split(tl)
    torch.cuda.synchronize()
    v0.record()
    for _ in range(K):
        pipe.launch_split(tl)
    v1.record()
    torch.cuda.synchronize()
    lms = v0.elapsed_time(v1) / K
    lb = n * (1 + 8 + 8 + 8 + 8 + 8)
    out["launch_split"] = {
        "ms": lms, "bytes": lb, "achieved": lb / (lms * 1e-3) / 1e9,
        "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": lb / (lms * 1e-3) / 1e9 / HBM_PEAK_GBS}
    log(f"[bench] launch split {lms:.3f} ms")
    # the counter-pass join: the 16 counters split into seven serialized
    # passes (3, 3, 2, 2, 2, 2, 2 columns) and attached back to the records
    if trace_host.counters is not None:
        res = pipe.results()
        i0 = res["idx"][0]
        lab = np.full(n, 0xFFFFFFFF, np.uint32)
        lab[i0 != 0xFFFFFFFF] = trace_host.m_label[i0[i0 != 0xFFFFFFFF]]
        passes = tg.make_counter_passes(trace_host, lab, 5)
        tt = lambda a, dt_: torch.from_numpy(
            np.ascontiguousarray(a).view(dt_)).to(dev)
        dp = [dict(gpu=tt(q["gpu"], np.uint8), stream=tt(q["stream"], np.uint8),
                   cls=tt(q["cls"], np.uint8), label=tt(q["lab"], np.int32),
                   values=tt(q["values"], np.int64), dst=q["dst"])
              for q in passes]
        del passes, res
        pipe.join_counters(dp)
        torch.cuda.synchronize()
        v0.record()
        for _ in range(K):
            pipe.join_counters(dp)
        v1.record()
        torch.cuda.synchronize()
        jms = v0.elapsed_time(v1) / K
        # per pass entry gpu, stream, class, label and its columns read;
        # per record (once for all passes) order, gpu, stream, class and
        # its iteration marker read, the 16 counters and the matched bits
        # written
        cols = 16
        m_tot = sum(int(q["gpu"].shape[0]) for q in dp)
        jb = (m_tot * (1 + 1 + 1 + 4) + n * 8 * cols
              + n * (4 + 1 + 1 + 1 + 4) + n * 8 * cols + n)
        out["join_counters"] = {
            "ms": jms, "passes": len(dp), "bytes": jb,
            "achieved": jb / (jms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": jb / (jms * 1e-3) / 1e9 / HBM_PEAK_GBS}
        log(f"[bench] join counters {jms:.3f} ms")
        del dp
    if not args.no_cpu_baseline:
        whole = args.cpu_iters == 0 and n <= 25_000_000
        log("[bench] timing the CPU oracle")
        out["cpu_baseline"] = cpu_baseline(
            cid, args.cpu_iters or 500, trace_host if whole else None)
    del trace_host
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
