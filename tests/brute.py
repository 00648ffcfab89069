"""Brute-force reference computations used to pin the CPU oracle.

Each function takes the slowest obviously-correct route: per-nanosecond
timelines, linear scans over all markers, exact rational least squares with
Python integers, dictionary grouping.  Sizes must stay small.
"""
from __future__ import annotations

from fractions import Fraction
from typing import Dict, List, Tuple

import numpy as np

NONE = 0xFFFFFFFF


def rne(x: Fraction) -> int:
    """Round half to even of an exact rational."""
    f = x.numerator // x.denominator
    r = x - f
    if r > Fraction(1, 2) or (r == Fraction(1, 2) and f % 2 == 1):
        f += 1
    return f


def fit_fraction(xs: List[int], ys: List[int]) -> Tuple[int, int, int]:
    """Exact least squares of (y - x) against (x - x0), slope in Q48.

    Centred form: slope = sum((u-ubar)(w-wbar)) / sum((u-ubar)^2), then
    D = rne(slope * 2^48), C = rne(wbar - D * ubar / 2^48).
    """
    if not xs:
        return 0, 0, 0
    pairs = sorted(zip(xs, ys))
    x0 = pairs[0][0]
    u = [Fraction(x - x0) for x, _ in pairs]
    w = [Fraction(y - x) for x, y in pairs]
    n = len(u)
    ub = sum(u) / n
    wb = sum(w) / n
    sxx = sum((a - ub) ** 2 for a in u)
    if n == 1 or sxx == 0:
        D = 0
    else:
        sxy = sum((a - ub) * (b - wb) for a, b in zip(u, w))
        D = rne(sxy / sxx * (1 << 48))
    C = rne(wb - Fraction(D, 1 << 48) * ub)
    return x0, C, D


def attribute_scan(gpu, s, m_gpu, m_level, ms, me, depth) -> np.ndarray:
    """Linear scan: the last non-empty marker in (start', index) order with
    start' <= s', if it still contains s'."""
    n = len(gpu)
    out = np.full((depth, n), NONE, np.uint32)
    for k in range(n):
        for lev in range(depth):
            best = None
            for j in range(len(m_gpu)):
                if m_gpu[j] != gpu[k] or m_level[j] != lev:
                    continue
                if me[j] <= ms[j] or ms[j] > s[k]:
                    continue
                key = (int(ms[j]), j)
                if best is None or key > best[0]:
                    best = (key, j)
            if best is not None and s[k] < me[best[1]]:
                out[lev, k] = best[1]
    return out


def timelines(gpu, cls, s, e, n_gpus):
    """Per-GPU per-ns arrays of active compute and comm kernel counts over
    [lo, hi).  Returns lo, c[G][span], m[G][span]."""
    lo = int(min(s.min(), e.min())) - 2 if len(s) else 0
    hi = int(max(s.max(), e.max())) + 2 if len(s) else 1
    span = hi - lo
    c = np.zeros((n_gpus, span), np.int32)
    m = np.zeros((n_gpus, span), np.int32)
    for k in range(len(s)):
        if e[k] <= s[k]:
            continue
        arr = m if cls[k] in (5, 6) else c
        arr[gpu[k], s[k] - lo:e[k] - lo] += 1
    return lo, c, m


def window_counts(lo, c, m, g, a, b):
    """(CO, MO, OV, ID) ns in [a, b) on GPU g from the per-ns arrays; time
    outside [lo, lo+span) is idle."""
    if b <= a:
        return (0, 0, 0, 0)
    span = c.shape[1]
    aa, bb = max(a - lo, 0), min(b - lo, span)
    if bb <= aa:
        return (0, 0, 0, b - a)
    cc = c[g, aa:bb] > 0
    mm = m[g, aa:bb] > 0
    co = int(np.sum(cc & ~mm))
    mo = int(np.sum(~cc & mm))
    ov = int(np.sum(cc & mm))
    return (co, mo, ov, (b - a) - co - mo - ov)


def overlap_brute(gpu, stream, cls, s, e, m_gpu, ms, me, n_gpus):
    n = len(gpu)
    lo, c, m = timelines(gpu, cls, s, e, n_gpus)
    ovl = np.zeros(n, np.int64)
    for k in range(n):
        if e[k] > s[k]:
            ovl[k] = window_counts(lo, c, m, gpu[k], s[k], e[k])[2]
    mwin = np.zeros((len(m_gpu), 4), np.int64)
    for j in range(len(m_gpu)):
        mwin[j] = window_counts(lo, c, m, m_gpu[j], ms[j], me[j])
    gwin = np.zeros((n_gpus, 6), np.int64)
    for g in range(n_gpus):
        sel = np.nonzero(gpu == g)[0]
        if sel.size == 0:
            continue
        a, b = int(s[sel].min()), int(e[sel].max())
        gwin[g, :2] = (a, b)
        gwin[g, 2:] = window_counts(lo, c, m, g, a, b)
    # bubbles: previous compute kernel of the same (gpu, stream)
    gap = np.zeros(n, np.int64)
    for k in range(n):
        if cls[k] in (5, 6):
            continue
        best = None
        for j in range(n):
            if j == k or gpu[j] != gpu[k] or stream[j] != stream[k]:
                continue
            if cls[j] in (5, 6):
                continue
            if (s[j], j) < (s[k], k):
                if best is None or (s[j], j) > (s[best], best):
                    best = j
        if best is not None:
            gap[k] = max(0, int(s[k]) - int(e[best]))
    return dict(ovl=ovl, gap=gap, mwin=mwin, gwin=gwin)


def aggregate_brute(gpu, cls, s, e, idx, gap, ovl, counters, depth,
                    levels, sel=None) -> Dict[int, list]:
    """Rows per level as lists of dicts, grouped with Python dictionaries and
    ordered by (gpu, kind, tmin, first)."""
    n = len(gpu)
    keep = range(n) if sel is None else [k for k in range(n) if sel[k]]
    nc = 0 if counters is None else counters.shape[0]
    out = {}
    for lev in levels:
        groups: Dict[tuple, dict] = {}
        for k in keep:
            kind = 1 if cls[k] in (5, 6) else 0
            if lev == 100:
                key = (int(gpu[k]), (), kind)
            elif lev == 101:
                key = (0xFF, (), kind)
            else:
                key = (int(gpu[k]), tuple(int(idx[j][k]) for j in
                                          range(lev + 1)), kind)
            r = groups.setdefault(key, dict(n=0, dur=0, gap=0, ovl=0,
                                            tmin=None, tmax=None, first=None,
                                            ctr=[0] * nc))
            r["n"] += 1
            r["dur"] += int(e[k]) - int(s[k])
            r["gap"] += int(gap[k])
            r["ovl"] += int(ovl[k])
            if r["tmin"] is None or (int(s[k]), k) < (r["tmin"], r["first"]):
                r["tmin"], r["first"] = int(s[k]), k
            if r["tmax"] is None or int(e[k]) > r["tmax"]:
                r["tmax"] = int(e[k])
            for q in range(nc):
                r["ctr"][q] = (r["ctr"][q] + int(counters[q][k])) % (1 << 64)
        rows = []
        for (g, path, kind), r in groups.items():
            r = dict(r)
            r["gpu"], r["kind"] = g, kind
            r["path"] = list(path) + [NONE] * (depth - len(path))
            rows.append(r)
        rows.sort(key=lambda r: (r["gpu"], r["kind"], r["tmin"], r["first"]))
        out[lev] = rows
    return out


def aggregate_numpy(gpu, cls, s, e, idx, gap, ovl, counters, depth, levels,
                    sel=None):
    """Vectorized grouping for large traces: one sort of the records by
    (gpu, kind, path...), group boundaries per level from key changes,
    np.*.reduceat for sums, minima and maxima, first = smallest index at the
    group's minimum start, rows ordered by (gpu, kind, tmin, first).
    Returns {level: dict of row columns}."""
    n = len(gpu)
    keep = np.arange(n) if sel is None else np.nonzero(sel)[0]
    g = gpu[keep].astype(np.int64)
    kind = np.isin(cls[keep], (5, 6)).astype(np.int64)
    st = s[keep]
    paths = [idx[l][keep].astype(np.int64) for l in range(depth)]
    keys = paths[::-1] + [kind, g]
    o = np.lexsort(keys)
    rec = keep[o]
    g, kind, st = g[o], kind[o], st[o]
    paths = [p[o] for p in paths]
    en = e[rec]
    cols = dict(n=np.ones(len(rec), np.uint64),
                dur=(en - st).astype(np.int64), gap=gap[rec].astype(np.int64),
                ovl=ovl[rec].astype(np.int64))
    ctr = None if counters is None else counters[:, rec]
    out = {}
    base = dict(rec=rec, g=g, kind=kind, st=st, en=en, paths=paths, cols=cols,
                ctr=ctr)
    for lev in levels:
        if len(rec) == 0:
            out[lev] = None
            continue
        if lev == 101:
            # workload groups span GPUs: regroup by kind alone
            ko = np.argsort(base["kind"], kind="stable")
            rec, g, kind = base["rec"][ko], base["g"][ko], base["kind"][ko]
            st, en = base["st"][ko], base["en"][ko]
            cols = {k: v[ko] for k, v in base["cols"].items()}
            ctr = None if base["ctr"] is None else base["ctr"][:, ko]
            diff = kind[1:] != kind[:-1]
        else:
            diff = (g[1:] != g[:-1]) | (kind[1:] != kind[:-1])
            if lev < 100:
                for l in range(lev + 1):
                    diff |= paths[l][1:] != paths[l][:-1]
        b = np.concatenate([[0], np.nonzero(diff)[0] + 1])
        rows = {}
        for k, v in cols.items():
            rows[k] = np.add.reduceat(v, b)
        tmin = np.minimum.reduceat(st, b)
        gid = np.repeat(np.arange(len(b)), np.diff(np.append(b, len(rec))))
        at_min = np.where(st == tmin[gid], rec, np.int64(1) << 40)
        first = np.minimum.reduceat(at_min, b).astype(np.uint32)
        tmax = np.maximum.reduceat(en, b)
        rg = (np.full(len(b), 0xFF, np.int64) if lev == 101 else g[b])
        rk = kind[b]
        order = np.lexsort((first, tmin, rk, rg))
        r = dict(gpu=rg[order].astype(np.uint8), kind=rk[order].astype(np.uint8),
                 tmin=tmin[order], tmax=tmax[order], first=first[order])
        for k in cols:
            r[k] = rows[k][order]
        path = np.full((depth, len(b)), NONE, np.uint32)
        if lev < 100:
            for l in range(lev + 1):
                path[l] = paths[l][b].astype(np.uint32)
        r["path"] = path[:, order]
        if ctr is not None:
            r["ctr"] = np.add.reduceat(ctr, b, axis=1)[:, order]
        else:
            r["ctr"] = np.zeros((0, len(b)), np.uint64)
        out[lev] = r
    return out
