"""Brute-force recomputation with the Python standard library, for tiny inputs.

These are the pins of the oracle: independent, deliberately naive
restatements built on library routines (int.bit_length, min/max/sum/len over
dict-of-lists groups, statistics.median_low, numpy.quantile(method="lower"),
fractions.Fraction). They share nothing with the oracle's C code.
"""
from __future__ import annotations

import statistics
from collections import defaultdict
from fractions import Fraction

import numpy as np

NB = 32
I64_MAX = 2**63 - 1
I64_MIN = -(2**63)


def bin_of(d: int) -> int:
    return min(max(d.bit_length() - 1, 0), NB - 1)


def wrap64(v: int) -> int:
    v &= (1 << 64) - 1
    return v - (1 << 64) if v >= (1 << 63) else v


def summarize(ev, K, NS):
    kid, st = ev["kernel_id"].tolist(), ev["stream"].tolist()
    t0, t1 = ev["start_ns"].tolist(), ev["end_ns"].tolist()
    off = ev["seg_off"].tolist()
    G = len(off) - 1
    res = []
    for g in range(G):
        groups = defaultdict(list)
        per_stream = defaultdict(int)
        valid_starts, valid_ends, invalid = [], [], 0
        for i in range(off[g], off[g + 1]):
            ok = 0 <= kid[i] < K and 0 <= st[i] < NS and t0[i] >= 0 and t1[i] >= t0[i]
            if not ok:
                invalid += 1
                continue
            d = t1[i] - t0[i]
            groups[kid[i]].append(d)
            per_stream[st[i]] += d
            valid_starts.append(t0[i])
            valid_ends.append(t1[i])
        cells = {}
        for k, ds in groups.items():
            h = [0] * NB
            for d in ds:
                h[bin_of(d)] += 1
            cells[k] = dict(count=len(ds), sum=wrap64(sum(ds)), min=min(ds), max=max(ds), hist=h)
        n_valid = sum(len(v) for v in groups.values())
        busy = wrap64(sum(sum(v) for v in groups.values()))
        wire = sum(33 + 5 * sum(1 for b in c["hist"] if b) for c in cells.values())
        res.append(dict(cells=cells, n_valid=n_valid, n_invalid=invalid,
                        t_first=min(valid_starts) if valid_starts else I64_MAX,
                        t_last=max(valid_ends) if valid_ends else I64_MIN,
                        step=(max(valid_ends) - min(valid_starts)) if valid_starts else 0,
                        busy=busy, stream_busy=[wrap64(per_stream[s]) for s in range(NS)], wire=wire))
    return res


def order_stats(xs):
    """Lower median, lower nearest-rank quartiles and lower-median MAD."""
    med = statistics.median_low(xs)
    q1 = int(np.quantile(np.array(xs, dtype=object).astype(np.int64), 0.25, method="lower"))
    q3 = int(np.quantile(np.array(xs, dtype=object).astype(np.int64), 0.75, method="lower"))
    mad = statistics.median_low([abs(x - med) for x in xs])
    return med, q1, q3, mad


def rel_std_ok(ys, cmax_pm):
    """Sample relative std (ddof 1) <= cmax_pm/1000, exactly with Fractions."""
    n = len(ys)
    if n < 2:
        return True
    mean = Fraction(sum(ys), n)
    var = sum((Fraction(y) - mean) ** 2 for y in ys) / (n - 1)
    return var <= Fraction(cmax_pm, 1000) ** 2 * mean ** 2


def iter_windows(y, W=5, theta_pm=1500, beta_pm=1200, rho_pm=1300, cmax_pm=100, min_seg=2):
    S = len(y)
    flags = [0] * S
    if any(v < 0 or v >= 2**40 for v in y):
        return dict(flags=flags, cls=0x80, eff_width=0, cp=-1)
    w = min(W, S)
    windows = [(t, t + w - 1) for t in range(S - w + 1)
               if Fraction(max(y[t:t + w])) > Fraction(theta_pm, 1000) * min(y[t:t + w])]
    intervals = []
    for a, b in windows:
        if intervals and a <= intervals[-1][1] + 1:
            intervals[-1][1] = max(intervals[-1][1], b)
        else:
            intervals.append([a, b])
    eff = 0
    for a, b in intervals:
        outside = [y[i] for i in range(S) if i < a or i > b]
        base = statistics.median_low(outside if outside else y)
        run = 0
        for i in range(a, b + 1):
            flags[i] |= 1
            if Fraction(y[i]) > Fraction(beta_pm, 1000) * base:
                flags[i] |= 2
                run += 1
                eff = max(eff, run)
            else:
                run = 0
    best, best_ratio = -1, None
    for t in range(min_seg, S - min_seg + 1):
        L, Rr = y[:t], y[t:]
        if sum(L) == 0:
            continue
        ratio = Fraction(sum(Rr), len(Rr)) / Fraction(sum(L), len(L))
        if ratio < Fraction(rho_pm, 1000):
            continue
        if not (rel_std_ok(L, cmax_pm) and rel_std_ok(Rr, cmax_pm)):
            continue
        if best_ratio is None or ratio > best_ratio:
            best, best_ratio = t, ratio
    if best >= 0:
        for i in range(best, S):
            flags[i] |= 4
    cls = (1 if eff > 0 else 0) | (2 if best >= 0 else 0)
    return dict(flags=flags, cls=cls, eff_width=eff, cp=best, ratio=best_ratio)
