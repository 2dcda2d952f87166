"""The oracle's KDE against Eq. 1 evaluated without its quantisations.

The oracle (and the GPU path) reads section 5.2 with three quantisations:
each log-duration is floored onto the 1/64-octave grid before the density is
formed, the bandwidth is rounded to 1/256 grid step, and the Gaussian weights
are 16-bit integers. Here Eq. 1 is evaluated as printed, in float64: the
Gaussian kernel at the raw log-durations u_i = 64 log2 d_i, with
h = 1.06 sigma n^(-1/5) from the sample standard deviation of the raw u_i,
at the centre of every grid cell (the binned density at grid point j stands
for the raw density at j + 1/2, since flooring moves each sample down by half
a cell on average). The same valley, filter and cap rules (the library's
readings, restated below) turn both densities into clusters; a sample
belongs to the cluster of its grid cell in both.

What is asserted, per group:
* both give the same number of clusters;
* every boundary of the oracle lies within one grid step of the unbinned
  one, or the cells between the two hold no sample (a zero-density gap,
  where the exact minimum and the middle of the quantised zero run differ),
  or Eq. 1's own density at the oracle's boundary exceeds its value at its
  own valley by at most FLAT = 1e-3 (a flat valley bottom between
  overlapping modes, where the argmin is ill-conditioned: the worst seen is
  5.4e-4, a 3-step shift);
* the cluster counts differ only by the samples in the cells between paired
  boundaries ("moved" samples), bounded over each test's groups: 1e-3 of all
  samples for random overlapping mixtures (worst seen 6.5e-4), none for the
  tiny trace and 1e-5 for rank-steps of the other workloads (at most 3 of
  700,000 seen);
* where the counts agree, p50 (lower median) and p99 (nearest rank) of the
  oracle equal those of the sorted raw durations of the unbinned clusters.
"""
import math

import numpy as np
import pytest

import oracle
import tracegen

P = oracle.KDE_DEFAULTS
FLAT = 1e-3  # relative excess of Eq. 1's density allowed at a displaced boundary
SQRT_2PI = math.sqrt(2.0 * math.pi)


def exact_bin(d: int, s: int = 6) -> int:
    """floor(2^s log2 d') with d' = d truncated to 24 significant bits (the
    grid's cells), by exact integer arithmetic."""
    if d < 2:
        return 0
    e = d.bit_length() - 1
    if e > 23:
        d = (d >> (e - 23)) << (e - 23)
    return (d ** (1 << s)).bit_length() - 1


def eq1_density(u, lo, hi, h):
    """Eq. 1, (1/n) sum_i K((x - u_i) / h) / h with the Gaussian kernel, at
    x = j + 1/2 for every grid point j in [lo, hi]."""
    x = np.arange(lo, hi + 1, dtype=np.float64) + 0.5
    f = np.zeros(x.size)
    for a in range(0, u.size, 4096):
        z = (x[:, None] - u[None, a:a + 4096]) / h
        f += np.exp(-0.5 * z * z).sum(axis=1)
    return f / (u.size * h * SQRT_2PI)


def valleys(f):
    """(position, value) of every maximal run of equal values strictly below
    both neighbouring values, at the middle of the run (rounded down)."""
    out, j, G = [], 1, len(f)
    while j <= G - 2:
        if f[j] < f[j - 1]:
            k = j
            while k + 1 < G and f[k + 1] == f[j]:
                k += 1
            if k + 1 < G and f[k + 1] > f[j]:
                out.append(((j + k) // 2, f[j]))
            j = k + 1
        else:
            j += 1
    return out


def apply_filters(cands, cells, n, G, frac_pm, min_count, gap, maxc):
    """The library's readings of the two filters of section 5.2 and its cap.
    cands: [(grid index, density)], cells: samples per grid index."""
    pos = [p for p, _ in cands]
    val = [v for _, v in cands]
    pref = np.concatenate([[0], np.cumsum(cells)])

    def size(a, b):  # samples in grid indices a..b
        return int(pref[b + 1] - pref[a])

    def drop_between(q, m):  # q: a gap/cluster index 0..m, drop one of its valleys
        if q == 0:
            return 0
        if q == m:
            return m - 1
        return q - 1 if val[q - 1] > val[q] else q

    need = max(min_count, (frac_pm * n + 999) // 1000)
    while pos:
        m = len(pos)
        sizes = [size(0 if q == 0 else pos[q - 1] + 1, G - 1 if q == m else pos[q]) for q in range(m + 1)]
        best = int(np.argmin(sizes))  # first minimum
        if sizes[best] >= need:
            break
        i = drop_between(best, m)
        del pos[i], val[i]
    while pos:
        m = len(pos)
        bounds = [0] + pos + [G - 1]
        hit = next((q for q in range(m + 1) if bounds[q + 1] - bounds[q] < gap), None)
        if hit is None:
            break
        i = drop_between(hit, m)
        del pos[i], val[i]
    while len(pos) > maxc - 1:
        i = max(range(len(pos)), key=lambda q: (val[q], q))  # largest density, the upper one on ties
        del pos[i], val[i]
    return pos


def eq1_clusters(d, s=P["sub_bits"], frac_pm=P["frac_pm"], min_count=P["min_count"], gap=P["gap"]):
    d = np.sort(np.asarray(d, dtype=np.uint64))
    n = d.size
    x = np.array([exact_bin(int(v), s) for v in d], dtype=np.int64)
    lo, hi = int(x[0]), int(x[-1])
    G = hi - lo + 1
    cells = np.bincount(x - lo, minlength=G)
    bounds, f = [], None
    if n >= 2 and G >= 3:
        u = (1 << s) * np.log2(np.maximum(d, 1).astype(np.float64))
        h = 1.06 * float(np.std(u, ddof=1)) * n ** -0.2
        if h > 0:
            f = eq1_density(u, lo, hi, h)
            bounds = apply_filters(valleys(f), cells, n, G, frac_pm, min_count, gap, oracle.KDE_MAXC)
    return {"bounds": bounds, "cells": cells, "x": x - lo, "d": d, "G": G, "f": f}


def _p50_p99(v):
    m = v.size
    return int(v[(m - 1) // 2]), int(v[(99 * m + 99) // 100 - 1])


def compare(d, stats, **params):
    """Compare the oracle's clusters of group d with the unbinned Eq. 1
    clusters; returns the number of samples assigned differently. Asserts
    the structural agreement listed in the module docstring."""
    r = oracle.kde_group(d, debug=True, **params)
    e = eq1_clusters(d, **params)
    n = e["d"].size
    if n == 0:
        assert r["n_clusters"] == 0
        return 0
    # the oracle's final boundaries: the grid index ending each cluster
    ncl = r["n_clusters"]
    ocounts = [int(c) for c in r["count"][:ncl]]
    ob = list(np.searchsorted(np.cumsum(e["cells"]), np.cumsum(ocounts)[:-1], side="left"))
    eb = e["bounds"]
    assert ncl == len(eb) + 1, ("cluster count", ncl, len(eb) + 1, ob, eb)
    pref = np.concatenate([[0], np.cumsum(e["cells"])])
    moved = 0
    for bo, br in zip(ob, eb):
        a, b = min(bo, br), max(bo, br)
        between = int(pref[b + 1] - pref[a + 1])  # samples in cells a+1..b
        # the unbinned density at the oracle's boundary, relative to its value
        # at its own valley: the oracle's boundary is a near-minimum of Eq. 1
        excess = float(e["f"][bo] / e["f"][br] - 1.0)
        assert b - a <= 1 or between == 0 or excess <= FLAT, ("boundary", bo, br, between, excess)
        moved += between
        if between:
            stats["max_shift"] = max(stats.get("max_shift", 0), b - a)
            stats["max_excess"] = max(stats.get("max_excess", 0.0), excess)
    # counts and percentiles of the unbinned partition
    edges = [0] + [int(pref[b + 1]) for b in eb] + [n]
    ecounts = [edges[q + 1] - edges[q] for q in range(len(edges) - 1)]
    diff = sum(abs(a - b) for a, b in zip(ocounts, ecounts))
    assert diff <= 2 * moved, (ocounts, ecounts, moved)
    if ocounts == ecounts:
        for q in range(ncl):
            p50, p99 = _p50_p99(e["d"][edges[q]:edges[q + 1]])
            assert (int(r["p50_ns"][q]), int(r["p99_ns"][q])) == (p50, p99), q
    stats["groups"] = stats.get("groups", 0) + 1
    stats["samples"] = stats.get("samples", 0) + n
    stats["moved"] = stats.get("moved", 0) + moved
    stats["multi"] = stats.get("multi", 0) + (ncl > 1)
    stats["differing_groups"] = stats.get("differing_groups", 0) + (ocounts != ecounts)
    return moved


def _lognormal(rng, m, median, sigma):
    return np.exp(np.log(median) + sigma * rng.normal(0, 1, m)).astype(np.uint64)


def test_eq1_density_reference_itself():
    # the reference density is a normalised Gaussian mixture: it integrates
    # to 1 over a wide grid, and with one sample it is the normal density
    u = np.array([640.0])
    f = eq1_density(u, 600, 700, 5.0)
    x = np.arange(600, 701) + 0.5
    assert np.allclose(f, np.exp(-0.5 * ((x - 640) / 5) ** 2) / (5 * SQRT_2PI), rtol=1e-12)
    rng = np.random.default_rng(0)
    u = rng.normal(1000, 20, 5000)
    f = eq1_density(u, 850, 1150, 4.0)
    assert abs(f.sum() - 1.0) < 1e-6


@pytest.mark.parametrize("seed", range(12))
def test_mixtures_match_unbinned_eq1(seed):
    """Uni-, bi- and trimodal lognormal mixtures: separated, close (shallow
    valleys) and unbalanced components, sigma 0.05-0.3 in ln."""
    rng = np.random.default_rng(1000 + seed)
    stats = {}
    for rep in range(25):
        k = int(rng.integers(1, 4))
        sizes = rng.integers(20, 3000, k)
        sep = float(rng.uniform(0.6, 3.0))  # octaves between components
        sig = float(rng.uniform(0.05, 0.3))
        base = float(rng.uniform(2e3, 2e6))
        d = np.concatenate([_lognormal(rng, int(m), base * 2 ** (sep * i), sig) for i, m in enumerate(sizes)])
        compare(d, stats)
    assert stats["moved"] <= 1e-3 * stats["samples"], stats


@pytest.mark.parametrize("n", [3, 10, 64, 300, 5000, 40000])
def test_unimodal_match_unbinned_eq1(n):
    rng = np.random.default_rng(n)
    stats = {}
    for rep in range(6):
        compare(_lognormal(rng, n, float(rng.uniform(3e3, 3e6)), 0.1), stats)
    assert stats["moved"] == 0 and stats["differing_groups"] == 0, stats


def _groups(trace, segs):
    """(segment, kernel id, durations) of every present group of the given
    rank-steps (segment indices), from the host generator."""
    for g in segs:
        ev = trace.fill_host(g, g + 1)
        kid, d = ev["kernel_id"], (ev["end_ns"] - ev["start_ns"]).astype(np.uint64)
        order = np.argsort(kid, kind="stable")
        kk, dd = kid[order], d[order]
        ks, starts = np.unique(kk, return_index=True)
        ends = np.append(starts[1:], kk.size)
        for k, s0, s1 in zip(ks, starts, ends):
            yield g, int(k), dd[s0:s1]


def test_tiny_trace_groups_match_unbinned_eq1():
    trace = tracegen.make("tiny")
    stats = {}
    for g, k, d in _groups(trace, list(range(trace.cfg.n_segments))):
        compare(d, stats)
    assert stats["groups"] == 8 * 4 * 64 and stats["multi"] > 0
    assert stats["moved"] == 0, stats


@pytest.mark.parametrize("workload,segs", [("medium", [0, 9, 100, 517, 1024, 1500, 2047]), ("production", [0, 513]),
                                           ("cluster", [3, 4000]), ("skew", [0, 7])])
def test_trace_groups_match_unbinned_eq1(workload, segs):
    """Every kernel of a few rank-steps of the larger workloads: Zipf ids
    (groups of 10 to about 70,000 durations, modes at 1x, 3x and 9x of a
    position's scale) and the skew workload's heavy-tailed Pareto hot ids."""
    trace = tracegen.make(workload)
    stats = {}
    for g, k, d in _groups(trace, segs):
        compare(d, stats)
    assert stats["groups"] > 400 * len(segs) and stats["multi"] > 0
    assert stats["moved"] <= 1e-5 * stats["samples"], stats
