"""Pins of the oracle's cross-rank W1 scores (section 6.2, Eq. 2 - 4):

* the reconstructed mixture CDF against the normal distribution (scipy):
  0.5 at p50, Phi(2.326) at p99, count weights between separated clusters,
  unit steps for point masses;
* W1 of two lognormals of equal shape against the closed form of the
  integral of their CDF difference over the grid range (lognormal partial
  expectations);
* the exact score relation of one outlier among identical ranks, and its
  flag;
* a pure-Python recomputation of grid bounds, pairwise sums, scores,
  quartiles, fence and flags on small random cluster sets;
* recovery of planted stragglers and degraded pairs from oracle clusters of
  a seeded trace.
"""
import math

import numpy as np
import pytest
from scipy.stats import norm

import oracle
import tracegen

MAXC = oracle.KDE_MAXC
Z99 = 2.326


def test_cdf_reconstruction_points():
    assert oracle.w1_cdf_q([10], [1000], [2000], 1000.0) == 32768
    for p50, p99 in [(1000, 2000), (50_000, 51_000), (7, 300)]:
        expect = math.floor(65536 * norm.cdf(Z99))
        assert abs(oracle.w1_cdf_q([5], [p50], [p99], float(p99)) - expect) <= 1
    # two far-apart clusters weighted 3:1
    assert oracle.w1_cdf_q([3, 1], [1000, 10**9], [1100, 1.1e9], 1e6) == 49152
    # a point mass is a unit step at its value
    assert oracle.w1_cdf_q([4], [5000], [5000], 4999.0) == 0
    assert oracle.w1_cdf_q([4], [5000], [5000], 5000.0) == 65535


def _cells(ranks):
    """ranks: list of per-rank cluster lists [(count, p50, p99), ...]; S = K = 1."""
    R = len(ranks)
    ncl = np.zeros(R, np.uint8)
    cnt = np.zeros((R, MAXC), np.uint32)
    a = np.zeros((R, MAXC), np.int64)
    b = np.zeros((R, MAXC), np.int64)
    for r, cl in enumerate(ranks):
        ncl[r] = len(cl)
        for c, (n, x, y) in enumerate(cl):
            cnt[r, c], a[r, c], b[r, c] = n, x, y
    return ncl, cnt, a, b


def _int_cdf(lo, hi, m, s):
    """Closed form of the integral of the lognormal CDF F over [lo, hi]."""
    mu = math.log(m)
    F = lambda x: norm.cdf((math.log(x) - mu) / s)  # noqa: E731
    pm = lambda x: math.exp(mu + s * s / 2) * norm.cdf((math.log(x) - mu - s * s) / s)  # noqa: E731
    return hi * F(hi) - lo * F(lo) - (pm(hi) - pm(lo))


@pytest.mark.parametrize("m1,m2,ratio", [(100_000, 130_000, 1.3), (10_000, 11_000, 1.05), (5_000, 20_000, 2.0)])
def test_w1_of_two_lognormals_closed_form(m1, m2, ratio):
    s = math.log(ratio) / Z99
    ranks = [[(100, m1, round(m1 * ratio))], [(100, m2, round(m2 * ratio))]]
    r = oracle.w1(*_cells(ranks), 2, 1, 1, grid=256, min_ranks=2)
    lo, hi = int(r["lo_ns"][0]), int(r["hi_ns"][0])
    assert lo == (m1 * m1) // round(m1 * ratio)
    assert hi == -(-(round(m2 * ratio) ** 2) // m2)
    # F1 >= F2 everywhere (same shape, larger median): W1 = int F1 - int F2
    expect = _int_cdf(lo, hi, m1, s) - _int_cdf(lo, hi, m2, s)
    assert r["score"][0] == pytest.approx(expect, rel=2e-3)
    assert r["score"][1] == r["score"][0]


@pytest.mark.parametrize("n", [5, 9, 40])
def test_one_outlier_among_identical_ranks(n):
    normal = [(50, 20_000, 23_000), (10, 60_000, 66_000)]
    slow = [(50, 26_000, 30_000), (10, 78_000, 86_000)]
    ranks = [normal] * n
    ranks[n // 2] = slow
    r = oracle.w1(*_cells(ranks), n, 1, 1)
    sc = r["score"]
    d = sc[0]
    assert d > 0
    assert sc[n // 2] == pytest.approx((n - 1) * d, rel=1e-12)
    assert r["q1"][0] == d and r["q3"][0] == d and r["fence"][0] == d
    assert list(np.nonzero(r["flag"])[0]) == [n // 2] and r["n_flag"][0] == 1


def test_too_few_ranks_and_absent_cells():
    ranks = [[(5, 1000, 1100)], [], [(7, 1200, 1300)]]
    r = oracle.w1(*_cells(ranks), 3, 1, 1)
    assert r["n_present"][0] == 2 and r["score"].sum() == 0 and r["flag"].sum() == 0
    r = oracle.w1(*_cells(ranks), 3, 1, 1, min_ranks=2)
    assert r["score"][1] == 0 and r["score"][0] > 0 and r["score"][0] == r["score"][2]


def _python_reference(ncl, cnt, a, b, R, S, K, G, min_ranks, alpha_pm):
    out = {"score": np.zeros(R * S * K), "flag": np.zeros(R * S * K, np.uint8), "fence": np.zeros(S * K)}
    for s in range(S):
        for k in range(K):
            cells = [(r * S + s) * K + k for r in range(R)]
            pres = [c for c in cells if ncl[c] > 0]
            n = len(pres)
            if n < max(min_ranks, 2):
                continue
            lo, hi = None, 0
            for c in pres:
                for cl in range(ncl[c]):
                    x, y = max(int(a[c, cl]), 1), max(int(b[c, cl]), 1)
                    y = max(y, x)
                    lo = x * x // y if lo is None else min(lo, x * x // y)
                    hi = max(hi, min(-(-(y * y) // x), 2**63 - 1))
            lo = max(lo, 1)
            lnlo, lnhi = math.log(lo), math.log(hi)
            du = (lnhi - lnlo) / (G - 1)
            xs = [math.exp(lnlo + g * du) for g in range(G)]
            q = {c: [oracle.w1_cdf_q(cnt[c, :ncl[c]], a[c, :ncl[c]], b[c, :ncl[c]], xs[g]) for g in range(G)]
                 for c in pres}
            sc = {}
            for c in pres:
                acc = 0.0
                for g in range(G):
                    tot = sum(abs(q[c][g] - q[e][g]) for e in pres)
                    w = (xs[min(g + 1, G - 1)] - xs[max(g - 1, 0)]) / 2.0
                    acc += w * float(tot)
                sc[c] = acc / (65536.0 * (n - 1))
            v = sorted(sc.values())
            q1, q3 = v[(n - 1) // 4], v[3 * (n - 1) // 4]
            fence = q3 + alpha_pm * (q3 - q1) / 1000.0
            out["fence"][s * K + k] = fence
            for c in pres:
                out["score"][c] = sc[c]
                out["flag"][c] = sc[c] > fence
    return out


@pytest.mark.parametrize("seed", range(4))
def test_bruteforce_small(seed):
    rng = np.random.default_rng(seed)
    R, S, K = int(rng.integers(3, 9)), 2, 3
    C = R * S * K
    ncl = rng.integers(0, 4, size=C).astype(np.uint8)
    cnt = np.zeros((C, MAXC), np.uint32)
    a = np.zeros((C, MAXC), np.int64)
    b = np.zeros((C, MAXC), np.int64)
    for c in range(C):
        base = rng.uniform(1e3, 1e6)
        for cl in range(ncl[c]):
            cnt[c, cl] = rng.integers(1, 100)
            a[c, cl] = int(base * 3**cl * rng.uniform(0.9, 1.2))
            b[c, cl] = int(a[c, cl] * rng.choice([1.0, rng.uniform(1.01, 1.6)]))
    G = int(rng.choice([2, 7, 33]))
    r = oracle.w1(ncl, cnt, a, b, R, S, K, grid=G, min_ranks=3, alpha_pm=1500)
    ref = _python_reference(ncl, cnt, a, b, R, S, K, G, 3, 1500)
    assert np.allclose(r["score"], ref["score"], rtol=1e-12, atol=0)
    assert np.array_equal(r["flag"], ref["flag"])
    assert np.allclose(r["fence"], ref["fence"], rtol=1e-12, atol=0)


def test_planted_faults_flagged_from_oracle_clusters():
    t = tracegen.make("tiny")
    c = t.cfg
    R, S, K = c.n_ranks, c.n_steps, c.n_kernels
    kd = oracle.kde(t.fill_host(), K, c.n_streams)
    r = oracle.w1(kd["n_clusters"], kd["count"], kd["p50_ns"], kd["p99_ns"], R, S, K)
    flag = r["flag"].reshape(R, S, K)
    truth = t.truth()
    (strag,) = truth["stragglers"]
    present = kd["n_clusters"].reshape(R, S, K) > 0
    # the 1.3x straggler is flagged on (nearly) every kernel, each step
    assert flag[strag].sum() >= 0.95 * present[strag].sum()
    for (pr, pk) in truth["pairs"]:
        assert flag[pr, :, pk].all()
    others = np.setdiff1d(np.arange(R), [strag])
    assert flag[others].sum() <= 0.05 * present[others].sum()


def test_malformed_cluster_records_are_left_out():
    # a cell with more clusters than the record holds, and one whose cluster
    # counts sum to 0, take no part: the scores equal those of the same
    # ranks with the two cells absent
    good = [(20, 1000, 1100)]
    ranks = [good, [(20, 1300, 1400)], good, [(0, 5000, 6000)], good, [(7, 2000, 2100)]]
    ncl, cnt, a, b = _cells(ranks)
    ncl[5] = MAXC + 3
    r = oracle.w1(ncl, cnt, a, b, 6, 1, 1)
    assert r["malformed"] == 2 and r["n_present"][0] == 4
    ncl2 = ncl.copy()
    ncl2[3] = ncl2[5] = 0
    r2 = oracle.w1(ncl2, cnt, a, b, 6, 1, 1)
    assert r2["malformed"] == 0
    for f in ("score", "flag", "fence", "q1", "q3", "lo_ns", "hi_ns", "n_present"):
        assert np.array_equal(r[f], r2[f]), f
    assert r["score"][3] == 0 and r["score"][5] == 0
