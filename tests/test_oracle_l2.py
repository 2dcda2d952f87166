"""Pins of the oracle's group-aware L2 comparison (section 6.1 routing table,
Appendix B, Eq. 5) against values fixed outside the oracle:

* exact rational brute force (fractions.Fraction, statistics.variance) of
  every group's size, CV class and every rank's straggler flag on random
  groups, with the reported mean / std / CV / z against those exact values;
* numpy's mean and std(ddof=1) on a plain group;
* the closed form z = (n - 1) / sqrt(n) of one outlier among equal values,
  flagged at z > 3 exactly when n >= 11, and at thresholds just below / just
  above the closed form;
* CV class boundaries worked by hand (CV exactly 0.02 and 0.05);
* routing, membership (duplicates, malformed groups), absent cells and the
  2^40 ns domain;
* recovery of the medium trace's planted stragglers inside their
  data-parallel groups.
"""
import math
import statistics
from fractions import Fraction

import numpy as np
import pytest

import oracle
import tracegen

NE = oracle.L2_NOT_EVALUATED


def _one_group(xs, **params):
    """One step, one event routed to dimension 0, one group of all ranks."""
    R = len(xs)
    cnt = np.ones(R, np.uint32)
    sm = np.asarray(xs, np.int64)
    off = np.array([[0, R]], np.int32)
    mem = np.arange(R, dtype=np.int32).reshape(1, R)
    return oracle.l2(cnt, sm, R, 1, 1, np.zeros(1, np.uint8), off, mem, **params)


def test_numpy_mean_std():
    xs = [1000, 1100, 990, 1020, 1500, 1010]
    r = _one_group(xs)
    assert r["mean_ns"][0] == pytest.approx(np.mean(xs), rel=1e-15)
    assert r["std_ns"][0] == pytest.approx(np.std(xs, ddof=1), rel=1e-14)
    assert r["cv"][0] == pytest.approx(np.std(xs, ddof=1) / np.mean(xs), rel=1e-14)
    z = (np.asarray(xs) - np.mean(xs)) / np.std(xs, ddof=1)
    assert np.allclose(r["z"], z, rtol=1e-6)


@pytest.mark.parametrize("n", [3, 5, 10, 11, 12, 40])
def test_one_outlier_closed_form(n):
    xs = [10_000] * n
    xs[n // 3] = 13_000
    r = _one_group(xs)
    z = (n - 1) / math.sqrt(n)
    assert r["z"][n // 3] == pytest.approx(z, rel=1e-6)
    assert r["z"][0] == pytest.approx(-1 / math.sqrt(n), rel=1e-6)
    flagged = np.nonzero(r["flags"] & 2)[0].tolist()
    assert flagged == ([n // 3] if n >= 11 else [])
    assert r["n_strag"][0] == len(flagged)
    # a threshold just below / above the closed form
    zpm = int(z * 1000)
    assert r is not None
    assert (_one_group(xs, z_pm=zpm)["flags"][n // 3] & 2) == 2
    assert (_one_group(xs, z_pm=zpm + 1)["flags"][n // 3] & 2) == 0


@pytest.mark.parametrize("d,cls", [(99, 0), (100, 1), (249, 1), (250, 2)])
def test_cv_class_boundaries(d, cls):
    # values m - d, m, m + d have sample std d, so CV = d / m exactly
    r = _one_group([5000 - d, 5000, 5000 + d])
    assert r["cls"][0] == cls
    assert r["cv"][0] == pytest.approx(d / 5000, rel=1e-15)


def test_identical_and_zero_groups():
    r = _one_group([7000] * 6)
    assert r["cls"][0] == 0 and r["std_ns"][0] == 0 and (r["z"] == 0).all() and (r["flags"] == 1).all()
    r = _one_group([0] * 4)
    assert r["cls"][0] == 0 and r["mean_ns"][0] == 0 and r["cv"][0] == 0


def test_routing_membership_and_domain():
    R, S, E = 6, 2, 3
    cnt = np.ones(R * S * E, np.uint32)
    sm = np.full(R * S * E, 5000, np.int64)
    sm[((1 * S + 0) * E + 1)] = 9000
    cnt[((2 * S + 1) * E + 1)] = 0                # absent cell
    sm[((3 * S + 1) * E + 1)] = 1 << 41           # out of the domain
    route = np.array([0xFF, 0, 1], np.uint8)      # event 0 not compared
    # dim 0: groups {0,1,2} {3,4,5}; dim 1: {0..5} with rank 2 listed twice
    off = np.array([[0, 3, 6], [0, 6, 6]], np.int32)
    mem = np.array([[0, 1, 2, 3, 4, 5], [0, 1, 2, 3, 2, 5]], np.int32)
    r = oracle.l2(cnt, sm, R, S, E, route, off, mem, min_group=2)
    assert r["status"] == 2 | 4
    cls = r["cls"].reshape(S, E, 2)
    n = r["n"].reshape(S, E, 2)
    assert (cls[:, 0] == NE).all()
    assert n[0, 1].tolist() == [3, 3] and n[1, 1].tolist() == [2, 2]  # absent, out of domain
    assert n[0, 2].tolist() == [5, 0] and cls[0, 2, 1] == NE          # rank 4 is not listed in dim 1
    fl = r["flags"].reshape(R, S, E)
    assert fl[4, :, 2].tolist() == [0, 0]
    assert (fl[:, :, 0] == 0).all()
    # malformed group range and member id
    off2 = np.array([[0, 4, 2], [0, 6, 6]], np.int32)
    mem2 = np.array([[0, 1, 9, 3, 4, 5], [0, 1, 2, 3, 4, 5]], np.int32)
    r2 = oracle.l2(cnt, sm, R, S, E, route, off2, mem2, min_group=2)
    assert r2["status"] & 1
    assert r2["n"].reshape(S, E, 2)[0, 1].tolist() == [3, 0]


def _exact(xs):
    n = len(xs)
    mu = Fraction(sum(xs), n)
    var = statistics.variance([Fraction(x) for x in xs])
    return mu, var


@pytest.mark.parametrize("seed", range(6))
def test_rational_bruteforce(seed):
    rng = np.random.default_rng(seed)
    R, S, E = int(rng.integers(3, 30)), 2, 5
    cnt = rng.integers(0, 4, size=R * S * E).astype(np.uint32)
    base = rng.integers(1000, 10**9, size=E)
    sm = np.zeros(R * S * E, np.int64)
    for c in range(R * S * E):
        e = c % E
        sm[c] = int(cnt[c]) * int(base[e] * rng.uniform(0.9, 1.4))
    n_dims, G = 3, 4
    off = np.zeros((n_dims, G + 1), np.int32)
    mem = np.zeros((n_dims, R), np.int32)
    for d in range(n_dims):
        perm = rng.permutation(R)
        cuts = np.sort(rng.integers(0, R + 1, size=G - 1))
        off[d, 1:G] = cuts
        off[d, G] = R
        mem[d] = perm
    mem[1, 0] = mem[1, R - 1]                           # a duplicate listing
    route = rng.integers(0, n_dims + 1, size=E).astype(np.uint8)
    route[route == n_dims] = 0xFF
    p = dict(min_group=2, cv_mild_pm=int(rng.integers(5, 60)), cv_severe_pm=int(rng.integers(60, 200)),
             z_pm=int(rng.integers(500, 2500)))
    r = oracle.l2(cnt, sm, R, S, E, route, off, mem, **p)
    for s in range(S):
        for e in range(E):
            d = route[e]
            for g in range(G):
                o = (s * E + e) * G + g
                if d == 0xFF:
                    assert r["cls"][o] == NE and r["n"][o] == 0
                    continue
                seen, xs, rk = set(), [], []
                for i in range(off[d, g], off[d, g + 1]):
                    m = int(mem[d, i])
                    if m in seen or any(m in mem[d, off[d, h]:off[d, h + 1]] for h in range(g)):
                        continue
                    seen.add(m)
                    c = (m * S + s) * E + e
                    if cnt[c]:
                        xs.append(int(sm[c]) // int(cnt[c]))
                        rk.append(m)
                assert r["n"][o] == len(xs)
                if len(xs) < 2:
                    assert r["cls"][o] == NE
                    continue
                mu, var = _exact(xs)
                cv2 = var / (mu * mu) if mu > 0 else Fraction(0)
                exp_cls = 0 if cv2 < Fraction(p["cv_mild_pm"], 1000) ** 2 else (
                    1 if cv2 < Fraction(p["cv_severe_pm"], 1000) ** 2 else 2)
                assert r["cls"][o] == exp_cls
                assert r["mean_ns"][o] == pytest.approx(float(mu), rel=1e-15)
                assert r["std_ns"][o] == pytest.approx(math.sqrt(var), rel=1e-14)
                thr = Fraction(p["z_pm"], 1000)
                nst = 0
                for x, m in zip(xs, rk):
                    c = (m * S + s) * E + e
                    strag = x > mu and var > 0 and (x - mu) ** 2 > thr * thr * var
                    assert bool(r["flags"][c] & 2) == strag
                    assert r["flags"][c] & 1
                    nst += strag
                    if var > 0:
                        assert r["z"][c] == pytest.approx(float((x - mu) / Fraction(math.sqrt(var))), rel=1e-6,
                                                          abs=1e-6)
                assert r["n_strag"][o] == nst


def test_planted_stragglers_in_dp_groups():
    t = tracegen.make("medium")
    c = t.cfg
    R, S, K = c.n_ranks, c.n_steps, c.n_kernels
    so = oracle.summarize(t.fill_host(), K, c.n_streams)
    off, mem, _ = tracegen.parallel_groups(R, tp=2, pp=4, ep=4)
    route = np.full(K, 2, np.uint8)  # every kernel compared across its data-parallel group (32 ranks)
    r = oracle.l2(so["count"], so["sum_ns"], R, S, K, route, off, mem)
    fl = r["flags"].reshape(R, S, K)
    ev = (fl & 1) > 0
    strag = sorted(t.truth()["stragglers"])
    frac = (fl[strag] & 2).sum(axis=(1, 2)) / 2 / ev[strag].sum(axis=(1, 2))
    assert (frac >= 0.9).all(), frac
    others = np.setdiff1d(np.arange(R), strag)
    assert (fl[others] & 2).sum() / 2 <= 0.01 * ev[others].sum()
