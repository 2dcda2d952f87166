"""GPU parity of argus_w1 (section 6.2, Eq. 2 - 4) through the C ABI against
the CPU oracle.

Integer outputs (present ranks, grid bounds) must match exactly. Scores,
quartiles and fences are doubles computed by the same sequence of double
operations on both sides; they must agree within 1e-5 relative (they differ
only where the device's log / exp / erfc round differently from the host's).
Flags must match exactly except on a cell whose oracle score lies within
that tolerance of its fence, where either answer is correct (counted, and
required to be rare).

Cases: hand-built cluster sets (point masses, p99 below p50, non-positive
percentiles, durations near 2^63, identical ranks, one present rank, too few
ranks, malformed records, the smallest and a large grid, ragged rank counts
up to the 16,384-rank limit), W1 over the oracle's own KDE clusters of the
tiny and medium traces, the full GPU chain summarize -> kde -> w1 on the tiny
trace, and the production, cluster and skew workloads at full size in the
launch configuration the benchmark times: there every KDE cell is compared
with the oracle, and W1 on 48-64 kernels that include the ten heaviest ids
(the skew workload's eight hot Pareto ids among them).

The 16-bit CDF values the score is built from (the workspace) are compared
with the oracle's at sampled grid points of every case: they may differ by
one unit only where the mixture lies within rounding of a multiple of
1/65536 (device and host log / erfc differ in the last place), and the test
counts such points and bounds them.
"""
import gc
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
import paper_2606_20374_amd as pa
import tracegen
from tests import parity as P

pytestmark = pytest.mark.gpu
DEV = "cuda"
MAXC = pa.argus.KDE_MAXC
RTOL = 1e-5
INT_FIELDS = ["n_present", "lo_ns", "hi_ns"]
SK_FLOAT = ["q1", "q3", "fence"]


def _announce(name):
    print(f"\n[gpu-case] {name}", flush=True)


def _dev_clusters(ncl, cnt, a, b):
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x).reshape(-1)).to(DEV)  # noqa: E731
    return {"n_clusters": t(ncl.astype(np.uint8)), "count": t(cnt.astype(np.uint32).view(np.int32)),
            "p50_ns": t(a.astype(np.int64)), "p99_ns": t(b.astype(np.int64))}


def _close(g, o):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    return np.abs(g - o) <= RTOL * np.abs(o)


def assert_w1_equal(gw: dict, ow: dict, R, S, K, what, kernels=None, max_ambiguous=0):
    """gw: GPU output dict (torch); ow: oracle output over the kernels listed
    in `kernels` (all when None), laid out [R][S][len(kernels)]."""
    ks = np.arange(K) if kernels is None else np.asarray(kernels)
    nk = len(ks)
    sk_idx = (np.arange(S)[:, None] * K + ks[None, :]).reshape(-1)
    for f in INT_FIELDS:
        g = P.to_np(gw[f])[sk_idx]
        o = np.asarray(ow[f]).reshape(-1)
        assert np.array_equal(g.view(o.dtype) if g.dtype != o.dtype else g, o), (what, f)
    for f in SK_FLOAT:
        g = P.to_np(gw[f])[sk_idx]
        ok = _close(g, ow[f])
        assert ok.all(), (what, f, np.nonzero(~ok)[0][:5], g[~ok][:5], np.asarray(ow[f])[~ok][:5])
    score = P.to_np(gw["score"]).reshape(R, S, K)[:, :, ks].reshape(-1)
    flag = P.to_np(gw["flag"]).reshape(R, S, K)[:, :, ks].reshape(-1)
    osc = np.asarray(ow["score"]).reshape(-1)
    ofl = np.asarray(ow["flag"]).reshape(-1)
    ok = _close(score, osc)
    assert ok.all(), (what, "score", np.nonzero(~ok)[0][:5], score[~ok][:5], osc[~ok][:5])
    fence = np.broadcast_to(np.asarray(ow["fence"]).reshape(1, S, nk), (R, S, nk)).reshape(-1)
    amb = np.abs(osc - fence) <= RTOL * np.abs(fence)
    bad = (flag != ofl) & ~amb
    assert not bad.any(), (what, "flag", np.nonzero(bad)[0][:5])
    n_amb = int(((flag != ofl) & amb).sum())
    assert n_amb <= max_ambiguous, (what, "ambiguous flags", n_amb)
    # n_flag is the GPU's own flag count
    gnf = P.to_np(gw["n_flag"])[sk_idx]
    assert np.array_equal(gnf, flag.reshape(R, S, nk).sum(axis=0).reshape(-1).astype(gnf.dtype)), (what, "n_flag")
    if n_amb == 0:
        assert np.array_equal(gnf.view(np.uint32), np.asarray(ow["n_flag"]).reshape(-1)), (what, "n_flag oracle")
    return n_amb


def check_cdf_values(gw, ncl, cnt, a, b, R, S, K, what, n_points=4000, seed=0, kernels=None):
    """Sampled 16-bit CDF values of the workspace ([S][K][G][R]) against the
    oracle's at the same grid points. ncl/cnt/a/b: the clusters W1 ran on,
    [R][S][K] (cnt/a/b with KDE_MAXC slots). Returns the number of points
    that differ (by one unit at most)."""
    G = int(gw["_grid"])
    ncl = np.asarray(ncl).reshape(R, S, K)
    cnt = np.asarray(cnt).reshape(R, S, K, MAXC)
    a = np.asarray(a).reshape(R, S, K, MAXC)
    b = np.asarray(b).reshape(R, S, K, MAXC)
    npres = P.to_np(gw["n_present"]).reshape(S, K)
    lo = P.to_np(gw["lo_ns"]).reshape(S, K)
    hi = P.to_np(gw["hi_ns"]).reshape(S, K)
    ks = np.arange(K) if kernels is None else np.asarray(kernels)
    ev_sk = [(s, k) for s in range(S) for k in ks if npres[s, k] >= 3]
    if not ev_sk:
        return 0
    rng = np.random.default_rng(seed)
    pts = []
    while len(pts) < n_points:
        s, k = ev_sk[int(rng.integers(len(ev_sk)))]
        r = int(rng.integers(R))
        if 1 <= ncl[r, s, k] <= MAXC and cnt[r, s, k, :ncl[r, s, k]].sum() > 0:
            pts.append((s, k, int(rng.integers(G)), r))
    Rp = R + (R & 1)  # workspace rows: the rank count rounded up to even
    idx = torch.tensor([((s * K + k) * G + g) * Rp + r for s, k, g, r in pts], dtype=torch.int64)
    ws = gw["_workspace"].view(torch.int16)
    got = ws[idx.to(ws.device)].cpu().numpy().view(np.uint16).astype(np.int64)
    want = np.array([oracle.w1_cdf_q_grid(cnt[r, s, k, :ncl[r, s, k]], a[r, s, k, :ncl[r, s, k]],
                                          b[r, s, k, :ncl[r, s, k]], lo[s, k], hi[s, k], g, G)
                     for s, k, g, r in pts], dtype=np.int64)
    diff = np.abs(got - want)
    assert diff.max() <= 1, (what, "cdf values", pts[int(diff.argmax())], got[diff.argmax()], want[diff.argmax()])
    n_diff = int((diff > 0).sum())
    assert n_diff <= max(1, n_points // 1000), (what, "cdf values differing by one unit", n_diff)
    return n_diff


def _both(ncl, cnt, a, b, R, S, K, what, **params):
    gw = pa.w1(_dev_clusters(ncl, cnt, a, b), R, S, K, **params)
    torch.cuda.synchronize()
    ow = oracle.w1(ncl, cnt, a, b, R, S, K, **params)
    assert_w1_equal(gw, ow, R, S, K, what)
    check_cdf_values(gw, ncl, cnt, a, b, R, S, K, what, n_points=500)
    expect = pa.argus.DEV_W1_INPUT if ow["malformed"] else 0
    assert int(gw["dev_status"].item()) == expect, what
    return gw, ow


def _random_clusters(rng, R, S, K, p_absent=0.1, outliers=0.05, malformed=0):
    C = R * S * K
    ncl = rng.integers(1, MAXC + 1, size=C).astype(np.uint8)
    ncl[rng.random(C) < p_absent] = 0
    cnt = np.zeros((C, MAXC), np.uint32)
    a = np.zeros((C, MAXC), np.int64)
    b = np.zeros((C, MAXC), np.int64)
    base = np.exp(rng.uniform(np.log(2e3), np.log(5e6), size=K))
    slow = np.where(rng.random(R) < outliers, rng.uniform(1.05, 1.6, size=R), 1.0)
    for c in range(C):
        r, k = c // (S * K), c % K
        for cl in range(ncl[c]):
            cnt[c, cl] = rng.integers(1, 500)
            a[c, cl] = int(base[k] * 3**cl * slow[r] * rng.uniform(0.97, 1.03))
            b[c, cl] = int(a[c, cl] * (1.0 if rng.random() < 0.1 else rng.uniform(1.02, 1.6)))
    if malformed:
        idx = rng.choice(C, size=malformed, replace=False)
        for i, c in enumerate(idx):
            if i % 2:
                ncl[c] = MAXC + 1 + i % 200
            else:
                ncl[c] = max(ncl[c], 1)
                cnt[c, :] = 0
    return ncl, cnt, a, b


def _cells(ranks):
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


def test_w1_hand_built_groups():
    _announce("w1 hand-built groups")
    normal = [(50, 20_000, 23_000), (10, 60_000, 66_000)]
    slow = [(50, 26_000, 30_000), (10, 78_000, 86_000)]
    cases = {
        "one outlier": [normal] * 4 + [slow] + [normal] * 4,
        "identical": [normal] * 7,
        "point masses": [[(5, 1000, 1000)], [(5, 1000, 1000)], [(5, 1200, 1200)], [(3, 900, 900), (2, 5000, 5000)]],
        "p99 below p50, non-positive": [[(4, 5000, 100)], [(4, 0, -7)], [(4, -3, 2)], [(4, 4000, 4400)]],
        "near 2^63": [[(9, 2**62, 2**62 + 2**60)], [(9, 2**61, 2**62)], [(9, 2**40, 2**62)], [(9, 7, 2**63 - 1)]],
        "one present": [[(5, 1000, 1100)], [], []],
        "two present": [[(5, 1000, 1100)], [], [(5, 1300, 1500)]],
    }
    for name, ranks in cases.items():
        ncl, cnt, a, b = _cells(ranks)
        R = len(ranks)
        for params in (dict(), dict(min_ranks=2), dict(grid=2), dict(grid=2048, alpha_pm=0)):
            _both(ncl, cnt, a, b, R, 1, 1, f"{name} {params}", **params)


@pytest.mark.parametrize("R,S,K,seed", [(5, 3, 7, 0), (64, 2, 33, 1), (257, 1, 9, 2), (1000, 2, 5, 3),
                                         (1500, 1, 4, 4), (3001, 1, 3, 5), (16384, 1, 2, 6)])
def test_w1_random_cluster_sets(R, S, K, seed):
    _announce(f"w1 random clusters R={R} S={S} K={K}")
    rng = np.random.default_rng(seed)
    ncl, cnt, a, b = _random_clusters(rng, R, S, K, malformed=3 if R >= 64 else 0)
    _both(ncl, cnt, a, b, R, S, K, f"random {R}x{S}x{K}")


def test_w1_malformed_records_are_reported():
    _announce("w1 malformed records")
    rng = np.random.default_rng(11)
    ncl, cnt, a, b = _random_clusters(rng, 40, 2, 6, malformed=10)
    gw, ow = _both(ncl, cnt, a, b, 40, 2, 6, "malformed")
    assert ow["malformed"] == 10


def test_w1_on_oracle_kde_clusters():
    for name in ("tiny", "medium"):
        _announce(f"w1 over oracle KDE clusters, {name}")
        t = tracegen.make(name)
        c = t.cfg
        R, S, K = c.n_ranks, c.n_steps, c.n_kernels
        kd = P.oracle_kde_segments(t, range(c.n_segments))
        _both(kd["n_clusters"], kd["count"], kd["p50_ns"], kd["p99_ns"], R, S, K, f"{name} oracle clusters")


def test_w1_full_chain_tiny():
    _announce("w1 full GPU chain on the tiny trace")
    t = tracegen.make("tiny")
    c = t.cfg
    R, S, K, NS = c.n_ranks, c.n_steps, c.n_kernels, c.n_streams
    ev = t.fill_device(device=DEV)
    s = pa.summarize(ev, R, S, K, NS)
    kd = pa.kde(ev, s, R, S, K, NS)
    gw = pa.w1(kd, R, S, K)
    torch.cuda.synchronize()
    assert int(gw["dev_status"].item()) == 0
    ko = oracle.kde(t.fill_host(), K, NS)
    ow = oracle.w1(ko["n_clusters"], ko["count"], ko["p50_ns"], ko["p99_ns"], R, S, K)
    assert_w1_equal(gw, ow, R, S, K, "tiny chain")
    check_cdf_values(gw, ko["n_clusters"], ko["count"], ko["p50_ns"], ko["p99_ns"], R, S, K, "tiny chain")
    truth = t.truth()
    (strag,) = truth["stragglers"]
    flag = P.to_np(gw["flag"]).reshape(R, S, K)
    present = P.to_np(kd["n_clusters"]).reshape(R, S, K) > 0
    assert flag[strag].sum() >= 0.95 * present[strag].sum()
    for (pr, pk) in truth["pairs"]:
        assert flag[pr, :, pk].all()


def heaviest_ids(trace, n):
    """The n kernel ids with the most events in the workload's template."""
    counts = np.bincount(trace.tmpl_kid, minlength=trace.cfg.n_kernels)
    return np.argsort(-counts, kind="stable")[:n]


def oracle_w1_kernels(ko, R, S, K, ks, n_threads=None):
    """The oracle's W1 of kernels ks only (one pairwise oracle call per
    kernel, kernels in parallel host threads), laid out [R][S][len(ks)] and
    [S][len(ks)] as assert_w1_equal expects."""
    sl = lambda x, k, w: np.ascontiguousarray(np.asarray(x).reshape(R, S, K, *w)[:, :, k:k + 1])  # noqa: E731

    def one(k):
        return oracle.w1(sl(ko["n_clusters"], k, ()), sl(ko["count"], k, (MAXC,)), sl(ko["p50_ns"], k, (MAXC,)),
                         sl(ko["p99_ns"], k, (MAXC,)), R, S, 1)

    with ThreadPoolExecutor(n_threads or P.host_threads()) as ex:
        parts = list(ex.map(one, [int(k) for k in ks]))
    out = {}
    for f in ("n_present", "lo_ns", "hi_ns", "q1", "q3", "fence", "n_flag"):
        out[f] = np.stack([np.asarray(p[f]).reshape(S) for p in parts], axis=1).reshape(-1)  # [S][nk]
    for f in ("score", "flag"):
        out[f] = np.stack([np.asarray(p[f]).reshape(R, S) for p in parts], axis=2).reshape(-1)  # [R][S][nk]
    return out


def _full_size(name, n_sample, n_heavy=10):
    """GPU summarize -> kde -> w1 at full size; every KDE cell against the
    oracle, W1 on n_sample kernels: the n_heavy heaviest ids and random
    others."""
    _announce(f"w1 full size {name}: GPU summarize -> kde -> w1, all KDE cells, {n_sample} W1 kernels")
    t = tracegen.make(name)
    c = t.cfg
    R, S, K, NS = c.n_ranks, c.n_steps, c.n_kernels, c.n_streams
    ev = t.fill_device(device=DEV)
    s = pa.summarize(ev, R, S, K, NS)
    kd = pa.kde(ev, s, R, S, K, NS)
    gw = pa.w1(kd, R, S, K)
    torch.cuda.synchronize()
    assert int(kd["dev_status"].item()) == 0 and int(gw["dev_status"].item()) == 0
    kd_h = {f: kd[f].cpu() for f in P.KDE_FIELDS}
    ws = gw.pop("_workspace")
    gw = {f: (v.cpu() if isinstance(v, torch.Tensor) else v) for f, v in gw.items()}
    del ev, s, kd
    gc.collect()
    torch.cuda.empty_cache()
    print(f"[gpu-case] {name}: GPU chain done, oracle KDE over {c.n_segments} segments", flush=True)
    ko = P.oracle_kde_segments(t, range(c.n_segments))
    P.assert_kde_equal(kd_h, ko, f"{name} full-size KDE, every cell")
    del kd_h
    print(f"[gpu-case] {name}: all {c.n_segments * K} KDE cells agree", flush=True)
    rng = np.random.default_rng(5)
    heavy = heaviest_ids(t, n_heavy)
    rest = rng.choice(np.setdiff1d(np.arange(K), heavy), size=n_sample - len(heavy), replace=False)
    ks = np.sort(np.concatenate([heavy, rest]))
    print(f"[gpu-case] {name}: oracle W1 on kernels {ks.tolist()} (heaviest {sorted(heavy.tolist())})", flush=True)
    ow = oracle_w1_kernels(ko, R, S, K, ks)
    n_amb = assert_w1_equal(gw, ow, R, S, K, f"{name} full", kernels=ks, max_ambiguous=2)
    gw["_workspace"] = ws
    n_q = check_cdf_values(gw, ko["n_clusters"], ko["count"], ko["p50_ns"], ko["p99_ns"], R, S, K, f"{name} full",
                           n_points=20000, kernels=ks)
    print(f"[gpu-case] {name}: sampled kernels agree ({n_amb} flags within rounding of the fence, "
          f"{n_q} of 20000 CDF values one unit apart)", flush=True)


@pytest.mark.timeout(900)
def test_w1_full_production():
    _full_size("production", 48)


@pytest.mark.timeout(1100)
def test_w1_full_cluster():
    _full_size("cluster", 64)


@pytest.mark.timeout(1100)
def test_w1_full_skew():
    _full_size("skew", 64)
