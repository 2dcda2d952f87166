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
trace, and the production and cluster workloads at full size in the launch
configuration the benchmark times, checked on sampled kernels.
"""
import gc

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


def _both(ncl, cnt, a, b, R, S, K, what, **params):
    gw = pa.w1(_dev_clusters(ncl, cnt, a, b), R, S, K, **params)
    torch.cuda.synchronize()
    ow = oracle.w1(ncl, cnt, a, b, R, S, K, **params)
    assert_w1_equal(gw, ow, R, S, K, what)
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
    truth = t.truth()
    (strag,) = truth["stragglers"]
    flag = P.to_np(gw["flag"]).reshape(R, S, K)
    present = P.to_np(kd["n_clusters"]).reshape(R, S, K) > 0
    assert flag[strag].sum() >= 0.95 * present[strag].sum()
    for (pr, pk) in truth["pairs"]:
        assert flag[pr, :, pk].all()


def _full_size(name, n_sample):
    _announce(f"w1 full size {name}: GPU summarize -> kde -> w1, {n_sample} sampled kernels")
    t = tracegen.make(name)
    c = t.cfg
    R, S, K, NS = c.n_ranks, c.n_steps, c.n_kernels, c.n_streams
    ev = t.fill_device(device=DEV)
    s = pa.summarize(ev, R, S, K, NS)
    kd = pa.kde(ev, s, R, S, K, NS)
    gw = pa.w1(kd, R, S, K)
    torch.cuda.synchronize()
    assert int(gw["dev_status"].item()) == 0
    gw = {f: (v.cpu() if isinstance(v, torch.Tensor) else v) for f, v in gw.items() if f != "_workspace"}
    del ev, s, kd
    gc.collect()
    torch.cuda.empty_cache()
    print(f"[gpu-case] {name}: GPU chain done, oracle KDE over {c.n_segments} segments", flush=True)
    ko = P.oracle_kde_segments(t, range(c.n_segments))
    rng = np.random.default_rng(5)
    ks = np.sort(rng.choice(K, size=n_sample, replace=False))
    sl = lambda x, w: np.ascontiguousarray(np.asarray(x).reshape(R, S, K, *w)[:, :, ks])  # noqa: E731
    print(f"[gpu-case] {name}: oracle W1 on kernels {ks.tolist()}", flush=True)
    ow = oracle.w1(sl(ko["n_clusters"], ()), sl(ko["count"], (MAXC,)), sl(ko["p50_ns"], (MAXC,)),
                   sl(ko["p99_ns"], (MAXC,)), R, S, len(ks))
    n_amb = assert_w1_equal(gw, ow, R, S, K, f"{name} full", kernels=ks, max_ambiguous=2)
    print(f"[gpu-case] {name}: sampled kernels agree ({n_amb} flags within rounding of the fence)", flush=True)


@pytest.mark.timeout(900)
def test_w1_full_production():
    _full_size("production", 48)


@pytest.mark.timeout(1100)
def test_w1_full_cluster():
    _full_size("cluster", 3)
