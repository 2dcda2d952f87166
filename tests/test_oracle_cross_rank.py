"""Pins of the oracle's cross-rank step (per-kernel robust statistics, flags,
rank scores).

Pinned by: hand-worked order statistics (tests/golden/order_stats.json),
statistics.median_low / numpy.quantile(method="lower") on random inputs,
exact threshold boundaries worked by hand, the all-identical special case,
and recovery of every planted straggler and degraded pair in seeded traces.
"""
import json
import os

import numpy as np
import pytest

import oracle
import tracegen
from tests import bruteforce as bf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _from_x(x, count=10):
    """count/sum arrays with floor(sum/count) == x exactly."""
    x = np.asarray(x, dtype=np.int64)
    cnt = np.where(x >= 0, count, 0).astype(np.uint32)
    return cnt, np.where(x >= 0, x * count, 0).astype(np.int64)


def test_golden_order_statistics():
    cases = json.load(open(os.path.join(GOLDEN, "order_stats.json")))["cases"]
    for c in cases:
        x = c["x"]
        cnt, sm = _from_x(np.array(x)[:, None])  # R = len(x), S = 1, K = 1
        out = oracle.cross_rank(cnt, sm, len(x), 1, 1)
        assert (out["med_ns"][0], out["q1_ns"][0], out["q3_ns"][0], out["mad_ns"][0]) == \
            (c["med"], c["q1"], c["q3"], c["mad"]), c
        assert out["n_present"][0] == len(x)
        assert out["xmean_ns"][0] == np.float32(sum(x) / len(x))


def test_order_statistics_vs_library():
    rng = np.random.default_rng(11)
    R, S, K = 37, 3, 9
    x = rng.integers(1000, 3000, size=(R, S, K))
    absent = rng.random((R, S, K)) < 0.2
    cnt = rng.integers(1, 30, size=(R, S, K)).astype(np.uint32)
    cnt[absent] = 0
    sm = (x * cnt + rng.integers(0, 1, size=x.shape)).astype(np.int64)
    sm = sm + (cnt > 0) * rng.integers(0, np.maximum(cnt, 1))  # sum/count floors back to x
    out = oracle.cross_rank(cnt, sm, R, S, K)
    for s in range(S):
        for k in range(K):
            xs = [int(sm[r, s, k]) // int(cnt[r, s, k]) for r in range(R) if cnt[r, s, k] > 0]
            i = s * K + k
            med, q1, q3, mad = bf.order_stats(xs)
            assert out["n_present"][i] == len(xs)
            assert (out["med_ns"][i], out["q1_ns"][i], out["q3_ns"][i], out["mad_ns"][i]) == (med, q1, q3, mad)


def test_too_few_ranks_is_not_evaluated():
    cnt, sm = _from_x(np.array([[100], [-1], [300], [-1]]))
    out = oracle.cross_rank(cnt, sm, 4, 1, 1)
    assert out["n_present"][0] == 2
    assert out["med_ns"][0] == -1 and out["mad_ns"][0] == -1 and out["q1_ns"][0] == -1 and out["q3_ns"][0] == -1
    assert out["xmean_ns"][0] == 0.0
    assert not out["flags"].any() and not out["z"].any()
    assert out["mean_ns"].tolist() == [100.0, 0.0, 300.0, 0.0]
    assert (out["score_pm"] == -1).all() and not out["n_eval"].any()


def test_identical_ranks():
    R, K = 16, 12
    x = np.tile(np.arange(1, K + 1) * 1000, (R, 1))[:, None, :]
    cnt, sm = _from_x(x)
    out = oracle.cross_rank(cnt, sm, R, 1, K)
    assert (out["mad_ns"] == 0).all()
    assert not out["z"].any()
    assert (out["flags"] == 4).all()  # evaluated, nothing else
    assert (out["score_pm"] == 1000).all() and (out["n_eval"] == K).all()
    assert not out["straggler"].any()


def test_mad_threshold_boundary():
    # x = 90, 95, 100, 105, 110, 115, X: med 105, mad 10 (golden), q1 95, q3 110.
    # bit0 needs 1000 (X - 105) > 5189 * 10, i.e. X >= 157.
    for X, want in [(156, 0), (157, 1)]:
        cnt, sm = _from_x(np.array([90, 95, 100, 105, 110, 115, X])[:, None, None], count=8)
        out = oracle.cross_rank(cnt, sm, 7, 1, 1)
        assert out["flags"][6] & 1 == want, X
        assert out["mad_ns"][0] == 10
    # count 7 < c_min_pair hides the same cell
    cnt, sm = _from_x(np.array([90, 95, 100, 105, 110, 115, 200])[:, None, None], count=7)
    assert oracle.cross_rank(cnt, sm, 7, 1, 1)["flags"][6] & 1 == 0


def test_iqr_fence_boundary():
    # fence: 1000 (X - q3) > 1500 (q3 - q1) with q1 = 95, q3 = 110: X >= 133
    for X, want in [(132, 0), (133, 2)]:
        cnt, sm = _from_x(np.array([90, 95, 100, 105, 110, 115, X])[:, None, None])
        out = oracle.cross_rank(cnt, sm, 7, 1, 1)
        assert out["flags"][6] & 2 == want, X


def test_ratio_guard_boundary():
    # mad 0 (madf 1): the 1.25x ratio guard binds: 1000 X >= 1250 * 100 needs X >= 125
    for X, want in [(124, 0), (125, 1)]:
        cnt, sm = _from_x(np.array([100] * 6 + [X])[:, None, None])
        out = oracle.cross_rank(cnt, sm, 7, 1, 1)
        assert out["flags"][6] & 1 == want, X


def test_robust_z_value():
    cnt, sm = _from_x(np.array([90, 95, 100, 105, 110, 115, 157])[:, None, None])
    out = oracle.cross_rank(cnt, sm, 7, 1, 1)
    # (157 - 105) / (1.4826 * 10)
    assert out["z"][6] == np.float32(52 / (1.4826 * 10))
    assert out["z"][0] == np.float32(-15 / (1.4826 * 10))


def test_straggler_boundary_and_degraded_pairs():
    R, K = 9, 10
    base = (np.arange(K) + 1) * 1000
    for mult_pm, want in [(1019, 0), (1020, 1)]:
        x = np.tile(base, (R, 1))
        x[4] = base * mult_pm // 1000
        x[2, 3] = base[3] * 2  # one degraded kernel on a normal rank
        cnt, sm = _from_x(x[:, None, :])
        out = oracle.cross_rank(cnt, sm, R, 1, K)
        assert out["score_pm"][4] == mult_pm
        assert out["straggler"].tolist() == [0, 0, 0, 0, want, 0, 0, 0, 0]
        flags = out["flags"].reshape(R, K)
        assert flags[2, 3] == 4 | 1 | 8 | 2
        assert out["n_degraded"][3] == 1 and out["n_flag"][3] == 1
        assert out["n_flag_rank"][2] == 1


def test_min_kernels_guard():
    R, K = 9, 7  # fewer than 8 evaluated kernels: never a straggler
    x = np.tile((np.arange(K) + 1) * 1000, (R, 1))
    x[0] *= 2
    cnt, sm = _from_x(x[:, None, :])
    out = oracle.cross_rank(cnt, sm, R, 1, K)
    assert out["score_pm"][0] == 2000 and out["straggler"][0] == 0
    # then every flagged cell of rank 0 counts as a degraded pair
    assert (out["flags"].reshape(R, K)[0] & 8).all()


def _recover(trace):
    cfg = trace.cfg
    ev = trace.fill_host()
    sm = oracle.summarize(ev, cfg.n_kernels, cfg.n_streams)
    R, S, K = cfg.n_ranks, cfg.n_steps, cfg.n_kernels
    xr = oracle.cross_rank(sm["count"], sm["sum_ns"], R, S, K)
    return sm, xr


@pytest.mark.parametrize("name,over", [
    ("tiny", {}),
    ("medium", dict(n_ranks=32, n_steps=4)),
    ("cluster", dict(n_ranks=48, n_stragglers=2, n_pairs=6)),
    ("skew", dict(n_ranks=24, n_steps=2)),
])
def test_recovery_of_planted_faults(name, over):
    trace = tracegen.make(name, **over)
    truth = trace.truth()
    R, S, K = trace.cfg.n_ranks, trace.cfg.n_steps, trace.cfg.n_kernels
    _, xr = _recover(trace)
    strag = xr["straggler"].reshape(R, S)
    flags = xr["flags"].reshape(R, S, K)
    for s in range(S):
        assert set(np.nonzero(strag[:, s])[0].tolist()) == truth["stragglers"], s
        got_pairs = {(int(r), int(k)) for r, k in zip(*np.nonzero(flags[:, s, :] & 8))}
        assert got_pairs == truth["pairs"], s
