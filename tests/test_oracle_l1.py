"""Pins of the oracle's L1 iteration-window detector.

Pinned by: hand-worked series (tests/golden/l1_series.json), an exact
rational brute force (fractions.Fraction, statistics.median_low) on random
short series, boundary cases of the ratio gate and of the change-point
tests, and recovery of planted host stalls on a seeded trace.
"""
import json
import os

import numpy as np
import pytest

import oracle
import tracegen
from tests import bruteforce as bf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _run(y, **p):
    y = np.asarray(y, np.int64)
    return oracle.iter_windows(y, 1, len(y), **p)


@pytest.mark.parametrize("case", json.load(open(os.path.join(GOLDEN, "l1_series.json")))["cases"],
                         ids=lambda c: c["name"])
def test_golden_series(case):
    out = _run(case["y"])
    assert out["cls"][0] == case["cls"]
    assert out["eff_width"][0] == case["eff_width"]
    assert out["cp"][0] == case["cp"]
    assert out["flags"].tolist() == case["flags"]


def test_change_point_ratio_value():
    out = _run([100] * 6 + [200] * 6)
    assert out["cp_ratio"][0] == np.float32(2.0)


def test_bruteforce_random_series():
    rng = np.random.default_rng(5)
    for trial in range(400):
        S = int(rng.integers(1, 14))
        base = int(rng.integers(1, 10**6))
        y = (base * (1 + 0.04 * rng.standard_normal(S))).astype(np.int64).clip(0)
        kind = trial % 4
        if kind == 1 and S > 2:
            y[rng.integers(0, S)] *= int(rng.integers(2, 4))
        elif kind == 2 and S > 3:
            t = int(rng.integers(1, S))
            y[t:] = y[t:] * int(rng.integers(13, 25)) // 10
        elif kind == 3:
            y = rng.integers(0, 5, size=S).astype(np.int64)  # tiny values, zeros included
        W = int(rng.integers(1, 7))
        p = dict(W=W, theta_pm=1500, beta_pm=1200, rho_pm=1300, cmax_pm=100, min_seg=int(rng.integers(1, 3)))
        out = _run(y, **p)
        ref = bf.iter_windows([int(v) for v in y], **p)
        assert out["flags"].tolist() == ref["flags"], (y, p)
        assert (out["cls"][0], out["eff_width"][0], out["cp"][0]) == (ref["cls"], ref["eff_width"], ref["cp"]), (y, p)
        if ref["cp"] >= 0:
            assert out["cp_ratio"][0] == np.float32(float(ref["ratio"]))


def test_ratio_gate_is_strict():
    # max/min exactly theta is not a candidate window
    assert _run([100, 150, 100, 100, 100], W=2)["flags"].tolist() == [0, 0, 0, 0, 0]
    assert _run([100, 151, 100, 100, 100], W=2)["flags"].tolist() == [1, 3, 1, 0, 0]


def test_zero_series_and_zero_left_side():
    assert _run([0, 0, 0, 0, 0, 0])["cls"][0] == 0
    # left mean zero: the regression ratio is undefined, no change point there
    out = _run([0, 0, 0, 5, 5, 5])
    assert out["cp"][0] == -1


def test_out_of_domain_series():
    out = _run([100, -1, 100])
    assert out["cls"][0] == 0x80 and not out["flags"].any() and out["cp"][0] == -1
    out = _run([100, 2**40, 100])
    assert out["cls"][0] == 0x80
    assert _run([100, 2**40 - 1, 100])["cls"][0] != 0x80


def test_relative_std_boundary():
    # right side [100, 110]: relative sample std = 7.07/105 = 0.0673; left
    # side [60, 60]: zero. Ratio 105/60 = 1.75. cmax 0.067 rejects, 0.068 accepts.
    y = [60, 60, 100, 110]
    assert _run(y, cmax_pm=67, W=1)["cp"][0] == -1
    assert _run(y, cmax_pm=68, W=1)["cp"][0] == 2


def test_degenerate_lengths():
    assert _run([123])["cls"][0] == 0
    out = oracle.iter_windows(np.zeros(0, np.int64), 3, 0)
    assert out["cls"].tolist() == [0, 0, 0]


def test_recovery_of_stalled_steps():
    trace = tracegen.make("medium", n_ranks=24, n_steps=8)
    cfg = trace.cfg
    sm = oracle.summarize(trace.fill_host(), cfg.n_kernels, cfg.n_streams)
    out = oracle.iter_windows(sm["step_ns"], cfg.n_ranks, cfg.n_steps)
    flags = out["flags"].reshape(cfg.n_ranks, cfg.n_steps)
    got = {(int(r), int(s)) for r, s in zip(*np.nonzero(flags & 2))}
    assert got == trace.truth()["anomalous"]
    for r, _ in got:
        assert out["cls"][r] == 1 and out["eff_width"][r] == 1
    assert (out["cls"][[r for r in range(cfg.n_ranks) if r not in {a for a, _ in got}]] == 0).all()
