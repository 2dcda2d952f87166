"""Pins of the oracle's summarize step (group-by per (segment, kernel id)).

Pinned by: the library bit_length (bins), brute force with dict-of-lists on
tiny traces, a closed form on a noise-free hand-built trace, summary
invariants on every segment of generated traces, and edge cases.
"""
import numpy as np
import pytest

import oracle
import tracegen
from tests import bruteforce as bf

NB = 32


def _ev(kid, st, t0, t1, lens):
    off = np.zeros(len(lens) + 1, np.int64)
    off[1:] = np.cumsum(lens)
    return {"kernel_id": np.asarray(kid, np.int32), "stream": np.asarray(st, np.int32),
            "start_ns": np.asarray(t0, np.int64), "end_ns": np.asarray(t1, np.int64), "seg_off": off}


def _compare_to_bruteforce(ev, K, NS):
    out = oracle.summarize(ev, K, NS)
    ref = bf.summarize(ev, K, NS)
    G = len(ev["seg_off"]) - 1
    for g in range(G):
        rg = ref[g]
        assert out["n_valid"][g] == rg["n_valid"]
        assert out["n_invalid"][g] == rg["n_invalid"]
        assert out["t_first"][g] == rg["t_first"]
        assert out["t_last"][g] == rg["t_last"]
        assert out["step_ns"][g] == rg["step"]
        assert out["busy_ns"][g] == rg["busy"]
        assert out["stream_busy_ns"][g].tolist() == rg["stream_busy"]
        assert out["wire_bytes"][g] == rg["wire"]
        for k in range(K):
            c = g * K + k
            cell = rg["cells"].get(k)
            if cell is None:
                assert out["count"][c] == 0 and out["sum_ns"][c] == 0
                assert out["min_ns"][c] == bf.I64_MAX and out["max_ns"][c] == bf.I64_MIN
                assert not out["hist"][c].any()
            else:
                assert out["count"][c] == cell["count"]
                assert out["sum_ns"][c] == cell["sum"]
                assert out["min_ns"][c] == cell["min"]
                assert out["max_ns"][c] == cell["max"]
                assert out["hist"][c].tolist() == cell["hist"]
    return out


def test_bin_matches_bit_length():
    vals = [0, 1, 2, 3, 4, 5, 7, 8, 1023, 1024, 1025, 2**31 - 1, 2**31, 2**31 + 1, 2**40, 2**63 - 1]
    vals += [2**k for k in range(64)] + [2**k - 1 for k in range(1, 64)]
    rng = np.random.default_rng(0)
    vals += [int(v) for v in rng.integers(0, 2**62, size=2000)]
    for v in vals:
        assert oracle.bin_of(v) == bf.bin_of(v), v


def test_bruteforce_generated_tiny_with_corruption():
    t = tracegen.make("tiny", n_ranks=3, n_steps=2, events_per_seg=700, tmpl_len=200, invalid_ppm=30_000)
    ev = t.fill_host()
    out = _compare_to_bruteforce(ev, t.cfg.n_kernels, t.cfg.n_streams)
    assert out["n_invalid"].sum() > 0  # corruption actually exercised


def test_bruteforce_skew_pareto():
    t = tracegen.make("skew", n_ranks=2, n_steps=2, events_per_seg=1500, tmpl_len=500, n_kernels=300)
    ev = t.fill_host()
    out = _compare_to_bruteforce(ev, t.cfg.n_kernels, t.cfg.n_streams)
    # Pareto kernels spread over several octave bins
    assert (np.count_nonzero(out["hist"], axis=1) >= 4).any()


def test_bruteforce_ragged_and_empty_segments():
    cfg = tracegen.config("tiny", n_ranks=3, n_steps=3, tmpl_len=100, invalid_ppm=50_000)
    t = tracegen.Trace(cfg, seg_lengths=[0, 1, 63, 64, 65, 0, 257, 1000, 3])
    ev = t.fill_host()
    _compare_to_bruteforce(ev, t.cfg.n_kernels, t.cfg.n_streams)


def test_closed_form_noise_free_template():
    # template of 6 launches over 3 ids with fixed durations, repeated m times
    tmpl_kid = [0, 1, 0, 2, 1, 0]
    dur = {0: 1000, 1: 4096, 2: 2**31 + 5}
    m = 50
    kid, st, t0, t1 = [], [], [], []
    t = 10**18
    for _ in range(m):
        for k in tmpl_kid:
            kid.append(k)
            st.append(k % 2)
            t0.append(t)
            t1.append(t + dur[k])
            t += 10_000
    ev = _ev(kid, st, t0, t1, [len(kid)])
    out = oracle.summarize(ev, 4, 2)
    mult = {0: 3, 1: 2, 2: 1}
    for k in range(3):
        assert out["count"][k] == m * mult[k]
        assert out["sum_ns"][k] == m * mult[k] * dur[k]
        assert out["min_ns"][k] == dur[k] and out["max_ns"][k] == dur[k]
    # 1000 ns lies in [512, 1024): bin 9; 4096 = 2^12 exactly: bin 12; >= 2^31 saturates to bin 31
    assert out["hist"][0][9] == m * 3 and out["hist"][1][12] == m * 2 and out["hist"][2][31] == m
    assert out["count"][3] == 0
    assert out["busy_ns"][0] == m * (3 * 1000 + 2 * 4096 + 2**31 + 5)
    assert out["stream_busy_ns"][0].tolist() == [m * (3 * 1000 + 2**31 + 5), m * 2 * 4096]
    assert out["t_first"][0] == 10**18
    # the last launch of id 2 (template position 3 of the last repetition) ends last
    assert out["t_last"][0] == 10**18 + (6 * (m - 1) + 3) * 10_000 + 2**31 + 5
    assert out["wire_bytes"][0] == 3 * (33 + 5)


def test_edge_durations_and_big_timestamps():
    base = 2**60 + 12345  # well past 2^53
    ds = [0, 1, 2, 3, 2**20, 2**20 - 1, 2**31 - 1, 2**31, 2**40]
    ev = _ev([0] * len(ds), [0] * len(ds), [base] * len(ds), [base + d for d in ds], [len(ds)])
    out = _compare_to_bruteforce(ev, 1, 1)
    assert out["min_ns"][0] == 0 and out["max_ns"][0] == 2**40
    assert out["hist"][0][0] == 2  # d = 0 and d = 1
    assert out["hist"][0][31] == 2  # 2^31 and 2^40 saturate


def test_invalid_records_touch_nothing():
    # ids out of range, bad stream, end < start, negative start
    kid = [0, 5, -1, 0, 0, 0, 1]
    st = [0, 0, 0, 3, 0, 0, 1]
    t0 = [100, 100, 100, 100, 200, -5, 300]
    t1 = [150, 900, 900, 900, 199, 10, 310]
    ev = _ev(kid, st, t0, t1, [len(kid)])
    out = _compare_to_bruteforce(ev, 2, 2)
    assert out["n_valid"][0] == 2 and out["n_invalid"][0] == 5
    assert out["t_first"][0] == 100 and out["t_last"][0] == 310
    all_bad = _ev([7, 7], [0, 0], [1, 1], [2, 2], [2])
    o2 = _compare_to_bruteforce(all_bad, 2, 1)
    assert o2["step_ns"][0] == 0 and o2["t_first"][0] == bf.I64_MAX


def test_malformed_offsets_become_empty_segments():
    ev = _ev([0] * 10, [0] * 10, list(range(10)), list(range(1, 11)), [10])
    ev["seg_off"] = np.array([0, 6, 4, 12], np.int64)  # decreasing, then past the end
    out = oracle.summarize(ev, 1, 1)
    assert out["bad_segments"] == 2
    assert out["n_valid"].tolist() == [6, 0, 0]


def test_order_independence():
    t = tracegen.make("tiny", n_ranks=1, n_steps=1, events_per_seg=3000, tmpl_len=300, n_stragglers=0, n_pairs=0)
    ev = t.fill_host()
    a = oracle.summarize(ev, 64, 4)
    perm = np.random.default_rng(3).permutation(3000)
    ev2 = dict(ev, **{k: np.ascontiguousarray(ev[k][perm]) for k in ("kernel_id", "stream", "start_ns", "end_ns")})
    b = oracle.summarize(ev2, 64, 4)
    for k in a:
        if isinstance(a[k], np.ndarray):
            assert np.array_equal(a[k], b[k]), k


def _check_invariants(out, ev, K, NS):
    G = len(ev["seg_off"]) - 1
    cnt = out["count"].reshape(G, K).astype(np.int64)
    sm = out["sum_ns"].reshape(G, K)
    mn, mx = out["min_ns"].reshape(G, K), out["max_ns"].reshape(G, K)
    hist = out["hist"].reshape(G, K, NB).astype(np.int64)
    lens = np.diff(ev["seg_off"])
    assert (cnt.sum(1) == out["n_valid"]).all()
    assert (sm.sum(1) == out["busy_ns"]).all()
    assert (out["stream_busy_ns"].sum(1) == out["busy_ns"]).all()
    assert (hist.sum(2) == cnt).all()
    pres = cnt > 0
    xbar = np.where(pres, sm // np.maximum(cnt, 1), 0)
    assert (mn[pres] <= xbar[pres]).all() and (xbar[pres] <= mx[pres]).all()
    bins = np.arange(NB)
    lo = np.array([bf.bin_of(int(v)) if p else 0 for v, p in zip(mn.ravel(), pres.ravel())]).reshape(G, K)
    hi = np.array([bf.bin_of(int(v)) if p else 0 for v, p in zip(mx.ravel(), pres.ravel())]).reshape(G, K)
    outside = (hist > 0) & ((bins[None, None, :] < lo[..., None]) | (bins[None, None, :] > hi[..., None]))
    assert not outside.any()
    assert ((out["n_valid"].astype(np.int64) + out["n_invalid"]) == lens).all()
    ne = out["n_valid"] > 0
    assert (out["t_first"][ne] <= out["t_last"][ne]).all()
    nnz = (hist > 0).sum(2)
    assert (out["wire_bytes"] == np.where(pres, 33 + 5 * nnz, 0).sum(1)).all()


@pytest.mark.parametrize("name,over", [
    ("tiny", {}),
    ("medium", dict(n_ranks=8, n_steps=4, invalid_ppm=100)),
    ("skew", dict(n_ranks=4, n_steps=2, events_per_seg=40_000)),
    ("cluster", dict(n_ranks=4, events_per_seg=80_000, n_stragglers=1, n_pairs=2)),
])
def test_invariants_generated(name, over):
    t = tracegen.make(name, **over)
    ev = t.fill_host()
    out = oracle.summarize(ev, t.cfg.n_kernels, t.cfg.n_streams)
    _check_invariants(out, ev, t.cfg.n_kernels, t.cfg.n_streams)


def test_compression_ratio_arithmetic():
    # The paper's kernel-trace figures: 10 MB raw to 2.7 KB of summaries per
    # rank per step, quoted as about 3,700x (section 8.3, Table "data-volume").
    assert round(10e6 / 2.7e3) == 3704
    # Ours: raw bytes (24 per event) over uploaded record bytes.
    t = tracegen.make("tiny")
    ev = t.fill_host()
    out = oracle.summarize(ev, 64, 4)
    ratio = 24 * np.diff(ev["seg_off"]) / out["wire_bytes"]
    assert (ratio > 100).all()
