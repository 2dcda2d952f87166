"""GPU parity: libargus (through its C ABI) against the CPU oracle.

Integers, order statistics and flags must match bit for bit; float32 z,
means and ratios within 1e-5 relative. Inputs are seeded: the GPU side
fills events on the device, the oracle side on the host, from the same
generator (checked by per-segment checksums).
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2606_20374_amd as pa
import tracegen
from tests import parity as P

pytestmark = pytest.mark.gpu
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
DEV = "cuda"


def _announce(name):
    print(f"\n[gpu-case] {name}", flush=True)


def _dev_events(ev):
    return {k: torch.from_numpy(np.ascontiguousarray(v)).to(DEV) for k, v in ev.items()}


def _summarize_both(ev_h, R, S, K, NS):
    g = pa.summarize(_dev_events(ev_h), R, S, K, NS)
    torch.cuda.synchronize()
    o = oracle.summarize(ev_h, K, NS, n_events=len(ev_h["kernel_id"]))
    return g, o


def _full_step_parity(trace, what):
    cfg = trace.cfg
    R, S, K, NS = cfg.n_ranks, cfg.n_steps, cfg.n_kernels, cfg.n_streams
    ev_d = trace.fill_device(device=DEV)
    assert np.array_equal(trace.checksum_device(ev_d), trace.checksum_host(trace.fill_host()))
    s, x, w = pa.run_step(ev_d, R, S, K, NS)
    torch.cuda.synchronize()
    so = oracle.summarize(trace.fill_host(), K, NS)
    P.assert_int_equal(s, so, P.SUM_INT_FIELDS, what)
    xo = oracle.cross_rank(so["count"], so["sum_ns"], R, S, K)
    P.assert_int_equal(x, xo, P.XR_INT_FIELDS, what)
    P.assert_float_close(x, xo, P.XR_FLOAT_FIELDS, what)
    wo = oracle.iter_windows(so["step_ns"], R, S)
    P.assert_int_equal(w, wo, P.L1_INT_FIELDS, what)
    P.assert_float_close(w, wo, ["cp_ratio"], what)
    assert int(s["dev_status"].item()) == 0
    return s, x, w


def test_device_generator_matches_host():
    _announce("tracegen device == host")
    t = tracegen.make("tiny", invalid_ppm=2000)
    ev_d = t.fill_device(device=DEV)
    ev_h = t.fill_host()
    for k in ("kernel_id", "stream", "start_ns", "end_ns"):
        assert np.array_equal(ev_d[k].cpu().numpy(), ev_h[k]), k
    m = tracegen.make("medium", n_ranks=16)
    assert np.array_equal(m.checksum_device(m.fill_device(device=DEV)), m.checksum_host(m.fill_host()))


def test_tiny_full_step():
    _announce("tiny full step")
    t = tracegen.make("tiny")
    _, x, _ = _full_step_parity(t, "tiny")
    strag = set(np.nonzero(x["straggler"].cpu().numpy().reshape(8, 4)[:, 0])[0].tolist())
    assert strag == t.truth()["stragglers"]


def test_medium_reduced_full_step():
    _announce("medium R=32 full step")
    t = tracegen.make("medium", n_ranks=32)
    _full_step_parity(t, "medium32")


def test_ragged_corrupt_segments():
    _announce("ragged + corrupt segments")
    rng = np.random.default_rng(7)
    lens = rng.integers(0, 3000, size=6 * 5)
    lens[[0, 7, 13]] = 0
    lens[[3, 9]] = [1, 4097]
    cfg = tracegen.config("tiny", n_ranks=6, n_steps=5, tmpl_len=300, invalid_ppm=40_000)
    t = tracegen.Trace(cfg, seg_lengths=lens)
    g, o = _summarize_both(t.fill_host(), 6, 5, cfg.n_kernels, cfg.n_streams)
    P.assert_int_equal(g, o, P.SUM_INT_FIELDS, "ragged")


def test_unaligned_event_arrays():
    _announce("summarize with event arrays off 16-byte alignment")
    t = tracegen.make("tiny", invalid_ppm=3000)
    c = t.cfg
    ev = t.fill_host()
    d = {}
    for k, v in ev.items():
        h = torch.from_numpy(np.ascontiguousarray(v))
        if k == "seg_off":
            d[k] = h.to(DEV)
            continue
        buf = torch.empty(h.numel() + 1, dtype=h.dtype, device=DEV)
        d[k] = buf[1:]
        d[k].copy_(h.to(DEV))
        assert d[k].data_ptr() % 16 != 0
    g = pa.summarize(d, c.n_ranks, c.n_steps, c.n_kernels, c.n_streams)
    torch.cuda.synchronize()
    o = oracle.summarize(ev, c.n_kernels, c.n_streams)
    P.assert_int_equal(g, o, P.SUM_INT_FIELDS, "unaligned")
    assert int(g["dev_status"].item()) == 0


def test_hand_built_edge_events():
    _announce("hand-built edge events")
    base = 2**60 + 7
    ds = [0, 1, 2, 3, 2**20, 2**20 - 1, 2**31 - 1, 2**31, 2**40, 2**62]
    kid = [0] * len(ds) + [1, 2, -1, 5, 0, 1]
    st = [0] * len(ds) + [1, 0, 0, 0, 2, 1]
    t0 = [base] * len(ds) + [10, 20, 30, 40, 50, -3]
    t1 = [base + d for d in ds] + [15, 19, 40, 50, 60, 4]
    # segments: [all edge durations], [mixed invalid], [empty], [only invalid]
    lens = [len(ds), 6, 0, 0]
    kid += [9, 9]
    st += [0, 0]
    t0 += [1, 1]
    t1 += [2, 2]
    lens[3] = 2
    off = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    ev = {"kernel_id": np.array(kid, np.int32), "stream": np.array(st, np.int32),
          "start_ns": np.array(t0, np.int64), "end_ns": np.array(t1, np.int64), "seg_off": off}
    g, o = _summarize_both(ev, 2, 2, 3, 2)
    P.assert_int_equal(g, o, P.SUM_INT_FIELDS, "edge")


def test_malformed_segments_raise_device_status():
    _announce("malformed seg_off")
    ev = {"kernel_id": np.zeros(10, np.int32), "stream": np.zeros(10, np.int32),
          "start_ns": np.arange(10, dtype=np.int64), "end_ns": np.arange(1, 11, dtype=np.int64),
          "seg_off": np.array([0, 6, 4, 12], np.int64)}
    g, o = _summarize_both(ev, 3, 1, 1, 1)
    assert o["bad_segments"] == 2
    P.assert_int_equal(g, o, P.SUM_INT_FIELDS, "malformed")
    assert int(g["dev_status"].item()) == pa.argus.DEV_BAD_SEGMENT


def test_large_kernel_id_space_multi_range():
    _announce("K=8200 id ranges")
    t = tracegen.make("skew", n_ranks=6, n_steps=2, events_per_seg=30_000)
    g, o = _summarize_both(t.fill_host(), 6, 2, t.cfg.n_kernels, t.cfg.n_streams)
    P.assert_int_equal(g, o, P.SUM_INT_FIELDS, "skew-small")


def test_full_histogram_pool_exhaustion():
    _announce("pool exhaustion: many wide kernels")
    # 300 kernel ids, each with durations spread over ~24 octaves: every id
    # needs a full histogram record, far more than one pass holds
    rng = np.random.default_rng(3)
    n = 60_000
    kid = rng.integers(0, 300, size=n).astype(np.int32)
    d = (2 ** rng.uniform(0, 34, size=n)).astype(np.int64)
    t0 = rng.integers(0, 2**50, size=n).astype(np.int64)
    ev = {"kernel_id": kid, "stream": (kid % 3).astype(np.int32), "start_ns": t0, "end_ns": t0 + d,
          "seg_off": np.array([0, n // 2, n], np.int64)}
    g, o = _summarize_both(ev, 1, 2, 300, 3)
    P.assert_int_equal(g, o, P.SUM_INT_FIELDS, "pool")


def _random_events(n, K, NS, seed, spread_octaves=3, seg_lengths=None, wide_ids=()):
    rng = np.random.default_rng(seed)
    kid = rng.integers(0, K, size=n).astype(np.int32)
    base = rng.integers(1000, 10**6, size=K)
    d = (base[kid] * 2.0 ** rng.uniform(0, spread_octaves, size=n)).astype(np.int64)
    wide = np.isin(kid, np.asarray(wide_ids, dtype=np.int64))
    d[wide] = (2 ** rng.uniform(0, 34, size=int(wide.sum()))).astype(np.int64)
    t0 = rng.integers(0, 2**50, size=n).astype(np.int64)
    lens = [n] if seg_lengths is None else seg_lengths
    return {"kernel_id": kid, "stream": (kid % NS).astype(np.int32), "start_ns": t0, "end_ns": t0 + d,
            "seg_off": np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)}


def test_mapped_slot_overflow():
    _announce("mapped ids: more distinct ids in a segment than LDS slots")
    K = 6000
    ev = _random_events(60_000, K, 16, seed=21, seg_lengths=[30_000, 25_000, 5_000])
    g, o = _summarize_both(ev, 3, 1, K, 16)
    P.assert_int_equal(g, o, P.SUM_INT_FIELDS, "mapped-overflow")


def test_mapped_several_id_ranges():
    _announce("mapped ids: id space of 40,000 (several ranges)")
    K = 40_000
    ev = _random_events(50_000, K, 8, seed=22, seg_lengths=[20_000, 0, 30_000, 0])
    g, o = _summarize_both(ev, 2, 2, K, 8)
    P.assert_int_equal(g, o, P.SUM_INT_FIELDS, "mapped-ranges")


def test_mapped_pool_exhaustion():
    _announce("mapped ids: wide kernels exhaust the histogram pool")
    K = 3000
    ev = _random_events(80_000, K, 4, seed=23, seg_lengths=[40_000, 40_000], wide_ids=range(0, 3000, 15))
    g, o = _summarize_both(ev, 2, 1, K, 4)
    P.assert_int_equal(g, o, P.SUM_INT_FIELDS, "mapped-pool")


def test_single_kernel_and_stream():
    _announce("K=1 NS=1")
    t = tracegen.make("tiny", n_kernels=1, n_streams=1, n_stragglers=0, n_pairs=0)
    g, o = _summarize_both(t.fill_host(), 8, 4, 1, 1)
    P.assert_int_equal(g, o, P.SUM_INT_FIELDS, "K1")


def test_determinism():
    _announce("determinism")
    t = tracegen.make("medium", n_ranks=8)
    ev = t.fill_device(device=DEV)
    cfg = t.cfg
    a = pa.run_step(ev, cfg.n_ranks, cfg.n_steps, cfg.n_kernels, cfg.n_streams)
    b = pa.run_step(ev, cfg.n_ranks, cfg.n_steps, cfg.n_kernels, cfg.n_streams)
    torch.cuda.synchronize()
    pres = a[0]["count"] != 0
    for da, db in zip(a, b):
        for k in da:
            if k.startswith("_"):
                continue
            if da is a[0] and k in P.PRESENT_ONLY:  # written for present cells only
                per = da[k].numel() // pres.numel()
                keep = pres.repeat_interleave(per)
                assert torch.equal(da[k][keep], db[k][keep]), k
            else:
                assert torch.equal(da[k], db[k]), k


# ------------------------------------------------------------- cross-rank
def _xr_both(cnt, sm, R, S, K, **p):
    g = pa.cross_rank(torch.from_numpy(cnt.view(np.int32)).to(DEV), torch.from_numpy(sm).to(DEV), R, S, K, **p)
    torch.cuda.synchronize()
    o = oracle.cross_rank(cnt, sm, R, S, K, **p)
    P.assert_int_equal(g, o, P.XR_INT_FIELDS, "xr")
    P.assert_float_close(g, o, P.XR_FLOAT_FIELDS, "xr")
    return g, o


def _from_x(x, count=10):
    x = np.asarray(x, dtype=np.int64)
    cnt = np.where(x >= 0, count, 0).astype(np.uint32).reshape(-1)
    return cnt, np.where(x >= 0, x * count, 0).astype(np.int64).reshape(-1)


def test_cross_rank_golden_and_boundaries():
    _announce("cross-rank golden + boundaries")
    for c in json.load(open(os.path.join(GOLDEN, "order_stats.json")))["cases"]:
        cnt, sm = _from_x(c["x"])
        g, _ = _xr_both(cnt, sm, len(c["x"]), 1, 1)
        assert (g["med_ns"].item(), g["q1_ns"].item(), g["q3_ns"].item(), g["mad_ns"].item()) == \
            (c["med"], c["q1"], c["q3"], c["mad"])
    for X in (124, 125, 132, 133, 156, 157):
        cnt, sm = _from_x([90, 95, 100, 105, 110, 115, X], count=8)
        _xr_both(cnt, sm, 7, 1, 1)
    cnt, sm = _from_x([[100], [-1], [300], [-1]])
    _xr_both(cnt, sm, 4, 1, 1)


def test_cross_rank_random_with_absent_cells():
    _announce("cross-rank random")
    rng = np.random.default_rng(12)
    for R, S, K in [(37, 3, 9), (3000, 1, 40), (16384, 1, 3), (5, 2, 3000), (64, 1, 16384)]:
        x = rng.integers(0, 2**40, size=(R, S, K)) >> rng.integers(0, 40, size=(R, S, K))
        cnt = rng.integers(1, 50, size=(R, S, K)).astype(np.uint32)
        cnt[rng.random((R, S, K)) < 0.3] = 0
        sm = (x * cnt).astype(np.int64)
        _xr_both(cnt.reshape(-1), sm.reshape(-1), R, S, K)


def test_cross_rank_identical_and_huge_values():
    _announce("cross-rank identical / huge")
    R, K = 16, 12
    cnt, sm = _from_x(np.tile(np.arange(1, K + 1) * 1000, (R, 1)))
    g, _ = _xr_both(cnt, sm, R, 1, K)
    assert (g["score_pm"].cpu().numpy() == 1000).all()
    # sums near the top of the int64 range, and wrapped sums
    cnt = np.full(R * 2, 3, np.uint32)
    sm = np.full(R * 2, 2**63 - 5, np.int64)
    sm[::5] = -7
    cnt[::7] = 1  # (2^64 - 7) / 1 saturates at INT64_MAX
    _xr_both(cnt, sm, R, 1, 2)


def test_cross_rank_quotient_paths():
    # the exact mean floor(sum / count) takes a double quotient below 2^53 and
    # the integer division above; permille ratios likewise below 2^53 / 1000
    _announce("cross-rank quotient paths")
    rng = np.random.default_rng(5)
    R, K = 48, 6
    cnt = rng.integers(1, 2**32, size=(R, K), dtype=np.uint64)
    cnt[:, 0] = 1 << 20
    cnt[:, 1] = 3
    q = (np.uint64(2**53) - np.uint64(1)) // cnt  # largest quotient with sum < 2^53
    sm = q * cnt + (cnt - np.uint64(1)) * (rng.random((R, K)) < 0.5)
    sm[::4, 2] = np.uint64(2**53)  # exactly 2^53: the integer path
    sm[1::4, 3] = np.uint64(2**53) - np.uint64(1)
    # means around 9e12: 1000 x on both sides of 2^53 (about 9.007e15)
    cnt[:, 4] = rng.integers(1, 1000, R).astype(np.uint64)
    sm[:, 4] = rng.integers(8 * 10**12, 10**13, R).astype(np.uint64) * cnt[:, 4]
    _xr_both(cnt.reshape(-1).astype(np.uint32), sm.reshape(-1).astype(np.int64), R, 1, K)


# ------------------------------------------------------------------- L1
def test_l1_golden_and_random():
    _announce("L1 golden + random")
    for c in json.load(open(os.path.join(GOLDEN, "l1_series.json")))["cases"]:
        y = np.array(c["y"], np.int64)
        g = pa.iter_windows(torch.from_numpy(y).to(DEV), 1, len(y))
        torch.cuda.synchronize()
        assert g["flags"].cpu().numpy().tolist() == c["flags"], c["name"]
        assert (g["cls"].item(), g["eff_width"].item(), g["cp"].item()) == (c["cls"], c["eff_width"], c["cp"])
    rng = np.random.default_rng(9)
    for R, S in [(200, 12), (64, 100), (17, 1000), (5, 4096), (3, 1), (3, 0)]:
        y = (10**6 * (1 + 0.05 * rng.standard_normal((R, S)))).astype(np.int64)
        if S > 3:
            y[::3, S // 2:] = y[::3, S // 2:] * 3 // 2
            y[1::4, S // 3] *= 3
        if R > 2 and S > 0:
            y[2, 0] = -1
        for p in (dict(), dict(W=3, min_seg=1, cmax_pm=150)):
            g = pa.iter_windows(torch.from_numpy(y.reshape(-1)).to(DEV), R, S, **p)
            torch.cuda.synchronize()
            o = oracle.iter_windows(y.reshape(-1), R, S, **p)
            if R * S == 0:
                g = {k: v[:max(R, 0)] if k != "flags" else v[:0] for k, v in g.items()}
            P.assert_int_equal(g, o, P.L1_INT_FIELDS, f"l1 {R}x{S}")
            P.assert_float_close(g, o, ["cp_ratio"], f"l1 {R}x{S}")


@pytest.mark.parametrize("K,keyed", [(64, False), (2048, False), (6000, False), (40_000, False), (300, True)])
def test_absent_cells_keep_their_buffers(K, keyed):
    """Only the count of an absent cell is written: its sum, min, max and
    histogram keep what the caller's buffers held (a sentinel here), while
    every present cell matches the oracle. Dense (K <= 2048), mapped
    (larger K, one and several id ranges) and (kernel, stream) keys; half of
    the ids never occur."""
    _announce(f"absent cells untouched: K={K} keyed={keyed}")
    NS = 4
    ev = _random_events(40_000, K // 2, NS, seed=31 + K, seg_lengths=[25_000, 0, 15_000])
    ev["stream"] = np.random.default_rng(K).integers(0, NS, size=40_000).astype(np.int32)
    cells = 3 * K * (NS if keyed else 1)
    out = pa.argus.alloc_summary(3, 1, K * (NS if keyed else 1), NS, DEV)
    sentinel = {"sum_ns": 0x5A5A5A5A5A5A5A5A, "min_ns": 0x1234567812345678, "max_ns": -0x0F0F0F0F0F0F0F0F,
                "hist": 0x3C3C3C3C}
    for f, v in sentinel.items():
        out[f].fill_(v)
    g = pa.summarize(_dev_events(ev), 3, 1, K, NS, out=out, keyed=keyed)
    torch.cuda.synchronize()
    o = oracle.summarize(ev, K, NS, keyed=keyed)
    P.assert_int_equal(g, o, P.SUM_INT_FIELDS, f"absent K={K} keyed={keyed}")
    absent = np.asarray(o["count"]).reshape(-1) == 0
    assert absent.sum() >= cells // 3, "the case needs absent cells"
    for f, v in sentinel.items():
        per = P.NB if f == "hist" else 1
        got = P.to_np(g[f]).reshape(cells, per)[absent]
        assert (got == v).all(), (f, "an absent cell's field was written")
