"""GPU parity of argus_kde (section 5.2, Eq. 1) through the C ABI against
the CPU oracle: cluster counts, per-cluster counts, p50, p99 and the
quantised bandwidth must match exactly in every cell.

Cases: the seeded tiny and medium traces (multimodal kernels), parameter
variants, ragged / corrupted / malformed segments, hand-built groups that
exercise every filter rule and both LDS paths (cells whose grid, kernel or
valley list do not fit the fast path are finished by the large-LDS path),
summaries that do not match the events, segments of 4-byte and 8-byte
bucket records in one call, a rank-step longer than 2^26 events (the
scatter's global-load path), the stream array skipped or read, and full-size
workloads (sampled segments checked against the oracle).
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


def _announce(name):
    print(f"\n[gpu-case] {name}", flush=True)


def _dev(ev):
    return {k: torch.from_numpy(np.ascontiguousarray(v)).to(DEV) for k, v in ev.items()}


def _kde_gpu(ev_d, R, S, K, NS, **params):
    s = pa.summarize(ev_d, R, S, K, NS)
    k = pa.kde(ev_d, s, R, S, K, NS, **params)
    torch.cuda.synchronize()
    return s, k


def _both(ev_h, R, S, K, NS, what, **params):
    s, k = _kde_gpu(_dev(ev_h), R, S, K, NS, **params)
    o = oracle.kde(ev_h, K, NS, n_events=len(ev_h["kernel_id"]), **params)
    P.assert_kde_equal(k, o, what)
    assert int(k["dev_status"].item()) == 0, what
    return k, o


def test_kde_tiny_trace():
    _announce("kde tiny trace")
    t = tracegen.make("tiny")
    c = t.cfg
    k, o = _both(t.fill_host(), c.n_ranks, c.n_steps, c.n_kernels, c.n_streams, "tiny")
    assert (o["n_clusters"] > 1).sum() > 100  # multimodal kernels are present


@pytest.mark.parametrize("params", [dict(sub_bits=1), dict(sub_bits=3), dict(sub_bits=5, gap=24),
                                    dict(frac_pm=0, min_count=1, gap=0), dict(frac_pm=200, min_count=10, gap=100)])
def test_kde_parameters(params):
    _announce(f"kde tiny {params}")
    t = tracegen.make("tiny")
    c = t.cfg
    _both(t.fill_host(), c.n_ranks, c.n_steps, c.n_kernels, c.n_streams, f"tiny {params}", **params)


def test_kde_medium_trace():
    _announce("kde medium trace (256 x 8 x 100k)")
    t = tracegen.make("medium")
    c = t.cfg
    R, S, K, NS = c.n_ranks, c.n_steps, c.n_kernels, c.n_streams
    _, k = _kde_gpu(t.fill_device(device=DEV), R, S, K, NS)
    assert int(k["dev_status"].item()) == 0
    o = P.oracle_kde_segments(t, range(c.n_segments))
    P.assert_kde_equal(k, o, "medium")


def test_kde_ragged_corrupt_and_malformed():
    _announce("kde ragged + corrupt + malformed")
    rng = np.random.default_rng(7)
    lens = rng.integers(0, 30_000, size=32)
    lens[[3, 17]] = 0
    t = tracegen.make("tiny", invalid_ppm=3000, seg_lengths=lens)
    c = t.cfg
    ev = t.fill_host()
    _both(ev, c.n_ranks, c.n_steps, c.n_kernels, c.n_streams, "ragged corrupt")
    # a malformed segment is summarized as empty and clusters as empty
    off = ev["seg_off"].copy()
    off[10] = off[11] + 5
    ev2 = dict(ev, seg_off=off)
    s, k = _kde_gpu(_dev(ev2), c.n_ranks, c.n_steps, c.n_kernels, c.n_streams)
    assert int(s["dev_status"].item()) & pa.argus.DEV_BAD_SEGMENT
    o = oracle.kde(ev2, c.n_kernels, c.n_streams, n_events=len(ev2["kernel_id"]))
    P.assert_kde_equal(k, o, "malformed")
    assert int(k["dev_status"].item()) == 0


def test_kde_stream_array_skipped_only_for_valid_segments():
    """Segments whose summary counts no invalid event are scattered without
    reading the stream array; the clusters equal those of the full read (no
    n_invalid passed) and the oracle's, with invalid events (bad streams
    among them) in the other segments of the same call."""
    _announce("kde stream array skipped for all-valid segments")
    lens = np.array([0, 5, 40, 3000, 20_000, 7, 1, 12_345] * 4)
    t = tracegen.make("tiny", invalid_ppm=300, seg_lengths=lens)
    c = t.cfg
    ev = t.fill_host()
    R, S, K, NS = c.n_ranks, c.n_steps, c.n_kernels, c.n_streams
    ev_d = _dev(ev)
    s = pa.summarize(ev_d, R, S, K, NS)
    n_inv = s["n_invalid"].cpu().numpy()
    assert (n_inv == 0).sum() >= 8 and (n_inv > 0).sum() >= 4, n_inv
    k_skip = pa.kde(ev_d, s, R, S, K, NS)
    k_full = pa.kde(ev_d, {f: v for f, v in s.items() if f != "n_invalid"}, R, S, K, NS)
    torch.cuda.synchronize()
    for f in ("n_clusters", "count", "p50_ns", "p99_ns", "bw_q8", "dev_status"):
        assert torch.equal(k_skip[f], k_full[f]), f
    o = oracle.kde(ev, K, NS, n_events=len(ev["kernel_id"]))
    P.assert_kde_equal(k_skip, o, "stream skip")
    assert int(k_skip["dev_status"].item()) == 0


def _groups_to_events(groups, K, NS, seed=0):
    """One segment; groups: list of duration arrays, group i -> kernel id i."""
    rng = np.random.default_rng(seed)
    kid = np.concatenate([np.full(len(d), i, np.int32) for i, d in enumerate(groups)])
    dur = np.concatenate([np.asarray(d, np.uint64) for d in groups])
    perm = rng.permutation(len(kid))
    kid, dur = kid[perm], dur[perm]
    start = rng.integers(0, 1 << 30, size=len(kid)).astype(np.int64)
    # keep end = start + d within int64 for the largest durations
    start = np.where(dur > (1 << 62), 0, start).astype(np.int64)
    end = (start.astype(np.uint64) + dur).astype(np.int64)
    return {"kernel_id": kid, "stream": (kid % NS).astype(np.int32), "start_ns": start, "end_ns": end,
            "seg_off": np.array([0, len(kid)], np.int64)}


def _lb(b):
    e, t = divmod(b, 64)
    th = int(oracle.kde_thresholds()[t])
    return th << (e - 23) if e >= 23 else -(-th >> (23 - e))


def _spikes(*pairs):
    return np.concatenate([np.full(n, d, np.uint64) for d, n in pairs])


def test_kde_hand_built_groups():
    _announce("kde hand-built groups (every filter rule, both LDS paths)")
    rng = np.random.default_rng(11)
    b0 = 64 * 12
    groups = [
        np.array([12345], np.uint64),
        np.full(50, 777, np.uint64),
        np.array([0, 1, 1, 0], np.uint64),
        _spikes((10_000, 1000), (1_000_000, 500)),
        _spikes((_lb(64 * 25), 2000), (_lb(64 * 25 + 96), 2000)),
        _spikes((_lb(64 * 25), 2000), (_lb(64 * 25 + 95), 2000)),
        _spikes((2**14, 1000), (2**19, 52)),
        _spikes((2**14, 1000), (2**19, 53)),
        _spikes((2**10, 3), (2**20, 3)),
        _spikes((2**10, 3), (2**20, 2)),
        _spikes(*[(2 ** (5 + 10 * i), 400_000) for i in range(6)]),  # cluster cap, grid 3201 points
        _spikes((2**20, 1_000_000), (_lb(64 * 20 + 200), 1_000_000)),  # zero plateau
        _spikes((_lb(64 * 20), 20), (_lb(64 * 20 + 50), 2), (_lb(64 * 20 + 100), 20)),
        _spikes(*[(_lb(b0 + o), c) for o, c in zip([0, 400, 500, 600, 1000],
                                                   [250_000, 500_000, 75_000, 250_000, 250_000])]),
        _spikes((_lb(b0), 100_000), (_lb(b0 + 300), 4000), (_lb(b0 + 600), 100_000)),
        _spikes((_lb(b0), 4000), (_lb(b0 + 300), 4000), (_lb(b0 + 600), 100_000)),
        # large-LDS path: 3,900-point grid whose kernel spans the grid
        _spikes((2, 3), (2**61 + 12345, 4)),
        # extremes of the duration range
        _spikes((2**63 - 1, 5), (2**62, 5), (3, 7)),
    ]
    for n in (2, 5, 20, 100, 256, 257, 1000, 2047, 2048, 2049, 20000):
        groups.append(np.exp(rng.normal(np.log(80_000), 0.1, n)).astype(np.uint64))
    for sizes in [(500, 200, 50), (60, 60, 60), (1000, 2000), (300, 400, 4000, 400)]:
        comps = [np.exp(np.log(30_000 * 4**i) + 0.1 * np.clip(rng.normal(0, 1, m), -4, 4)).astype(np.uint64)
                 for i, m in enumerate(sizes)]
        groups.append(np.concatenate(comps))
    # lane-pass cells whose target bins are wider than 2^32 ns (64-bit lists)
    # and just narrower (32-bit offsets close to 2^32), one bimodal
    for centre in (1e12, 3e11):
        groups.append(np.exp(rng.normal(np.log(centre), 0.05, 100)).astype(np.uint64))
    groups.append(np.concatenate([np.exp(rng.normal(np.log(c), 0.02, 60)).astype(np.uint64) for c in (1e12, 2e12)]))
    K = len(groups) + 3  # a few empty kernel ids
    ev = _groups_to_events(groups, K, 4)
    k, o = _both(ev, 1, 1, K, 4, "hand-built")
    # spot checks that the oracle pins carry over (cap, plateau, spacing)
    assert list(o["count"][10]) == [400_000, 400_000, 400_000, 1_200_000]
    assert o["n_clusters"][4] == 2 and o["n_clusters"][5] == 1
    assert o["n_clusters"][K - 1] == 0


def test_kde_summary_mismatch_is_reported():
    _announce("kde summary mismatch")
    t = tracegen.make("tiny")
    c = t.cfg
    R, S, K, NS = c.n_ranks, c.n_steps, c.n_kernels, c.n_streams
    ev_h = t.fill_host()
    ev_d = _dev(ev_h)
    s = pa.summarize(ev_d, R, S, K, NS)
    o = oracle.kde(ev_h, K, NS)
    # one cell claims an extra event; another's minimum is too large
    c1, c2 = 5 * K + 7, 9 * K + 3
    s["count"][c1] += 1
    s["min_ns"][c2] = s["max_ns"][c2]
    k = pa.kde(ev_d, s, R, S, K, NS)
    torch.cuda.synchronize()
    assert int(k["dev_status"].item()) == pa.argus.DEV_KDE_SUMMARY
    nc = k["n_clusters"].cpu().numpy()
    # the extra count shifts the later buckets of segment 5 by one: kernel 8
    # starts one past kernel 7's end and kernel 63 ends past the segment
    bad = [c1, c1 + 1, 5 * K + 63, c2]
    assert (nc[bad] == 0).all()
    keep = np.setdiff1d(np.arange(len(nc)), bad)
    P.assert_kde_equal(k, {f: np.asarray(o[f])[keep] for f in P.KDE_FIELDS}, "mismatch", rows=keep)


def _dev_unaligned(ev):
    """Device copies whose event arrays start 4 or 8 bytes past a 16-byte
    boundary: the kernels must take their element-wise load paths."""
    out = {}
    for k, v in ev.items():
        t = torch.from_numpy(np.ascontiguousarray(v))
        if k == "seg_off":
            out[k] = t.to(DEV)
            continue
        buf = torch.empty(t.numel() + 1, dtype=t.dtype, device=DEV)
        out[k] = buf[1:]
        out[k].copy_(t.to(DEV))
        assert out[k].data_ptr() % 16 != 0
    return out


def test_kde_unaligned_event_arrays():
    _announce("kde with event arrays off 16-byte alignment (tiny trace, cells of 40 to 6,000 durations)")
    t = tracegen.make("tiny")
    c = t.cfg
    ev = t.fill_host()
    _, k = _kde_gpu(_dev_unaligned(ev), c.n_ranks, c.n_steps, c.n_kernels, c.n_streams)
    P.assert_kde_equal(k, oracle.kde(ev, c.n_kernels, c.n_streams), "tiny unaligned")
    assert int(k["dev_status"].item()) == 0
    rng = np.random.default_rng(12)
    groups = [np.exp(rng.normal(np.log(30_000 * 3**i), 0.15, n)).astype(np.uint64)
              for i, n in enumerate((6000, 40, 700, 2500, 9, 3000))]
    ev = _groups_to_events(groups, len(groups), 3)
    _, k = _kde_gpu(_dev_unaligned(ev), 1, 1, len(groups), 3)
    P.assert_kde_equal(k, oracle.kde(ev, len(groups), 3), "groups unaligned")
    assert int(k["dev_status"].item()) == 0


def test_kde_summary_mismatch_in_large_cells():
    _announce("kde summary mismatch in cells of 3,000 and 50,000 durations")
    rng = np.random.default_rng(5)
    groups = [np.exp(rng.normal(np.log(50_000), 0.2, n)).astype(np.uint64) for n in (3000, 300, 50_000, 3000)]
    K = len(groups)
    ev = _groups_to_events(groups, K, 2)
    ev_d = _dev(ev)
    s = pa.summarize(ev_d, 1, 1, K, 2)
    o = oracle.kde(ev, K, 2)
    s["min_ns"][0] = s["max_ns"][0]  # durations below the summarized minimum
    s["max_ns"][2] = s["min_ns"][2]  # and above the maximum
    k = pa.kde(ev_d, s, 1, 1, K, 2)
    torch.cuda.synchronize()
    assert int(k["dev_status"].item()) == pa.argus.DEV_KDE_SUMMARY
    nc = k["n_clusters"].cpu().numpy()
    assert nc[0] == 0 and nc[2] == 0
    keep = np.array([1, 3])
    P.assert_kde_equal(k, {f: np.asarray(o[f])[keep] for f in P.KDE_FIELDS}, "large mismatch", rows=keep)


def _segments_to_events(segs, K, NS, seed=0):
    """Several segments in order; segs[g] is a list of duration arrays, array i
    of a segment -> kernel id i."""
    parts = [_groups_to_events(groups, K, NS, seed + g) for g, groups in enumerate(segs)]
    ev = {f: np.concatenate([q[f] for q in parts]) for f in ("kernel_id", "stream", "start_ns", "end_ns")}
    ev["seg_off"] = np.concatenate([[0], np.cumsum([len(q["kernel_id"]) for q in parts])]).astype(np.int64)
    return ev


def _record_widths(k, n_events, n_seg, cells):
    """Per-segment record width flags from the workspace (its layout, each part
    256-byte aligned: 256 B of counters, 8 B per event, 3 x 4 B and 2 B per
    cell, 8 KiB of class counters, then one byte per segment)."""
    al = lambda n: (n + 255) // 256 * 256  # noqa: E731
    off = 256 + al(8 * n_events) + 3 * al(4 * cells) + al(2 * cells) + al(8192)
    return k["_workspace"][off:off + n_seg].cpu().numpy()


def test_kde_record_widths_mixed():
    _announce("kde segments of 4-byte and 8-byte duration records in one call")
    rng = np.random.default_rng(21)

    def cells(top):
        # cells for every tier (60 to 40,000 durations); the last one's largest
        # duration is top
        gs = [np.exp(rng.normal(np.log(c), 0.2, n)).astype(np.uint64)
              for c, n in ((3e4, 60), (9e4, 250), (2e5, 1500), (5e5, 6000), (1e6, 40_000))]
        body = np.minimum(np.exp(rng.normal(np.log(1e9), 0.4, 500)), top - 1).astype(np.uint64)
        gs.append(np.concatenate([body, np.array([top], np.uint64)]))
        return gs

    # 4-byte records need every present maximum below 2^31
    tops = [2**31 - 1, 2**31, 2**31 - 1, 5 * 10**9, 2**31 - 1, 2**32]
    R, S, K, NS = 3, 2, 8, 3
    ev = _segments_to_events([cells(t) for t in tops], K, NS)
    n = len(ev["kernel_id"])
    k, o = _both(ev, R, S, K, NS, "mixed widths")
    assert list(_record_widths(k, n, R * S, R * S * K)) == [1, 0, 1, 0, 1, 0]
    assert (o["n_clusters"][np.arange(R * S) * K + 5] >= 1).all()

    # summaries that understate a maximum: segment 5 now looks 4-byte, its
    # durations from 2^31 up (the largest, 2^32, saturated) lie above the
    # stated maximum's octave, and only that cell is reported
    ev_d = _dev(ev)
    s = pa.summarize(ev_d, R, S, K, NS)
    bad = 5 * K + 5
    s["max_ns"][bad] = 2**31 - 1
    k2 = pa.kde(ev_d, s, R, S, K, NS)
    torch.cuda.synchronize()
    assert int(k2["dev_status"].item()) == pa.argus.DEV_KDE_SUMMARY
    assert list(_record_widths(k2, n, R * S, R * S * K)) == [1, 0, 1, 0, 1, 1]
    assert int(k2["n_clusters"][bad].item()) == 0
    keep = np.setdiff1d(np.arange(R * S * K), [bad])
    P.assert_kde_equal(k2, {f: np.asarray(o[f])[keep] for f in P.KDE_FIELDS}, "understated maximum", rows=keep)


def test_kde_long_segment_global_path():
    """A rank-step of more than 2^26 events is scattered with global loads and
    8-byte records (the buffer path covers shorter ones); with the stream
    array skipped (its summary counts no invalid event) and read (no
    n_invalid passed) its clusters equal the oracle's."""
    _announce("kde long rank-step (2^26 + 4093 events): global-load scatter path")
    lens = np.array([2**26 + 4093] + [3000] * 31)
    t = tracegen.make("tiny", seg_lengths=lens)
    c = t.cfg
    R, S, K, NS = c.n_ranks, c.n_steps, c.n_kernels, c.n_streams
    n = int(lens.sum())
    ev_d = t.fill_device(device=DEV)
    s = pa.summarize(ev_d, R, S, K, NS)
    k_skip = pa.kde(ev_d, s, R, S, K, NS)
    torch.cuda.synchronize()
    assert int(k_skip["dev_status"].item()) == 0
    assert list(_record_widths(k_skip, n, R * S, R * S * K)) == [0] + [1] * (R * S - 1)
    got = {f: k_skip[f].cpu() for f in P.KDE_FIELDS}
    del k_skip
    k_full = pa.kde(ev_d, {f: v for f, v in s.items() if f != "n_invalid"}, R, S, K, NS)
    torch.cuda.synchronize()
    for f in P.KDE_FIELDS:
        assert torch.equal(got[f], k_full[f].cpu()), f
    del k_full, ev_d, s
    gc.collect()
    torch.cuda.empty_cache()
    ev_h = t.fill_host(0, 1)
    o = oracle.kde(ev_h, K, NS, n_events=len(ev_h["kernel_id"]))
    assert (o["n_clusters"] > 1).sum() > 8  # multimodal kernels are present
    P.assert_kde_equal(got, o, "long rank-step", rows=np.arange(K))


@pytest.mark.parametrize("name,n_check", [("production", 96), ("cluster", 48), ("skew", 48)])
def test_kde_full_size(name, n_check):
    _announce(f"kde full-size {name}")
    t = tracegen.make(name)
    c = t.cfg
    R, S, K, NS = c.n_ranks, c.n_steps, c.n_kernels, c.n_streams
    ev = t.fill_device(device=DEV)
    s, k = _kde_gpu(ev, R, S, K, NS)
    assert int(s["dev_status"].item()) == 0 and int(k["dev_status"].item()) == 0
    del ev, s, k["_workspace"]
    gc.collect()
    torch.cuda.empty_cache()
    G = c.n_segments
    segs = sorted(set(np.linspace(0, G - 1, n_check).astype(int).tolist()))
    print(f"[gpu-case] {name}: oracle over {len(segs)} segments", flush=True)
    o = P.oracle_kde_segments(t, segs)
    rows = np.concatenate([np.arange(g * K, (g + 1) * K) for g in segs])
    P.assert_kde_equal(k, o, name, rows=rows)
    nc = k["n_clusters"].cpu().numpy()
    assert (nc > 1).any() and nc.max() <= MAXC
