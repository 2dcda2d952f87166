"""Pins of the oracle's (kernel, stream)-keyed summaries and of its uploaded
record stream (section 5.2 grouping per (kernel, stream, rank); the compact
summary whose size section 8.3 compares with the raw trace):

* keyed cells against a dict-of-lists brute force over (segment, kernel,
  stream) on random events whose kernels run on several streams;
* keyed cells summed over streams equal the kernel-id cells;
* with the generator's stream = kernel id mod NS, each kernel's only
  nonzero keyed cell is that stream's, equal to the kernel-id cell;
* the record stream parsed back with `struct` (independent of the oracle's
  writer) reproduces every present cell in key order; offsets are the
  running totals of the per-segment wire sizes, the total their sum; a
  short capacity keeps the offsets and writes only what fits.
"""
import struct
from collections import defaultdict

import numpy as np
import pytest

import oracle
import tracegen

NB = 32


def _bin(d):
    return min(d.bit_length() - 1, NB - 1) if d >= 2 else 0


def _random_events(rng, G, K, NS, n_per):
    lens = rng.integers(0, n_per, size=G)
    off = np.zeros(G + 1, np.int64)
    np.cumsum(lens, out=off[1:])
    n = int(off[-1])
    kid = rng.integers(-1, K + 1, size=n).astype(np.int32)
    st = rng.integers(-1, NS + 1, size=n).astype(np.int32)
    t0 = rng.integers(0, 10**12, size=n).astype(np.int64)
    d = (2.0 ** rng.uniform(0, 34, size=n)).astype(np.int64)
    t1 = t0 + d
    back = rng.random(n) < 0.02
    t1[back] = t0[back] - 5
    return {"kernel_id": kid, "stream": st, "start_ns": t0, "end_ns": t1, "seg_off": off}


@pytest.mark.parametrize("seed", range(3))
def test_keyed_bruteforce(seed):
    rng = np.random.default_rng(seed)
    G, K, NS = 5, 7, 3
    ev = _random_events(rng, G, K, NS, 400)
    o = oracle.summarize(ev, K, NS, keyed=True)
    groups = defaultdict(list)
    for g in range(G):
        for i in range(ev["seg_off"][g], ev["seg_off"][g + 1]):
            k, s, a, b = (int(ev[f][i]) for f in ("kernel_id", "stream", "start_ns", "end_ns"))
            if 0 <= k < K and 0 <= s < NS and a >= 0 and b >= a:
                groups[(g, k, s)].append(b - a)
    for g in range(G):
        for k in range(K):
            for s in range(NS):
                c = (g * K + k) * NS + s
                ds = groups.get((g, k, s), [])
                assert o["count"][c] == len(ds)
                assert o["sum_ns"][c] == sum(ds)
                assert o["min_ns"][c] == (min(ds) if ds else 2**63 - 1)
                assert o["max_ns"][c] == (max(ds) if ds else -2**63)
                h = np.zeros(NB, np.uint32)
                for d in ds:
                    h[_bin(d)] += 1
                assert np.array_equal(o["hist"][c], h)
    # per-segment aggregates do not depend on the keying
    u = oracle.summarize(ev, K, NS)
    for f in ("n_valid", "n_invalid", "t_first", "t_last", "step_ns", "busy_ns", "stream_busy_ns"):
        assert np.array_equal(o[f], u[f]), f
    # keyed cells folded over streams give the kernel-id cells
    cnt = o["count"].reshape(G, K, NS)
    assert np.array_equal(cnt.sum(axis=2), u["count"].reshape(G, K))
    assert np.array_equal(o["sum_ns"].reshape(G, K, NS).sum(axis=2), u["sum_ns"].reshape(G, K))
    assert np.array_equal(o["hist"].reshape(G, K, NS, NB).sum(axis=2), u["hist"].reshape(G, K, NB))
    mn = np.where(cnt > 0, o["min_ns"].reshape(G, K, NS), 2**63 - 1).min(axis=2)
    assert np.array_equal(mn, u["min_ns"].reshape(G, K))


def test_keyed_generator_streams():
    t = tracegen.make("tiny")
    c = t.cfg
    G, K, NS = c.n_segments, c.n_kernels, c.n_streams
    ev = t.fill_host()
    o = oracle.summarize(ev, K, NS, keyed=True)
    u = oracle.summarize(ev, K, NS)
    cnt = o["count"].reshape(G, K, NS)
    own = np.arange(K) % NS
    mask = np.zeros((K, NS), bool)
    mask[np.arange(K), own] = True
    assert (cnt[:, ~mask] == 0).all()
    assert np.array_equal(cnt[:, mask], u["count"].reshape(G, K))
    assert np.array_equal(o["sum_ns"].reshape(G, K, NS)[:, mask], u["sum_ns"].reshape(G, K))


def _parse(buf, off, G, NS):
    recs = []
    for g in range(G):
        p = int(off[g])
        while p < off[g + 1]:
            key, cnt, sm, mn, mx, nnz = struct.unpack_from("<IIqqqB", buf, p)
            p += 33
            bins = [struct.unpack_from("<BI", buf, p + 5 * j) for j in range(nnz)]
            p += 5 * nnz
            k, s = (key & 0xFFFFFF, key >> 24) if NS else (key, 0)
            recs.append((g, k, s, cnt, sm, mn, mx, bins))
        assert p == off[g + 1]
    return recs


@pytest.mark.parametrize("keyed", [False, True])
def test_compact_round_trip(keyed):
    rng = np.random.default_rng(7)
    G, K, NS = 6, 9, 4
    ev = _random_events(rng, G, K, NS, 300)
    o = oracle.summarize(ev, K, NS, keyed=keyed)
    KC = K * NS if keyed else K
    buf, off = oracle.compact(o, G, KC, NS if keyed else 0)
    assert off[0] == 0 and np.array_equal(np.diff(off), o["wire_bytes"]) and len(buf) == off[-1]
    recs = _parse(buf.tobytes(), off, G, NS if keyed else 0)
    present = [(g, c) for g in range(G) for c in range(KC) if o["count"][g * KC + c] > 0]
    assert len(recs) == len(present)
    for (g, c), r in zip(present, recs):
        i = g * KC + c
        k, s = (c // NS, c % NS) if keyed else (c, 0)
        assert r[:7] == (g, k, s, o["count"][i], o["sum_ns"][i], o["min_ns"][i], o["max_ns"][i])
        nz = np.nonzero(o["hist"][i])[0]
        assert r[7] == [(int(b), int(o["hist"][i][b])) for b in nz]


def test_compact_capacity_and_empty():
    rng = np.random.default_rng(3)
    G, K, NS = 4, 5, 2
    ev = _random_events(rng, G, K, NS, 200)
    o = oracle.summarize(ev, K, NS)
    full, off = oracle.compact(o, G, K)
    part, off2 = oracle.compact(o, G, K, cap=int(off[2]) + 7)
    assert np.array_equal(off, off2)
    assert np.array_equal(part[:off[2]], full[:off[2]])
    empty = {f: np.zeros_like(o[f]) for f in ("count", "sum_ns", "min_ns", "max_ns", "hist")}
    b, off3 = oracle.compact(empty, G, K)
    assert len(b) == 0 and (off3 == 0).all()


def test_compression_of_the_tiny_trace():
    t = tracegen.make("tiny")
    c = t.cfg
    o = oracle.summarize(t.fill_host(), c.n_kernels, c.n_streams)
    buf, off = oracle.compact(o, c.n_segments, c.n_kernels)
    raw = 24 * c.events_per_seg
    per_seg = np.diff(off)
    # 64 kernels present per rank-step, one or two octave bins each
    assert ((per_seg >= 64 * 38) & (per_seg <= 64 * 48)).all()
    assert raw / per_seg.mean() > 150
