"""GPU parity of argus_summarize_keyed and argus_compact through the C ABI
against the CPU oracle: every keyed summary field and every byte of the
record stream must match exactly, with identical segment offsets.

Cases: random events whose kernels run on several streams (with invalid
records), key spaces in the dense and the mapped (two passes) layout, the
tiny trace with re-drawn streams, the record stream of both keyings,
truncation at a short capacity and sizing at capacity 0, and full-size
production and cluster summaries compacted in the launch configuration the
benchmark times.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2606_20374_amd as pa
import tracegen
from tests import parity as P

pytestmark = pytest.mark.gpu
DEV = "cuda"
SUM_FIELDS = ["count", "sum_ns", "min_ns", "max_ns", "hist", "n_valid", "n_invalid", "t_first", "t_last", "step_ns",
              "busy_ns", "stream_busy_ns", "wire_bytes"]


def _announce(name):
    print(f"\n[gpu-case] {name}", flush=True)


def _dev(ev):
    return {k: torch.from_numpy(np.ascontiguousarray(v)).to(DEV) for k, v in ev.items()}


def _random_events(rng, G, K, NS, n_per, p_bad=0.02):
    lens = rng.integers(0, n_per, size=G)
    off = np.zeros(G + 1, np.int64)
    np.cumsum(lens, out=off[1:])
    n = int(off[-1])
    kid = rng.integers(0, K, size=n).astype(np.int32)
    st = rng.integers(0, NS, size=n).astype(np.int32)
    bad = rng.random(n) < p_bad
    kid[bad] = -3
    t0 = rng.integers(0, 10**13, size=n).astype(np.int64)
    t1 = t0 + (2.0 ** rng.uniform(0, 36, size=n)).astype(np.int64)
    return {"kernel_id": kid, "stream": st, "start_ns": t0, "end_ns": t1, "seg_off": off}


def _keyed_both(ev, R, S, K, NS, what):
    s = pa.summarize(_dev(ev), R, S, K, NS, keyed=True)
    torch.cuda.synchronize()
    o = oracle.summarize(ev, K, NS, keyed=True)
    P.assert_int_equal(s, o, SUM_FIELDS, what)
    assert int(s["dev_status"].item()) == 0
    return s, o


def _compact_both(s, o, G, C, NS, what, cap=None):
    g = pa.compact(s, G, 1, C, NS, capacity=cap)
    torch.cuda.synchronize()
    ob, ooff = oracle.compact(o, G, C, NS, cap=cap)
    assert np.array_equal(g["seg_byte_off"].cpu().numpy(), ooff), what
    total = int(ooff[-1])
    gb = g["bytes"].cpu().numpy()
    n = len(ob)
    if cap is None or cap >= total:
        assert n == total and np.array_equal(gb[:total], ob), what
        assert int(g["dev_status"].item()) == 0
    else:
        # both write the records that fit entirely: compare the written prefix
        last = int(ooff[np.searchsorted(ooff, cap, side="right") - 1])
        assert np.array_equal(gb[:last], ob[:last]), what
        assert int(g["dev_status"].item()) == pa.argus.DEV_COMPACT_CAPACITY
    return g


@pytest.mark.parametrize("G,K,NS,seed", [(6, 7, 3, 0), (5, 64, 32, 1), (3, 1000, 16, 2), (2, 2048, 16, 3)])
def test_keyed_random(G, K, NS, seed):
    _announce(f"keyed summarize random G={G} K={K} NS={NS}")
    rng = np.random.default_rng(seed)
    ev = _random_events(rng, G, K, NS, 30_000)
    s, o = _keyed_both(ev, G, 1, K, NS, f"keyed {G}x{K}x{NS}")
    _compact_both(s, o, G, K * NS, NS, "compact keyed")


def test_keyed_tiny_with_redrawn_streams():
    _announce("keyed summarize: tiny trace, streams redrawn per event")
    t = tracegen.make("tiny")
    c = t.cfg
    ev = t.fill_host()
    rng = np.random.default_rng(9)
    ev["stream"] = ((ev["kernel_id"] + rng.integers(0, 3, size=len(ev["stream"]))) % c.n_streams).astype(np.int32)
    s, o = _keyed_both(ev, c.n_ranks, c.n_steps, c.n_kernels, c.n_streams, "tiny keyed")
    _compact_both(s, o, c.n_segments, c.n_kernels * c.n_streams, c.n_streams, "tiny keyed compact")


def test_compact_kernel_keys_capacity_and_sizing():
    _announce("compact: kernel-id keys, capacity cut, sizing only")
    t = tracegen.make("tiny")
    c = t.cfg
    G, K, NS = c.n_segments, c.n_kernels, c.n_streams
    ev = t.fill_host()
    s = pa.summarize(_dev(ev), c.n_ranks, c.n_steps, K, NS)
    o = oracle.summarize(ev, K, NS)
    g = _compact_both(s, o, G, K, 0, "tiny compact")
    total = int(g["seg_byte_off"][-1].item())
    assert np.array_equal(np.diff(g["seg_byte_off"].cpu().numpy()), o["wire_bytes"])
    for cap in (1, 100, total // 3 + 5, total - 1):
        _compact_both(s, o, G, K, 0, f"cap {cap}", cap=cap)
    # capacity 0 sizes the stream and writes nothing
    off = torch.empty(G + 1, dtype=torch.int64, device=DEV)
    st = torch.empty(1, dtype=torch.int32, device=DEV)
    ws = torch.empty(8 * G, dtype=torch.uint8, device=DEV)
    sm = pa.argus.Summary(*[s[f].data_ptr() if f in ("count", "sum_ns", "min_ns", "max_ns", "hist") else None
                            for f in pa.argus.SUMMARY_FIELDS])
    rc = pa.lib().argus_compact(ctypes.byref(sm), G, 1, K, 0, None, 0, off.data_ptr(), st.data_ptr(), ws.data_ptr(),
                                ws.numel(), torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert rc == 0 and int(off[-1].item()) == total
    assert int(st.item()) == (pa.argus.DEV_COMPACT_CAPACITY if total > 0 else 0)


@pytest.mark.parametrize("name", ["production", "cluster"])
def test_compact_full_size(name):
    _announce(f"compact full size {name}")
    t = tracegen.make(name)
    c = t.cfg
    R, S, K, NS = c.n_ranks, c.n_steps, c.n_kernels, c.n_streams
    G = c.n_segments
    s = pa.summarize(t.fill_device(device=DEV), R, S, K, NS)
    g = pa.compact(s, R, S, K, 0)
    torch.cuda.synchronize()
    assert int(g["dev_status"].item()) == 0
    goff = g["seg_byte_off"].cpu().numpy()
    gbytes = g["bytes"]
    del s
    torch.cuda.empty_cache()
    # sampled segments: each regenerated and summarized by the oracle, its
    # records compared byte for byte at the GPU's offset
    rng = np.random.default_rng(1)
    segs = sorted(rng.choice(G, size=min(G, 48), replace=False).tolist()) + [G - 1]
    for seg in segs:
        ev = t.fill_host(seg, seg + 1)
        o = oracle.summarize(ev, K, NS)
        ob, ooff = oracle.compact(o, 1, K, 0)
        assert goff[seg + 1] - goff[seg] == ooff[1], (name, seg)
        got = gbytes[goff[seg]:goff[seg + 1]].cpu().numpy()
        assert np.array_equal(got, ob), (name, seg)
    raw = 24 * c.events_per_seg
    print(f"[gpu-case] {name}: {goff[-1] / G:.0f} B per rank-step vs {raw} B raw ({raw * G / goff[-1]:.0f}x)",
          flush=True)
