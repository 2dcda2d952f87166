"""argus_summarize_noalloc (no allocation, scratch in a static per-device
array) against argus_summarize (caller workspace), through the C ABI: two
calls in a row on the same device, the second with a smaller input, each
compared element by element with argus_summarize's output on the same
events, and both with the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_20374_amd as pa
import tracegen
from tests import parity as P

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _check(trace, what):
    c = trace.cfg
    R, S, K, NS = c.n_ranks, c.n_steps, c.n_kernels, c.n_streams
    print(f"\n[gpu-case] no-alloc summarize: {what} {R}x{S}x{c.events_per_seg} K={K}", flush=True)
    ev = trace.fill_device(device=DEV)
    ref = pa.summarize(ev, R, S, K, NS)
    got = pa.summarize_noalloc(ev, R, S, K, NS)
    torch.cuda.synchronize()
    assert int(got["dev_status"].item()) == 0
    o = oracle.summarize(trace.fill_host(), K, NS)
    P.assert_int_equal(ref, o, P.SUM_INT_FIELDS, what + " (workspace entry point)")
    P.assert_int_equal(got, o, P.SUM_INT_FIELDS, what + " (no-alloc entry point)")
    pres = ref["count"] != 0
    for f in P.SUM_INT_FIELDS:
        a, b = ref[f], got[f]
        if f in P.PRESENT_ONLY:
            keep = pres.repeat_interleave(a.numel() // pres.numel())
            a, b = a[keep], b[keep]
        assert torch.equal(a, b), (what, f)


def test_noalloc_matches_workspace_entry_point_twice():
    # the dense (2,048 ids) and then a smaller mapped (8,200 ids) input: the
    # second call reuses the scratch the first one left behind
    _check(tracegen.make("production", n_ranks=24), "first call")
    _check(tracegen.make("skew", n_ranks=6, n_steps=2, events_per_seg=30_000), "second, smaller call")
