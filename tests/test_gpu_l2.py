"""GPU parity of argus_l2 (section 6.1 routing; Appendix B, Eq. 5) through
the C ABI against the CPU oracle.

Group sizes, CV classes, straggler flags and counts must match exactly (both
sides decide them with exact integer comparisons); mean, std and CV (double)
and z (float) within 1e-5 relative. Cases: closed-form outlier groups, CV
boundaries, identical and all-zero groups, routing / membership / domain
rules with malformed and duplicate listings, random groups over ragged event
counts up to 65,536 ranks, and the medium trace through the GPU chain
summarize -> l2. The full-size workloads are checked in test_gpu_full.py.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2606_20374_amd as pa
import tracegen
from tests import parity as P

pytestmark = pytest.mark.gpu
DEV = "cuda"
STATUS_BITS = {1: pa.argus.DEV_GROUPS_MALFORMED, 2: pa.argus.DEV_GROUPS_DUPLICATE, 4: pa.argus.DEV_L2_DOMAIN}


def _announce(name):
    print(f"\n[gpu-case] {name}", flush=True)


def _t(x, dt):
    return torch.from_numpy(np.ascontiguousarray(np.asarray(x, dtype=dt))).to(DEV)


def assert_l2_equal(g: dict, o: dict, what: str):
    P.assert_int_equal(g, o, P.L2_INT_FIELDS, what)
    P.assert_float_close(g, o, P.L2_FLOAT_FIELDS, what)


def _both(cnt, sm, R, S, E, route, off, mem, what, **params):
    g = pa.l2(_t(np.asarray(cnt, np.uint32).view(np.int32), np.int32), _t(sm, np.int64), R, S, E, _t(route, np.uint8),
              _t(off, np.int32), _t(mem, np.int32), **params)
    torch.cuda.synchronize()
    o = oracle.l2(cnt, sm, R, S, E, route, off, mem, **params)
    assert_l2_equal(g, o, what)
    expect = sum(v for k, v in STATUS_BITS.items() if o["status"] & k)
    assert int(g["dev_status"].item()) == expect, (what, int(g["dev_status"].item()), o["status"])
    return g, o


def _one_group(xs, what, **params):
    R = len(xs)
    return _both(np.ones(R, np.uint32), np.asarray(xs, np.int64), R, 1, 1, np.zeros(1, np.uint8),
                 np.array([[0, R]], np.int32), np.arange(R, dtype=np.int32).reshape(1, R), what, **params)


def test_l2_hand_built_groups():
    _announce("l2 hand-built groups")
    for n in (3, 10, 11, 40):
        xs = [10_000] * n
        xs[n // 3] = 13_000
        g, _ = _one_group(xs, f"outlier n={n}")
        assert bool(P.to_np(g["flags"])[n // 3] & 2) == (n >= 11)
    for d in (99, 100, 249, 250):
        _one_group([5000 - d, 5000, 5000 + d], f"cv boundary d={d}")
    _one_group([7000] * 6, "identical")
    _one_group([0] * 4, "zeros")
    _one_group([2**40 - 1, 2**40 - 2, 3, 2**39], "near the domain edge")
    _one_group([5, 2**41, 6, 7], "out of the domain")


def test_l2_routing_membership_and_domain():
    _announce("l2 routing, membership, domain")
    R, S, E = 6, 2, 3
    cnt = np.ones(R * S * E, np.uint32)
    sm = np.full(R * S * E, 5000, np.int64)
    sm[((1 * S + 0) * E + 1)] = 9000
    cnt[((2 * S + 1) * E + 1)] = 0
    sm[((3 * S + 1) * E + 1)] = 1 << 41
    route = np.array([0xFF, 0, 1], np.uint8)
    off = np.array([[0, 3, 6], [0, 6, 6]], np.int32)
    mem = np.array([[0, 1, 2, 3, 4, 5], [0, 1, 2, 3, 2, 5]], np.int32)
    _both(cnt, sm, R, S, E, route, off, mem, "duplicate + domain", min_group=2)
    off2 = np.array([[0, 4, 2], [0, 6, 6]], np.int32)
    mem2 = np.array([[0, 1, 9, 3, 4, 5], [0, 1, 2, 3, 4, 5]], np.int32)
    _both(cnt, sm, R, S, E, route, off2, mem2, "malformed", min_group=2)
    off3 = np.array([[-1, 3, 7], [0, 6, 6]], np.int32)
    _both(cnt, sm, R, S, E, np.array([7, 0, 2], np.uint8), off3, mem2, "bad ranges and routes", min_group=2)


@pytest.mark.parametrize("R,S,E,seed", [(5, 2, 7, 0), (64, 3, 65, 1), (300, 1, 130, 2), (4099, 2, 33, 3),
                                        (65536, 1, 3, 4)])
def test_l2_random_groups(R, S, E, seed):
    _announce(f"l2 random groups R={R} S={S} E={E}")
    rng = np.random.default_rng(seed)
    cnt = rng.integers(0, 5, size=R * S * E).astype(np.uint32)
    base = rng.integers(1000, 10**8, size=E)
    slow = np.where(rng.random(R) < 0.02, rng.uniform(1.1, 1.6, size=R), 1.0)
    r_of = np.arange(R * S * E) // (S * E)
    xs = (base[np.arange(R * S * E) % E] * slow[r_of] * rng.uniform(0.97, 1.03, size=R * S * E)).astype(np.int64)
    sm = xs * cnt.astype(np.int64)
    n_dims, G = 3, max(2, R // 16)
    off = np.zeros((n_dims, G + 1), np.int32)
    mem = np.zeros((n_dims, R), np.int32)
    for d in range(n_dims):
        mem[d] = rng.permutation(R)
        off[d, 1:G] = np.sort(rng.integers(0, R + 1, size=G - 1))
        off[d, G] = R
    mem[2, :3] = mem[2, R - 3:]  # duplicate listings
    route = rng.integers(0, n_dims + 1, size=E).astype(np.uint8)
    route[route == n_dims] = 0xFF
    _both(cnt, sm, R, S, E, route, off, mem, f"random {R}x{S}x{E}", min_group=int(rng.integers(2, 5)),
          cv_mild_pm=int(rng.integers(5, 40)), cv_severe_pm=int(rng.integers(40, 120)),
          z_pm=int(rng.integers(1500, 3500)))


def test_l2_medium_chain():
    _announce("l2 medium trace: GPU summarize -> l2")
    t = tracegen.make("medium")
    c = t.cfg
    R, S, K, NS = c.n_ranks, c.n_steps, c.n_kernels, c.n_streams
    route, off, mem = tracegen.workload_groups("medium", R, K)
    s = pa.summarize(t.fill_device(device=DEV), R, S, K, NS)
    g = pa.l2(s["count"], s["sum_ns"], R, S, K, _t(route, np.uint8), _t(off, np.int32), _t(mem, np.int32))
    torch.cuda.synchronize()
    assert int(g["dev_status"].item()) == 0
    so = P.oracle_summary_sharded(t)
    o = oracle.l2(so["count"], so["sum_ns"], R, S, K, route, off, mem)
    assert_l2_equal(g, o, "medium chain")
