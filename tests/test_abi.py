"""The C-ABI library loads and exports every symbol the headers declare;
host-side argument checks reject bad calls before any launch (no GPU needed)."""
import ctypes
import glob
import os
import re

import pytest

import paper_2606_20374_amd as pa
from paper_2606_20374_amd import argus as A

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        for m in re.finditer(r"^\s*(?:const\s+)?[\w\s\*]+?\b(argus_\w+)\s*\(", text, flags=re.M):
            names.add(m.group(1))
    return names


def test_every_declared_symbol_is_exported():
    names = _declared_functions()
    assert {"argus_summarize", "argus_cross_rank", "argus_iter_windows", "argus_abi_version"} <= names
    L = ctypes.CDLL(A.LIB_PATH)
    for n in sorted(names):
        assert hasattr(L, n), n


def test_version_and_defaults():
    assert pa.lib().argus_abi_version() == 1
    assert pa.xr_defaults() == dict(min_ranks=3, c_min_pair=8, min_kernels=8, k_mad_pm=5189, ratio_pm=1250,
                                     alpha_pm=1500, tau_rank_pm=20)
    assert pa.l1_defaults() == dict(W=5, theta_pm=1500, beta_pm=1200, rho_pm=1300, cmax_pm=100, min_seg=2)
    assert pa.lib().argus_status_string(-1) == b"invalid argument"
    assert pa.kde_defaults() == dict(sub_bits=6, frac_pm=50, min_count=3, gap=48)


def test_workspace_sizes():
    assert pa.lib().argus_cross_rank_workspace(10240, 1, 2048) == 10240 * 2048 * 8
    assert pa.lib().argus_iter_windows_workspace(10, 10) == 0
    e = A.Events(0, 0, 0, 0, 0, 0, 1, 1, 1, 1)
    assert pa.lib().argus_summarize_workspace(ctypes.byref(e)) == 256
    # 256 fixed + 8 B per event + 3 x 4 B + 2 B per cell + 8 KB of class counters
    # + 1 B per rank-step (record width), each part 256-byte aligned
    assert pa.kde_workspace_bytes(4_096_000_000, 10240, 1, 2048) == (
        256 + 4_096_000_000 * 8 + 3 * 10240 * 2048 * 4 + 10240 * 2048 * 2 + 8192 + 10240)
    assert pa.kde_workspace_bytes(10, 1, 1, 3) == 256 + 256 + 3 * 256 + 256 + 8192 + 256


@pytest.mark.parametrize("mutate", [
    lambda e, s: setattr(e, "n_kernels", 0),
    lambda e, s: setattr(e, "n_kernels", 65537),
    lambda e, s: setattr(e, "n_streams", 65),
    lambda e, s: setattr(e, "n_ranks", -1),
    lambda e, s: setattr(e, "seg_off", None),
    lambda e, s: setattr(s, "hist", None),
    lambda e, s: setattr(s, "hist", 0x1008),  # misaligned histogram
    None,  # no workspace
])
def test_summarize_rejects_bad_arguments(mutate):
    e = A.Events(0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 10, 2, 2, 4, 2)
    s = A.Summary(*([0x1000] * 12 + [None, None]))
    ws, n = (0x2000, 256) if mutate else (None, 0)
    if mutate:
        mutate(e, s)
    assert pa.lib().argus_summarize(ctypes.byref(e), ctypes.byref(s), ws, n, None) == A.EINVAL


def test_cross_rank_and_l1_reject_bad_arguments():
    p = A.XrParams()
    pa.lib().argus_xr_default(ctypes.byref(p))
    o = A.XrOut(*([0x1000] * 16))
    L = pa.lib()
    assert L.argus_cross_rank(0x1000, 0x1000, 16385, 1, 4, ctypes.byref(p), ctypes.byref(o), 0x1000, 1 << 40,
                              None) == A.EINVAL
    assert L.argus_cross_rank(0x1000, 0x1000, 8, 1, 4, ctypes.byref(p), ctypes.byref(o), 0x1000, 8, None) == A.EINVAL
    p.min_ranks = 0
    assert L.argus_cross_rank(0x1000, 0x1000, 8, 1, 4, ctypes.byref(p), ctypes.byref(o), 0x1000, 1 << 20,
                              None) == A.EINVAL
    q = A.L1Params()
    L.argus_l1_default(ctypes.byref(q))
    assert L.argus_iter_windows(0x1000, 4, 4097, ctypes.byref(q), 0x1000, 0x1000, 0x1000, 0x1000, None, None, None,
                                0, None) == A.EINVAL
    q.W = 0
    assert L.argus_iter_windows(0x1000, 4, 8, ctypes.byref(q), 0x1000, 0x1000, 0x1000, 0x1000, None, None, None, 0,
                                None) == A.EINVAL


@pytest.mark.parametrize("mutate", [
    lambda e, s, p: setattr(e, "n_kernels", 16385),
    lambda e, s, p: setattr(s, "min_ns", None),
    lambda e, s, p: setattr(p, "sub_bits", 7),
    lambda e, s, p: setattr(p, "sub_bits", 0),
    lambda e, s, p: setattr(p, "frac_pm", 1001),
    lambda e, s, p: setattr(p, "min_count", 0),
    lambda e, s, p: setattr(p, "gap", -1),
    "misaligned", "small", "misaligned_out",
])
def test_kde_rejects_bad_arguments(mutate):
    e = A.Events(0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 10, 2, 2, 4, 2)
    s = A.Summary(*([0x1000] * 12 + [None, None]))
    p = A.KdeParams()
    pa.lib().argus_kde_default(ctypes.byref(p))
    o = A.KdeOut(0x1000, 0x1000, 0x1000, 0x1000, None, None)
    ws, n = 0x10000, 1 << 20
    if mutate == "misaligned":
        ws = 0x10080
    elif mutate == "small":
        n = 256
    elif mutate == "misaligned_out":
        o.p50_ns = 0x1008
    else:
        mutate(e, s, p)
    assert pa.lib().argus_kde(ctypes.byref(e), ctypes.byref(s), ctypes.byref(p), ctypes.byref(o), ws, n,
                              None) == A.EINVAL


def test_w1_defaults_and_workspace():
    assert pa.w1_defaults() == dict(grid=64, min_ranks=3, alpha_pm=1500)
    def al256(x):
        return (x + 255) // 256 * 256
    # CDF values (rows of an odd rank count padded to even), then 9 bytes per
    # (step, kernel, rank) of staged scores and flags
    assert pa.lib().argus_w1_workspace(10240, 1, 2048, 64) == 2 * 10240 * 2048 * 64 + 9 * 10240 * 2048
    assert pa.lib().argus_w1_workspace(3, 2, 5, 64) == al256(2 * 4 * 2 * 5 * 64) + 9 * 4 * 2 * 5
    assert pa.lib().argus_w1_workspace(3, 2, 5, 2) == al256(2 * 4 * 2 * 5 * 2) + 9 * 4 * 2 * 5


@pytest.mark.parametrize("mutate", [
    lambda c, p, o, d: setattr(p, "grid", 1),
    lambda c, p, o, d: setattr(p, "grid", 2049),
    lambda c, p, o, d: setattr(p, "min_ranks", 0),
    lambda c, p, o, d: setattr(p, "alpha_pm", -1),
    lambda c, p, o, d: setattr(c, "p99_ns", None),
    lambda c, p, o, d: setattr(c, "count", 0x1008),  # misaligned cluster counts
    lambda c, p, o, d: setattr(o, "score", None),
    lambda c, p, o, d: d.__setitem__("R", 16385),
    lambda c, p, o, d: d.__setitem__("S", 0),
    "misaligned", "small", "steps",
])
def test_w1_rejects_bad_arguments(mutate):
    c = A.KdeOut(0x1000, 0x1000, 0x1000, 0x1000, None, None)
    p = A.W1Params()
    pa.lib().argus_w1_default(ctypes.byref(p))
    o = A.W1Out(*([0x1000] * 9 + [None]))
    d = {"R": 8, "S": 2, "K": 4}
    ws, n = 0x10000, 1 << 20
    if mutate == "misaligned":
        ws = 0x10080
    elif mutate == "small":
        n = 2 * 8 * 2 * 4 * 64 - 1
    elif mutate == "steps":  # one step above the limit, everything else valid
        d["S"] = A.MAX_W1_STEPS + 1
        n = 2 * 8 * d["S"] * 4 * 64
    else:
        mutate(c, p, o, d)
    assert pa.lib().argus_w1(ctypes.byref(c), d["R"], d["S"], d["K"], ctypes.byref(p), ctypes.byref(o), ws, n,
                             None) == A.EINVAL


def test_l2_defaults_and_workspace():
    assert pa.l2_defaults() == dict(min_group=3, cv_mild_pm=20, cv_severe_pm=50, z_pm=3000)
    assert pa.lib().argus_l2_workspace(10240, 4) == 4 * 10240 * 4


@pytest.mark.parametrize("mutate", [
    lambda g, p, o, d: setattr(g, "n_dims", 0),
    lambda g, p, o, d: setattr(g, "n_dims", 17),
    lambda g, p, o, d: setattr(g, "max_groups", 0),
    lambda g, p, o, d: setattr(g, "max_groups", 65536),
    lambda g, p, o, d: setattr(g, "members", None),
    lambda g, p, o, d: setattr(p, "min_group", 1),
    lambda g, p, o, d: setattr(p, "z_pm", 1000001),
    lambda g, p, o, d: setattr(p, "cv_mild_pm", -1),
    lambda g, p, o, d: setattr(o, "cls", None),
    lambda g, p, o, d: d.__setitem__("R", 65537),
    lambda g, p, o, d: d.__setitem__("S", 65535),  # S * n_dims over the launch limit
    "misaligned", "small",
])
def test_l2_rejects_bad_arguments(mutate):
    g = A.Groups(0x1000, 0x1000, 0x1000, 2, 4)
    p = A.L2Params()
    pa.lib().argus_l2_default(ctypes.byref(p))
    o = A.L2Out(*([0x1000] * 8 + [None]))
    d = {"R": 8, "S": 2, "K": 4}
    ws, n = 0x10000, 1 << 20
    if mutate == "misaligned":
        ws = 0x10002
    elif mutate == "small":
        n = 4 * 8 * 2 - 1
    else:
        mutate(g, p, o, d)
    assert pa.lib().argus_l2(0x1000, 0x1000, d["R"], d["S"], d["K"], ctypes.byref(g), ctypes.byref(p),
                             ctypes.byref(o), ws, n, None) == A.EINVAL


def test_compact_workspace_and_bad_arguments():
    L = pa.lib()
    assert L.argus_compact_workspace(10240, 1) == 8 * 10240
    s = A.Summary(*([0x1000] * 12 + [None, None]))
    ok = dict(R=4, S=2, C=6, NS=0, out=0x1000, cap=100, seg=0x2000, ws=0x3000, n=1 << 10)
    bad = [dict(C=0), dict(NS=-1), dict(NS=65), dict(C=7, NS=2), dict(cap=-1), dict(out=None),
           dict(seg=None), dict(ws=0x3004), dict(n=63), dict(R=-1)]
    for b in bad:
        a = dict(ok, **b)
        assert L.argus_compact(ctypes.byref(s), a["R"], a["S"], a["C"], a["NS"], a["out"], a["cap"], a["seg"], None,
                               a["ws"], a["n"], None) == A.EINVAL, b
    s2 = A.Summary(*([0x1000] * 4 + [0x1008] + [0x1000] * 7 + [None, None]))  # misaligned histogram
    assert L.argus_compact(ctypes.byref(s2), 4, 2, 6, 0, 0x1000, 100, 0x2000, None, 0x3000, 1 << 10, None) == A.EINVAL


def test_summarize_keyed_rejects_large_key_space():
    e = A.Events(0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 10, 2, 2, 4097, 16)  # 4097 x 16 > 65536 keys
    s = A.Summary(*([0x1000] * 12 + [None, None]))
    assert pa.lib().argus_summarize_keyed(ctypes.byref(e), ctypes.byref(s), 0x2000, 256, None) == A.EINVAL


def test_summarize_noalloc_rejects_null_arguments():
    L = pa.lib()
    e = A.Events()
    s = A.Summary()
    assert L.argus_summarize_noalloc(None, ctypes.byref(s), None) == A.EINVAL
    assert L.argus_summarize_noalloc(ctypes.byref(e), None, None) == A.EINVAL
    # its scratch covers what argus_summarize asks for
    assert L.argus_summarize_workspace(ctypes.byref(e)) <= A.NOALLOC_SCRATCH_BYTES
