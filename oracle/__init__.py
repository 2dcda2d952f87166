"""ctypes wrapper of the plain C oracle (liboracle.so).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg are the only callers. The product path never imports this
package. Inputs and outputs are numpy arrays on the host.
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# ARGUS_ORACLE_LIB names another build of the same sources (the sanitizer
# build of the test suite)
LIB_PATH = os.environ.get("ARGUS_ORACLE_LIB") or os.path.join(HERE, "liboracle.so")
NB = 32

# Proposed defaults (the paper prints no values for these thresholds).
XR_DEFAULTS = dict(min_ranks=3, c_min_pair=8, min_kernels=8, k_mad_pm=5189, ratio_pm=1250, alpha_pm=1500,
                   tau_rank_pm=20)
L1_DEFAULTS = dict(W=5, theta_pm=1500, beta_pm=1200, rho_pm=1300, cmax_pm=100, min_seg=2)
KDE_DEFAULTS = dict(sub_bits=6, frac_pm=50, min_count=3, gap=48)
W1_DEFAULTS = dict(grid=64, min_ranks=3, alpha_pm=1500)
L2_DEFAULTS = dict(min_group=3, cv_mild_pm=20, cv_severe_pm=50, z_pm=3000)
L2_NOT_EVALUATED = 0xFF
KDE_MAXC = 4

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        V, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        L.orc_bin.argtypes = [ctypes.c_uint64]
        L.orc_bin.restype = ctypes.c_int
        L.orc_summarize.argtypes = [I64, I32, I32, I64] + [V] * 5 + [V] * 5 + [V] * 8
        L.orc_summarize.restype = I64
        L.orc_summarize_keyed.argtypes = [I64, I32, I32, I64] + [V] * 5 + [V] * 5 + [V] * 8
        L.orc_summarize_keyed.restype = I64
        L.orc_compact.argtypes = [I64, I64, I32] + [V] * 5 + [V, I64, V]
        L.orc_compact.restype = I64
        L.orc_cross_rank.argtypes = [I32, I32, I32, V, V] + [I32] * 7 + [V] * 8 + [V] * 3 + [V] * 4
        L.orc_cross_rank.restype = ctypes.c_int
        L.orc_iter_windows.argtypes = [I32, I32, V] + [I32] * 6 + [V] * 5
        L.orc_iter_windows.restype = ctypes.c_int
        L.orc_kde_thresholds.argtypes = [V]
        L.orc_kde_bin.argtypes = [ctypes.c_uint64, I32]
        L.orc_kde_bin.restype = ctypes.c_int
        L.orc_kde_group.argtypes = [I64, V] + [I32] * 4 + [V] * 8
        L.orc_kde_weights.argtypes = [I64, I32, V]
        L.orc_kde_root5.argtypes = [I64]
        L.orc_kde_root5.restype = ctypes.c_double
        L.orc_kde_bw_q8.argtypes = [ctypes.c_double, I64]
        L.orc_kde_bw_q8.restype = I64
        L.orc_kde_weights_many.argtypes = [V, V, I32, V]
        L.orc_kde_root5_many.argtypes = [V, I64, V]
        L.orc_kde_bw_q8_many.argtypes = [V, V, I64, V]
        L.orc_kde_bin_many.argtypes = [V, I64, V]
        L.orc_kde.argtypes = [I64, I32, I32, I64] + [V] * 5 + [I32] * 4 + [V] * 5
        L.orc_kde.restype = I64
        L.orc_w1.argtypes = [I32, I32, I32] + [V] * 4 + [I32] * 3 + [V] * 9
        L.orc_w1.restype = ctypes.c_int
        L.orc_w1_cdf_q.argtypes = [I32, V, V, V, ctypes.c_double]
        L.orc_w1_cdf_q.restype = ctypes.c_uint32
        L.orc_w1_cdf_q_at.argtypes = [I32, V, V, V, ctypes.c_double]
        L.orc_w1_cdf_q_at.restype = ctypes.c_uint32
        L.orc_l2.argtypes = [I32, I32, I32] + [V] * 5 + [I32] * 6 + [V] * 8
        L.orc_l2.restype = ctypes.c_int
        _lib = L
    return _lib


def _p(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be contiguous"
    return a.ctypes.data


def bin_of(d: int) -> int:
    return lib().orc_bin(d)


def summarize(ev: dict, n_kernels: int, n_streams: int, n_events: int | None = None, keyed: bool = False) -> dict:
    """Exact per-(segment, kernel) group-by (keyed: per (segment, kernel,
    stream), cells [G][K][NS]). ev: kernel_id, stream, start_ns, end_ns,
    seg_off (numpy). Returns dict of numpy outputs; 'bad_segments' counts
    malformed segments."""
    kid = np.ascontiguousarray(ev["kernel_id"], dtype=np.int32)
    st = np.ascontiguousarray(ev["stream"], dtype=np.int32)
    t0 = np.ascontiguousarray(ev["start_ns"], dtype=np.int64)
    t1 = np.ascontiguousarray(ev["end_ns"], dtype=np.int64)
    off = np.ascontiguousarray(ev["seg_off"], dtype=np.int64)
    G = len(off) - 1
    K, NS = n_kernels, n_streams
    KC = K * NS if keyed else K
    n = len(kid) if n_events is None else n_events
    out = {
        "count": np.empty(G * KC, np.uint32), "sum_ns": np.empty(G * KC, np.int64),
        "min_ns": np.empty(G * KC, np.int64), "max_ns": np.empty(G * KC, np.int64),
        "hist": np.empty(G * KC * NB, np.uint32),
        "n_valid": np.empty(G, np.uint32), "n_invalid": np.empty(G, np.uint32),
        "t_first": np.empty(G, np.int64), "t_last": np.empty(G, np.int64), "step_ns": np.empty(G, np.int64),
        "busy_ns": np.empty(G, np.int64), "stream_busy_ns": np.empty(G * NS, np.int64),
        "wire_bytes": np.empty(G, np.int64),
    }
    fn = lib().orc_summarize_keyed if keyed else lib().orc_summarize
    bad = fn(G, K, NS, n, _p(kid), _p(st), _p(t0), _p(t1), _p(off),
                              *[_p(out[k]) for k in ("count", "sum_ns", "min_ns", "max_ns", "hist", "n_valid",
                                                     "n_invalid", "t_first", "t_last", "step_ns", "busy_ns",
                                                     "stream_busy_ns", "wire_bytes")])
    out["hist"] = out["hist"].reshape(G * KC, NB)
    out["stream_busy_ns"] = out["stream_busy_ns"].reshape(G, NS)
    out["bad_segments"] = int(bad)
    return out


def compact(summary: dict, n_seg: int, n_cells: int, n_streams: int = 0, cap: int | None = None):
    """Record stream of dense summaries ([n_seg][n_cells] arrays): (bytes,
    seg_byte_off [n_seg + 1]). n_streams = 0 for kernel-id keys, else the
    stream count of (kernel, stream) keys."""
    f = {k: np.ascontiguousarray(summary[k]).reshape(-1) for k in ("count", "sum_ns", "min_ns", "max_ns", "hist")}
    ptrs = [_p(f[k]) for k in ("count", "sum_ns", "min_ns", "max_ns", "hist")]
    off = np.empty(n_seg + 1, np.int64)
    if cap is None:
        lib().orc_compact(n_seg, n_cells, n_streams, *ptrs, None, 0, _p(off))
        cap = int(off[-1])
    buf = np.zeros(max(cap, 1), np.uint8)
    total = lib().orc_compact(n_seg, n_cells, n_streams, *ptrs, _p(buf), cap, _p(off))
    return buf[:min(total, cap)], off


def cross_rank(count: np.ndarray, sum_ns: np.ndarray, R: int, S: int, K: int, **params) -> dict:
    p = dict(XR_DEFAULTS, **params)
    count = np.ascontiguousarray(count, dtype=np.uint32).reshape(-1)
    sum_ns = np.ascontiguousarray(sum_ns, dtype=np.int64).reshape(-1)
    assert count.size == R * S * K and sum_ns.size == R * S * K
    SK, C, RS = S * K, R * S * K, R * S
    out = {
        "n_present": np.empty(SK, np.uint32), "med_ns": np.empty(SK, np.int64), "mad_ns": np.empty(SK, np.int64),
        "q1_ns": np.empty(SK, np.int64), "q3_ns": np.empty(SK, np.int64), "xmean_ns": np.empty(SK, np.float32),
        "n_flag": np.empty(SK, np.uint32), "n_degraded": np.empty(SK, np.uint32),
        "z": np.empty(C, np.float32), "mean_ns": np.empty(C, np.float32), "flags": np.empty(C, np.uint8),
        "score_pm": np.empty(RS, np.int32), "n_eval": np.empty(RS, np.uint32), "n_flag_rank": np.empty(RS, np.uint32),
        "straggler": np.empty(RS, np.uint8),
    }
    rc = lib().orc_cross_rank(R, S, K, _p(count), _p(sum_ns), p["min_ranks"], p["c_min_pair"], p["min_kernels"],
                              p["k_mad_pm"], p["ratio_pm"], p["alpha_pm"], p["tau_rank_pm"],
                              *[_p(out[k]) for k in ("n_present", "med_ns", "mad_ns", "q1_ns", "q3_ns", "xmean_ns",
                                                     "n_flag", "n_degraded", "z", "mean_ns", "flags", "score_pm",
                                                     "n_eval", "n_flag_rank", "straggler")])
    if rc != 0:
        raise RuntimeError(f"orc_cross_rank failed: {rc}")
    return out


def iter_windows(step_ns: np.ndarray, R: int, S: int, **params) -> dict:
    p = dict(L1_DEFAULTS, **params)
    y = np.ascontiguousarray(step_ns, dtype=np.int64).reshape(-1)
    assert y.size == R * S
    out = {"flags": np.empty(R * S, np.uint8), "cls": np.empty(R, np.uint8), "eff_width": np.empty(R, np.int32),
           "cp": np.empty(R, np.int32), "cp_ratio": np.empty(R, np.float32)}
    rc = lib().orc_iter_windows(R, S, _p(y), p["W"], p["theta_pm"], p["beta_pm"], p["rho_pm"], p["cmax_pm"],
                                p["min_seg"], *[_p(out[k]) for k in ("flags", "cls", "eff_width", "cp", "cp_ratio")])
    if rc != 0:
        raise RuntimeError(f"orc_iter_windows failed: {rc}")
    return out


def kde_thresholds() -> np.ndarray:
    """The 64 mantissa thresholds ceil(2^(23 + t/64)) of the KDE log grid."""
    th = np.empty(64, np.uint32)
    lib().orc_kde_thresholds(_p(th))
    return th


def kde_bin(d: int, sub_bits: int = 6) -> int:
    return lib().orc_kde_bin(d, sub_bits)


def kde_bin_many(d: np.ndarray) -> np.ndarray:
    """kde_bin(d, 6) for an array of durations (uint64)."""
    d = np.ascontiguousarray(d, dtype=np.uint64)
    out = np.empty(d.size, np.int32)
    lib().orc_kde_bin_many(_p(d), d.size, _p(out))
    return out


def _kde_params(params: dict) -> dict:
    p = dict(KDE_DEFAULTS, **params)
    assert 1 <= p["sub_bits"] <= 6
    return p


def kde_group(durations, debug: bool = False, **params) -> dict:
    """Clusters of one group of durations (any order): n_clusters, count,
    p50, p99 (KDE_MAXC slots), bw_q8 (bandwidth in 1/256 grid steps) and
    n_cand (valleys before filtering). With debug, also the grid density
    "f" and the unfiltered valley positions "cand" (grid indices)."""
    p = _kde_params(params)
    d = np.ascontiguousarray(np.asarray(durations, dtype=np.uint64).reshape(-1))
    ncl = np.zeros(1, np.uint8)
    cnt = np.zeros(KDE_MAXC, np.uint32)
    p50 = np.zeros(KDE_MAXC, np.int64)
    p99 = np.zeros(KDE_MAXC, np.int64)
    bw = np.zeros(1, np.int32)
    nc = np.zeros(1, np.int32)
    f = np.zeros(4096, np.uint64) if debug else None
    cand = np.zeros(4096, np.int32) if debug else None
    lib().orc_kde_group(d.size, _p(d) if d.size else None, p["sub_bits"], p["frac_pm"], p["min_count"], p["gap"],
                        _p(ncl), _p(cnt), _p(p50), _p(p99), _p(bw), _p(nc), None if f is None else _p(f),
                        None if cand is None else _p(cand))
    out = {"n_clusters": int(ncl[0]), "count": cnt, "p50_ns": p50, "p99_ns": p99, "bw_q8": int(bw[0]),
           "n_cand": int(nc[0])}
    if debug and d.size:
        G = kde_bin(int(d.max()), p["sub_bits"]) - kde_bin(int(d.min()), p["sub_bits"]) + 1
        out["f"] = f[:G]
        out["cand"] = cand[:out["n_cand"]]
    return out


def kde_weights(H: int, nt: int) -> np.ndarray:
    """The integer weights w(0 .. nt-1) of bandwidth H (1/256 grid steps)."""
    w = np.empty(nt, np.uint32)
    lib().orc_kde_weights(H, nt, _p(w))
    return w


def kde_root5(n: int) -> float:
    """n^(-1/5) as the oracle's bandwidth takes it (the nearest double)."""
    return lib().orc_kde_root5(n)


def kde_bw_q8(var: float, n: int) -> int:
    """The quantised bandwidth H of a group of n grid values of variance var."""
    return lib().orc_kde_bw_q8(var, n)


def kde_weights_many(H: np.ndarray, off: np.ndarray) -> np.ndarray:
    """Weights of t = 0 .. off[i+1]-off[i]-1 for every bandwidth H[i], laid
    out at w[off[i]:off[i+1]]."""
    H = np.ascontiguousarray(H, dtype=np.int64)
    off = np.ascontiguousarray(off, dtype=np.int64)
    w = np.empty(int(off[-1]), np.uint32)
    lib().orc_kde_weights_many(_p(H), _p(off), len(H), _p(w))
    return w


def kde_root5_many(n: np.ndarray) -> np.ndarray:
    n = np.ascontiguousarray(n, dtype=np.int64)
    out = np.empty(n.size, np.float64)
    lib().orc_kde_root5_many(_p(n), n.size, _p(out))
    return out


def kde_bw_q8_many(var: np.ndarray, n: np.ndarray) -> np.ndarray:
    var = np.ascontiguousarray(var, dtype=np.float64)
    n = np.ascontiguousarray(n, dtype=np.int64)
    out = np.empty(n.size, np.int64)
    lib().orc_kde_bw_q8_many(_p(var), _p(n), n.size, _p(out))
    return out


def kde(ev: dict, n_kernels: int, n_streams: int, n_events: int | None = None, **params) -> dict:
    """Clusters of every (segment, kernel) group of a raw event trace."""
    p = _kde_params(params)
    kid = np.ascontiguousarray(ev["kernel_id"], dtype=np.int32)
    st = np.ascontiguousarray(ev["stream"], dtype=np.int32)
    t0 = np.ascontiguousarray(ev["start_ns"], dtype=np.int64)
    t1 = np.ascontiguousarray(ev["end_ns"], dtype=np.int64)
    off = np.ascontiguousarray(ev["seg_off"], dtype=np.int64)
    G = len(off) - 1
    C = G * n_kernels
    n = len(kid) if n_events is None else n_events
    out = {"n_clusters": np.empty(C, np.uint8), "count": np.empty(C * KDE_MAXC, np.uint32),
           "p50_ns": np.empty(C * KDE_MAXC, np.int64), "p99_ns": np.empty(C * KDE_MAXC, np.int64),
           "bw_q8": np.empty(C, np.int32)}
    bad = lib().orc_kde(G, n_kernels, n_streams, n, _p(kid), _p(st), _p(t0), _p(t1), _p(off), p["sub_bits"],
                        p["frac_pm"], p["min_count"], p["gap"],
                        *[_p(out[k]) for k in ("n_clusters", "count", "p50_ns", "p99_ns", "bw_q8")])
    for k in ("count", "p50_ns", "p99_ns"):
        out[k] = out[k].reshape(C, KDE_MAXC)
    out["bad_segments"] = int(bad)
    return out


def w1(n_clusters, count, p50, p99, R: int, S: int, K: int, **params) -> dict:
    """Cross-rank W1 deviation scores and IQR flags from per-cell clusters
    ([R][S][K] and [R][S][K][KDE_MAXC] arrays). 'malformed' counts cells with
    more than KDE_MAXC clusters or clusters of total count 0 (left out)."""
    p = dict(W1_DEFAULTS, **params)
    C = R * S * K
    ncl = np.ascontiguousarray(n_clusters, dtype=np.uint8).reshape(-1)
    cnt = np.ascontiguousarray(count, dtype=np.uint32).reshape(-1)
    a = np.ascontiguousarray(p50, dtype=np.int64).reshape(-1)
    b = np.ascontiguousarray(p99, dtype=np.int64).reshape(-1)
    assert ncl.size == C and cnt.size == a.size == b.size == C * KDE_MAXC
    SK = S * K
    out = {"n_present": np.empty(SK, np.uint32), "lo_ns": np.empty(SK, np.int64), "hi_ns": np.empty(SK, np.int64),
           "q1": np.empty(SK, np.float64), "q3": np.empty(SK, np.float64), "fence": np.empty(SK, np.float64),
           "n_flag": np.empty(SK, np.uint32), "score": np.empty(C, np.float64), "flag": np.empty(C, np.uint8)}
    bad = lib().orc_w1(R, S, K, _p(ncl), _p(cnt), _p(a), _p(b), p["grid"], p["min_ranks"], p["alpha_pm"],
                       *[_p(out[k]) for k in ("n_present", "lo_ns", "hi_ns", "q1", "q3", "fence", "n_flag", "score",
                                              "flag")])
    out["malformed"] = int(bad)
    return out


def w1_cdf_q(count, p50, p99, x: float) -> int:
    """Fixed-point (16-bit) mixture CDF of one rank's clusters at duration x."""
    cnt = np.ascontiguousarray(count, dtype=np.uint32)
    a = np.ascontiguousarray(p50, dtype=np.int64)
    b = np.ascontiguousarray(p99, dtype=np.int64)
    return lib().orc_w1_cdf_q(len(cnt), _p(cnt), _p(a), _p(b), x)


def w1_cdf_q_grid(count, p50, p99, lo: int, hi: int, g: int, G: int) -> int:
    """The 16-bit mixture CDF of one rank's clusters at grid point g of the
    W1 grid [lo, hi] with G points, u = ln lo + g (ln hi - ln lo) / (G - 1),
    as the oracle's W1 takes it."""
    cnt = np.ascontiguousarray(count, dtype=np.uint32)
    a = np.ascontiguousarray(p50, dtype=np.int64)
    b = np.ascontiguousarray(p99, dtype=np.int64)
    lnlo, lnhi = math.log(float(lo)), math.log(float(hi))
    u = lnlo + float(g) * ((lnhi - lnlo) / float(G - 1))
    return lib().orc_w1_cdf_q_at(len(cnt), _p(cnt), _p(a), _p(b), u)


def l2(count, sum_ns, R: int, S: int, E: int, route, group_off, members, **params) -> dict:
    """Group-aware L2 comparison (CV classes, z-scores, straggler flags) of
    per-(rank, step, event) summaries. route: [E] uint8 dimension per event
    (0xFF: not compared); group_off: [n_dims][max_groups + 1] int32 offsets
    into members: [n_dims][R] int32. 'status': bit 1 malformed groups, 2
    duplicate listings, 4 values out of the 2^40 ns domain."""
    p = dict(L2_DEFAULTS, **params)
    cnt = np.ascontiguousarray(count, dtype=np.uint32).reshape(-1)
    sm = np.ascontiguousarray(sum_ns, dtype=np.int64).reshape(-1)
    rt = np.ascontiguousarray(route, dtype=np.uint8).reshape(-1)
    off = np.ascontiguousarray(group_off, dtype=np.int32)
    mem = np.ascontiguousarray(members, dtype=np.int32)
    n_dims = off.shape[0] if off.ndim == 2 else 0
    max_groups = off.shape[1] - 1 if off.ndim == 2 else 0
    assert cnt.size == sm.size == R * S * E and rt.size == E and mem.size == n_dims * R
    GO = S * E * max_groups
    out = {"n": np.empty(GO, np.uint32), "mean_ns": np.empty(GO, np.float64), "std_ns": np.empty(GO, np.float64),
           "cv": np.empty(GO, np.float64), "cls": np.empty(GO, np.uint8), "n_strag": np.empty(GO, np.uint32),
           "z": np.empty(R * S * E, np.float32), "flags": np.empty(R * S * E, np.uint8)}
    st = lib().orc_l2(R, S, E, _p(cnt), _p(sm), _p(rt), _p(off) if off.size else None,
                      _p(mem) if mem.size else None, n_dims, max_groups, p["min_group"], p["cv_mild_pm"],
                      p["cv_severe_pm"], p["z_pm"],
                      *[_p(out[k]) for k in ("n", "mean_ns", "std_ns", "cv", "cls", "n_strag", "z", "flags")])
    out["status"] = int(st)
    return out
