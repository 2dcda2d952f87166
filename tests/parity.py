"""Helpers for GPU-vs-oracle parity tests.

Expected values always come from the CPU oracle run on host-generated
events; the GPU side runs on device-generated events of the same trace
(byte-identical by construction and checked by checksum).
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

import oracle

NB = 32
SUM_INT_FIELDS = ["count", "sum_ns", "min_ns", "max_ns", "hist", "n_valid", "n_invalid", "t_first", "t_last",
                  "step_ns", "busy_ns", "stream_busy_ns", "wire_bytes"]
XR_INT_FIELDS = ["n_present", "med_ns", "mad_ns", "q1_ns", "q3_ns", "n_flag", "n_degraded", "flags", "score_pm",
                 "n_eval", "n_flag_rank", "straggler"]
XR_FLOAT_FIELDS = ["xmean_ns", "z", "mean_ns"]
L1_INT_FIELDS = ["flags", "cls", "eff_width", "cp"]
L2_INT_FIELDS = ["n", "cls", "n_strag", "flags"]
L2_FLOAT_FIELDS = ["mean_ns", "std_ns", "cv", "z"]
RTOL = 1e-5  # float32 outputs: relative tolerance


def host_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def to_np(t, like=None):
    a = t.detach().cpu().numpy().reshape(-1)
    if like is not None and a.dtype != like.dtype and a.dtype.itemsize == like.dtype.itemsize:
        a = a.view(like.dtype)
    return a


# per-cell summary fields that argus_summarize writes only for present cells
# (count >= 1); the oracle writes identity values for absent ones
PRESENT_ONLY = ("sum_ns", "min_ns", "max_ns", "hist")


def present_rows(ref: dict):
    """Boolean mask of the present cells of an oracle summary."""
    return np.asarray(ref["count"]).reshape(-1) > 0


def assert_int_equal(gpu: dict, ref: dict, fields, what=""):
    """Exact comparison. For a summary (ref has "count"), the present-only
    fields are compared on the present cells, where the count itself has
    already been compared (count is in every summary field list first)."""
    for f in fields:
        r = np.asarray(ref[f]).reshape(-1)
        g = to_np(gpu[f], r)
        if f in PRESENT_ONLY and "count" in ref:
            pres = present_rows(ref)
            per = r.size // pres.size
            keep = np.repeat(pres, per)
            assert g.shape == r.shape, (what, f, g.shape, r.shape)
            r, g = r[keep], g[keep]
        assert g.shape == r.shape, (what, f, g.shape, r.shape)
        if not np.array_equal(g, r):
            bad = np.nonzero(g != r)[0]
            raise AssertionError(f"{what} {f}: {len(bad)} mismatches, first at {bad[:5]}: gpu {g[bad[:5]]} "
                                 f"oracle {r[bad[:5]]}")


def assert_float_close(gpu: dict, ref: dict, fields, what=""):
    for f in fields:
        r = np.asarray(ref[f]).reshape(-1)
        g = to_np(gpu[f], r)
        ok = np.abs(g.astype(np.float64) - r.astype(np.float64)) <= RTOL * np.abs(r.astype(np.float64))
        if not ok.all():
            bad = np.nonzero(~ok)[0]
            raise AssertionError(f"{what} {f}: {len(bad)} beyond rtol {RTOL}, first {bad[:5]}: gpu {g[bad[:5]]} "
                                 f"oracle {r[bad[:5]]}")


def oracle_summary_sharded(trace, g_begin=0, g_end=None, chunk=32, n_threads=None) -> dict:
    """Oracle summaries of segments [g_begin, g_end), regenerated on the host
    chunk by chunk and summarized by the unmodified single-threaded oracle on
    disjoint chunks in parallel (segments are independent). Also returns the
    generator's per-segment checksums of the host events ("checksum")."""
    cfg = trace.cfg
    K, NS = cfg.n_kernels, cfg.n_streams
    g_end = cfg.n_segments if g_end is None else g_end
    G = g_end - g_begin
    n_threads = n_threads or host_threads()
    out = {
        "count": np.empty(G * K, np.uint32), "sum_ns": np.empty(G * K, np.int64),
        "min_ns": np.empty(G * K, np.int64), "max_ns": np.empty(G * K, np.int64),
        "hist": np.empty((G * K, NB), np.uint32),
        "n_valid": np.empty(G, np.uint32), "n_invalid": np.empty(G, np.uint32),
        "t_first": np.empty(G, np.int64), "t_last": np.empty(G, np.int64), "step_ns": np.empty(G, np.int64),
        "busy_ns": np.empty(G, np.int64), "stream_busy_ns": np.empty((G, NS), np.int64),
        "wire_bytes": np.empty(G, np.int64), "checksum": np.empty(G, np.uint64),
    }

    def work(g0):
        g1 = min(g_end, g0 + chunk)
        ev = trace.fill_host(g0, g1, n_threads=1)
        out["checksum"][g0 - g_begin:g1 - g_begin] = trace.checksum_host(ev, g0, g1)
        o = oracle.summarize(ev, K, NS)
        a, b = g0 - g_begin, g1 - g_begin
        for f in ("count", "sum_ns", "min_ns", "max_ns", "hist"):
            out[f][a * K:b * K] = o[f]
        for f in ("n_valid", "n_invalid", "t_first", "t_last", "step_ns", "busy_ns", "stream_busy_ns",
                  "wire_bytes"):
            out[f][a:b] = o[f]

    with ThreadPoolExecutor(n_threads) as ex:
        list(ex.map(work, range(g_begin, g_end, chunk)))
    return out


KDE_FIELDS = ["n_clusters", "count", "p50_ns", "p99_ns", "bw_q8"]


def oracle_kde_segments(trace, segments, n_threads=None, **params) -> dict:
    """Oracle KDE clusters of the listed segments (each regenerated on the
    host and clustered by the unmodified oracle, segments in parallel).
    Returns arrays stacked in the order of `segments`."""
    cfg = trace.cfg
    K = cfg.n_kernels
    segments = list(segments)
    n_threads = n_threads or host_threads()
    out = {"n_clusters": np.empty(len(segments) * K, np.uint8),
           "count": np.empty((len(segments) * K, oracle.KDE_MAXC), np.uint32),
           "p50_ns": np.empty((len(segments) * K, oracle.KDE_MAXC), np.int64),
           "p99_ns": np.empty((len(segments) * K, oracle.KDE_MAXC), np.int64),
           "bw_q8": np.empty(len(segments) * K, np.int32)}

    def work(i):
        g = segments[i]
        ev = trace.fill_host(g, g + 1, n_threads=1)
        o = oracle.kde(ev, K, cfg.n_streams, **params)
        for f in KDE_FIELDS:
            out[f][i * K:(i + 1) * K] = o[f]

    with ThreadPoolExecutor(n_threads) as ex:
        list(ex.map(work, range(len(segments))))
    return out


def assert_kde_equal(gpu: dict, ref: dict, what="", rows=None):
    """Exact comparison of KDE outputs; rows: optional cell indices of the
    GPU arrays that correspond to the reference rows."""
    for f in KDE_FIELDS:
        r = np.asarray(ref[f])
        g = to_np(gpu[f], r)
        if r.ndim == 2:
            g = g.reshape(-1, r.shape[1])
        if rows is not None:
            g = g[rows]
        g = g.reshape(r.shape)
        if not np.array_equal(g, r):
            bad = np.nonzero((g != r).reshape(len(r), -1).any(axis=1))[0]
            raise AssertionError(f"{what} {f}: {len(bad)} cells differ, first {bad[:5]}: gpu {g[bad[:3]]} "
                                 f"oracle {r[bad[:3]]}")
