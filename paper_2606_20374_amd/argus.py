"""Thin Python binding of libargus (include/argus.h).

Argument marshalling only: every step of the path runs in the HIP kernels of
libargus.so. PyTorch supplies device memory (torch.empty on the GPU) and the
current stream. There is no CPU fallback: if the library is missing or the
device is not gfx950 the calls raise.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libargus.so")
NBINS = 32

OK, EINVAL, EUNSUPPORTED, EHIP = 0, -1, -2, -3
DEV_BAD_SEGMENT, DEV_L1_DOMAIN, DEV_KDE_SUMMARY, DEV_W1_INPUT = 1, 2, 4, 8
DEV_GROUPS_MALFORMED, DEV_GROUPS_DUPLICATE, DEV_L2_DOMAIN, DEV_COMPACT_CAPACITY = 16, 32, 64, 128
DEV_SUMMARY_STALLED = 256
KDE_MAXC = 4
MAX_W1_STEPS = 65535
NOALLOC_SCRATCH_BYTES = 256

V, I32, I64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64


class Events(ctypes.Structure):
    _fields_ = [("kernel_id", V), ("stream", V), ("start_ns", V), ("end_ns", V), ("seg_off", V),
                ("n_events", I64), ("n_ranks", I32), ("n_steps", I32), ("n_kernels", I32), ("n_streams", I32)]


SUMMARY_FIELDS = ["count", "sum_ns", "min_ns", "max_ns", "hist", "n_valid", "n_invalid", "t_first", "t_last",
                  "step_ns", "busy_ns", "stream_busy_ns", "wire_bytes", "dev_status"]


class Summary(ctypes.Structure):
    _fields_ = [(f, V) for f in SUMMARY_FIELDS]


class XrParams(ctypes.Structure):
    _fields_ = [(f, I32) for f in ("min_ranks", "c_min_pair", "min_kernels", "k_mad_pm", "ratio_pm", "alpha_pm",
                                   "tau_rank_pm")]


XR_FIELDS = ["n_present", "med_ns", "mad_ns", "q1_ns", "q3_ns", "xmean_ns", "n_flag", "n_degraded", "z", "mean_ns",
             "flags", "score_pm", "n_eval", "n_flag_rank", "straggler", "dev_status"]


class XrOut(ctypes.Structure):
    _fields_ = [(f, V) for f in XR_FIELDS]


class L1Params(ctypes.Structure):
    _fields_ = [(f, I32) for f in ("W", "theta_pm", "beta_pm", "rho_pm", "cmax_pm", "min_seg")]


class KdeParams(ctypes.Structure):
    _fields_ = [(f, I32) for f in ("sub_bits", "frac_pm", "min_count", "gap")]


KDE_FIELDS = ["n_clusters", "count", "p50_ns", "p99_ns", "bw_q8", "dev_status"]


class KdeOut(ctypes.Structure):
    _fields_ = [(f, V) for f in KDE_FIELDS]


class W1Params(ctypes.Structure):
    _fields_ = [(f, I32) for f in ("grid", "min_ranks", "alpha_pm")]


W1_FIELDS = ["n_present", "lo_ns", "hi_ns", "q1", "q3", "fence", "n_flag", "score", "flag", "dev_status"]


class W1Out(ctypes.Structure):
    _fields_ = [(f, V) for f in W1_FIELDS]


class L2Params(ctypes.Structure):
    _fields_ = [(f, I32) for f in ("min_group", "cv_mild_pm", "cv_severe_pm", "z_pm")]


class Groups(ctypes.Structure):
    _fields_ = [("route", V), ("group_off", V), ("members", V), ("n_dims", I32), ("max_groups", I32)]


L2_FIELDS = ["n", "mean_ns", "std_ns", "cv", "cls", "n_strag", "z", "flags", "dev_status"]


class L2Out(ctypes.Structure):
    _fields_ = [(f, V) for f in L2_FIELDS]


class ArgusError(RuntimeError):
    pass


_lib = None


def lib():
    """Load libargus.so; raises if it is not built (no fallback path exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ArgusError(f"{LIB_PATH} is missing: build it with __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.POINTER
        L.argus_abi_version.restype = ctypes.c_int
        L.argus_status_string.argtypes = [ctypes.c_int]
        L.argus_status_string.restype = ctypes.c_char_p
        L.argus_summarize_workspace.argtypes = [P(Events)]
        L.argus_summarize_workspace.restype = ctypes.c_size_t
        L.argus_summarize.argtypes = [P(Events), P(Summary), V, ctypes.c_size_t, V]
        L.argus_summarize.restype = ctypes.c_int
        L.argus_summarize_keyed.argtypes = [P(Events), P(Summary), V, ctypes.c_size_t, V]
        L.argus_summarize_noalloc.argtypes = [P(Events), P(Summary), V]
        L.argus_summarize_noalloc.restype = ctypes.c_int
        L.argus_summarize_keyed.restype = ctypes.c_int
        L.argus_compact_workspace.argtypes = [I32, I32]
        L.argus_compact_workspace.restype = ctypes.c_size_t
        L.argus_compact.argtypes = [P(Summary), I32, I32, I32, I32, V, I64, V, V, V, ctypes.c_size_t, V]
        L.argus_compact.restype = ctypes.c_int
        L.argus_xr_default.argtypes = [P(XrParams)]
        L.argus_cross_rank_workspace.argtypes = [I32, I32, I32]
        L.argus_cross_rank_workspace.restype = ctypes.c_size_t
        L.argus_cross_rank.argtypes = [V, V, I32, I32, I32, P(XrParams), P(XrOut), V, ctypes.c_size_t, V]
        L.argus_cross_rank.restype = ctypes.c_int
        L.argus_l1_default.argtypes = [P(L1Params)]
        L.argus_iter_windows_workspace.argtypes = [I32, I32]
        L.argus_iter_windows_workspace.restype = ctypes.c_size_t
        L.argus_iter_windows.argtypes = [V, I32, I32, P(L1Params), V, V, V, V, V, V, V, ctypes.c_size_t, V]
        L.argus_iter_windows.restype = ctypes.c_int
        L.argus_kde_default.argtypes = [P(KdeParams)]
        L.argus_kde_workspace.argtypes = [P(Events)]
        L.argus_kde_workspace.restype = ctypes.c_size_t
        L.argus_kde.argtypes = [P(Events), P(Summary), P(KdeParams), P(KdeOut), V, ctypes.c_size_t, V]
        L.argus_kde.restype = ctypes.c_int
        L.argus_w1_default.argtypes = [P(W1Params)]
        L.argus_w1_workspace.argtypes = [I32, I32, I32, I32]
        L.argus_w1_workspace.restype = ctypes.c_size_t
        L.argus_w1.argtypes = [P(KdeOut), I32, I32, I32, P(W1Params), P(W1Out), V, ctypes.c_size_t, V]
        L.argus_w1.restype = ctypes.c_int
        L.argus_l2_default.argtypes = [P(L2Params)]
        L.argus_l2_workspace.argtypes = [I32, I32]
        L.argus_l2_workspace.restype = ctypes.c_size_t
        L.argus_l2.argtypes = [V, V, I32, I32, I32, P(Groups), P(L2Params), P(L2Out), V, ctypes.c_size_t, V]
        L.argus_l2.restype = ctypes.c_int
        if L.argus_abi_version() != 1:
            raise ArgusError("libargus ABI version mismatch")
        _lib = L
    return _lib


def _check(rc: int, what: str):
    if rc != OK:
        raise ArgusError(f"{what}: {lib().argus_status_string(rc).decode()} ({rc})")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    assert t.is_cuda and t.is_contiguous(), "libargus takes contiguous device tensors"
    return t.data_ptr()


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def xr_defaults() -> dict:
    p = XrParams()
    lib().argus_xr_default(ctypes.byref(p))
    return {f: getattr(p, f) for f, _ in XrParams._fields_}


def l1_defaults() -> dict:
    p = L1Params()
    lib().argus_l1_default(ctypes.byref(p))
    return {f: getattr(p, f) for f, _ in L1Params._fields_}


def kde_defaults() -> dict:
    p = KdeParams()
    lib().argus_kde_default(ctypes.byref(p))
    return {f: getattr(p, f) for f, _ in KdeParams._fields_}


def w1_defaults() -> dict:
    p = W1Params()
    lib().argus_w1_default(ctypes.byref(p))
    return {f: getattr(p, f) for f, _ in W1Params._fields_}


def l2_defaults() -> dict:
    p = L2Params()
    lib().argus_l2_default(ctypes.byref(p))
    return {f: getattr(p, f) for f, _ in L2Params._fields_}


def _events(ev: dict, n_ranks: int, n_steps: int, n_kernels: int, n_streams: int) -> Events:
    return Events(_ptr(ev["kernel_id"]), _ptr(ev["stream"]), _ptr(ev["start_ns"]), _ptr(ev["end_ns"]),
                  _ptr(ev["seg_off"]), ev["kernel_id"].numel(), n_ranks, n_steps, n_kernels, n_streams)


# ------------------------------------------------------------------ summarize
def alloc_summary(n_ranks: int, n_steps: int, n_kernels: int, n_streams: int, device="cuda") -> dict:
    G, C = n_ranks * n_steps, n_ranks * n_steps * n_kernels
    e = lambda n, dt: torch.empty(n, dtype=dt, device=device)  # noqa: E731
    return {
        "count": e(C, torch.int32), "sum_ns": e(C, torch.int64), "min_ns": e(C, torch.int64),
        "max_ns": e(C, torch.int64), "hist": e(C * NBINS, torch.int32),
        "n_valid": e(G, torch.int32), "n_invalid": e(G, torch.int32), "t_first": e(G, torch.int64),
        "t_last": e(G, torch.int64), "step_ns": e(G, torch.int64), "busy_ns": e(G, torch.int64),
        "stream_busy_ns": e(G * n_streams, torch.int64), "wire_bytes": e(G, torch.int64),
        "dev_status": e(1, torch.int32), "_workspace": e(256, torch.uint8),
    }


def summarize(ev: dict, n_ranks: int, n_steps: int, n_kernels: int, n_streams: int,
              out: Optional[dict] = None, keyed: bool = False) -> dict:
    """argus_summarize (keyed: argus_summarize_keyed, cells per (kernel,
    stream)) over SoA device tensors ev = {kernel_id, stream, start_ns,
    end_ns, seg_off}. Unsigned outputs are returned in signed torch dtypes of
    the same width (reinterpret with .view on the host)."""
    dev = ev["kernel_id"].device
    if out is None:
        out = alloc_summary(n_ranks, n_steps, n_kernels * (n_streams if keyed else 1), n_streams, dev)
    e = _events(ev, n_ranks, n_steps, n_kernels, n_streams)
    s = Summary(*[_ptr(out.get(f)) for f in SUMMARY_FIELDS])
    ws = out["_workspace"]
    assert ws.numel() >= lib().argus_summarize_workspace(ctypes.byref(e))
    fn = lib().argus_summarize_keyed if keyed else lib().argus_summarize
    _check(fn(ctypes.byref(e), ctypes.byref(s), _ptr(ws), ws.numel(), _stream(dev)), "argus_summarize")
    return out


def summarize_noalloc(ev: dict, n_ranks: int, n_steps: int, n_kernels: int, n_streams: int,
                      out: Optional[dict] = None) -> dict:
    """argus_summarize_noalloc: argus_summarize with its scratch in the
    library's static per-device array (no workspace argument)."""
    dev = ev["kernel_id"].device
    if out is None:
        out = alloc_summary(n_ranks, n_steps, n_kernels, n_streams, dev)
    e = _events(ev, n_ranks, n_steps, n_kernels, n_streams)
    s = Summary(*[_ptr(out.get(f)) for f in SUMMARY_FIELDS])
    _check(lib().argus_summarize_noalloc(ctypes.byref(e), ctypes.byref(s), _stream(dev)), "argus_summarize_noalloc")
    return out


def compact(summary: dict, n_ranks: int, n_steps: int, n_cells: int, n_streams: int = 0,
            capacity: Optional[int] = None, out: Optional[torch.Tensor] = None) -> dict:
    """argus_compact: the record stream of a dense summary (n_streams = 0 for
    kernel-id keys, else the stream count of (kernel, stream) keys). With no
    capacity the stream is sized by a first call (one host synchronisation)."""
    dev = summary["count"].device
    G = n_ranks * n_steps
    seg = torch.empty(G + 1, dtype=torch.int64, device=dev)
    status = torch.empty(1, dtype=torch.int32, device=dev)
    ws = torch.empty(max(lib().argus_compact_workspace(n_ranks, n_steps), 8), dtype=torch.uint8, device=dev)
    sm = Summary(*[_ptr(summary.get(f)) if f in ("count", "sum_ns", "min_ns", "max_ns", "hist") else None
                   for f in SUMMARY_FIELDS])

    def call(buf, cap):
        _check(lib().argus_compact(ctypes.byref(sm), n_ranks, n_steps, n_cells, n_streams,
                                   None if buf is None else _ptr(buf), cap, _ptr(seg), _ptr(status), _ptr(ws),
                                   ws.numel(), _stream(dev)), "argus_compact")

    if out is None:
        if capacity is None:
            call(None, 0)
            capacity = int(seg[-1].item())
        out = torch.empty(max(capacity, 1), dtype=torch.uint8, device=dev)
    cap = out.numel() if capacity is None else capacity
    call(out, cap)
    return {"bytes": out, "seg_byte_off": seg, "dev_status": status, "capacity": cap}


# ----------------------------------------------------------------- cross-rank
def alloc_cross_rank(n_ranks: int, n_steps: int, n_kernels: int, device="cuda") -> dict:
    SK, C, RS = n_steps * n_kernels, n_ranks * n_steps * n_kernels, n_ranks * n_steps
    e = lambda n, dt: torch.empty(n, dtype=dt, device=device)  # noqa: E731
    ws = lib().argus_cross_rank_workspace(n_ranks, n_steps, n_kernels)
    return {
        "n_present": e(SK, torch.int32), "med_ns": e(SK, torch.int64), "mad_ns": e(SK, torch.int64),
        "q1_ns": e(SK, torch.int64), "q3_ns": e(SK, torch.int64), "xmean_ns": e(SK, torch.float32),
        "n_flag": e(SK, torch.int32), "n_degraded": e(SK, torch.int32),
        "z": e(C, torch.float32), "mean_ns": e(C, torch.float32), "flags": e(C, torch.uint8),
        "score_pm": e(RS, torch.int32), "n_eval": e(RS, torch.int32), "n_flag_rank": e(RS, torch.int32),
        "straggler": e(RS, torch.uint8), "dev_status": e(1, torch.int32),
        "_workspace": e(max(ws, 1), torch.uint8),
    }


def cross_rank(count: torch.Tensor, sum_ns: torch.Tensor, n_ranks: int, n_steps: int, n_kernels: int,
               out: Optional[dict] = None, **params) -> dict:
    dev = count.device
    if out is None:
        out = alloc_cross_rank(n_ranks, n_steps, n_kernels, dev)
    p = XrParams()
    lib().argus_xr_default(ctypes.byref(p))
    for k, v in params.items():
        setattr(p, k, v)
    o = XrOut(*[_ptr(out.get(f)) for f in XR_FIELDS])
    ws = out["_workspace"]
    _check(lib().argus_cross_rank(_ptr(count), _ptr(sum_ns), n_ranks, n_steps, n_kernels, ctypes.byref(p),
                                  ctypes.byref(o), _ptr(ws), ws.numel(), _stream(dev)), "argus_cross_rank")
    return out


# --------------------------------------------------------------- iter windows
def alloc_iter_windows(n_ranks: int, n_steps: int, device="cuda") -> dict:
    e = lambda n, dt: torch.empty(n, dtype=dt, device=device)  # noqa: E731
    return {"flags": e(max(n_ranks * n_steps, 1), torch.uint8), "cls": e(max(n_ranks, 1), torch.uint8),
            "eff_width": e(max(n_ranks, 1), torch.int32), "cp": e(max(n_ranks, 1), torch.int32),
            "cp_ratio": e(max(n_ranks, 1), torch.float32), "dev_status": e(1, torch.int32)}


def iter_windows(step_ns: torch.Tensor, n_ranks: int, n_steps: int, out: Optional[dict] = None, **params) -> dict:
    dev = step_ns.device
    if out is None:
        out = alloc_iter_windows(n_ranks, n_steps, dev)
    p = L1Params()
    lib().argus_l1_default(ctypes.byref(p))
    for k, v in params.items():
        setattr(p, k, v)
    _check(lib().argus_iter_windows(_ptr(step_ns), n_ranks, n_steps, ctypes.byref(p), _ptr(out["flags"]),
                                    _ptr(out["cls"]), _ptr(out["eff_width"]), _ptr(out["cp"]),
                                    _ptr(out["cp_ratio"]), _ptr(out["dev_status"]), None, 0, _stream(dev)),
           "argus_iter_windows")
    return out


# ------------------------------------------------------------------------ KDE
def kde_workspace_bytes(n_events: int, n_ranks: int, n_steps: int, n_kernels: int) -> int:
    e = Events(0, 0, 0, 0, 0, n_events, n_ranks, n_steps, n_kernels, 1)
    return lib().argus_kde_workspace(ctypes.byref(e))


def alloc_kde(n_events: int, n_ranks: int, n_steps: int, n_kernels: int, device="cuda") -> dict:
    C = n_ranks * n_steps * n_kernels
    e = lambda n, dt: torch.empty(n, dtype=dt, device=device)  # noqa: E731
    ws = kde_workspace_bytes(n_events, n_ranks, n_steps, n_kernels)
    return {"n_clusters": e(C, torch.uint8), "count": e(C * KDE_MAXC, torch.int32),
            "p50_ns": e(C * KDE_MAXC, torch.int64), "p99_ns": e(C * KDE_MAXC, torch.int64),
            "bw_q8": e(C, torch.int32), "dev_status": e(1, torch.int32),
            "_workspace": e(max(ws, 256), torch.uint8)}


def kde(ev: dict, summary: dict, n_ranks: int, n_steps: int, n_kernels: int, n_streams: int,
        out: Optional[dict] = None, **params) -> dict:
    """argus_kde: per-cell duration clusters (n_clusters, count, p50_ns,
    p99_ns, bw_q8) from the events and their argus_summarize output."""
    dev = ev["kernel_id"].device
    if out is None:
        out = alloc_kde(ev["kernel_id"].numel(), n_ranks, n_steps, n_kernels, dev)
    p = KdeParams()
    lib().argus_kde_default(ctypes.byref(p))
    for k, v in params.items():
        setattr(p, k, v)
    e = _events(ev, n_ranks, n_steps, n_kernels, n_streams)
    s = Summary(*[_ptr(summary.get(f)) if f in ("count", "min_ns", "max_ns", "n_invalid") else None
                  for f in SUMMARY_FIELDS])
    o = KdeOut(*[_ptr(out.get(f)) for f in KDE_FIELDS])
    ws = out["_workspace"]
    _check(lib().argus_kde(ctypes.byref(e), ctypes.byref(s), ctypes.byref(p), ctypes.byref(o), _ptr(ws),
                           ws.numel(), _stream(dev)), "argus_kde")
    return out


# ------------------------------------------------------------------------- W1
def alloc_w1(n_ranks: int, n_steps: int, n_kernels: int, grid: int = 64, device="cuda") -> dict:
    SK, C = n_steps * n_kernels, n_ranks * n_steps * n_kernels
    e = lambda n, dt: torch.empty(n, dtype=dt, device=device)  # noqa: E731
    ws = lib().argus_w1_workspace(n_ranks, n_steps, n_kernels, grid)
    return {"n_present": e(SK, torch.int32), "lo_ns": e(SK, torch.int64), "hi_ns": e(SK, torch.int64),
            "q1": e(SK, torch.float64), "q3": e(SK, torch.float64), "fence": e(SK, torch.float64),
            "n_flag": e(SK, torch.int32), "score": e(C, torch.float64), "flag": e(C, torch.uint8),
            "dev_status": e(1, torch.int32), "_workspace": e(max(ws, 256), torch.uint8), "_grid": grid}


def w1(clusters: dict, n_ranks: int, n_steps: int, n_kernels: int, out: Optional[dict] = None, **params) -> dict:
    """argus_w1: cross-rank W1 deviation scores and IQR flags per (step,
    kernel) from per-cell clusters (the n_clusters, count, p50_ns and p99_ns
    tensors of an argus_kde output)."""
    dev = clusters["n_clusters"].device
    p = W1Params()
    lib().argus_w1_default(ctypes.byref(p))
    for k, v in params.items():
        setattr(p, k, v)
    if out is None:
        out = alloc_w1(n_ranks, n_steps, n_kernels, p.grid, dev)
    cl = KdeOut(*[_ptr(clusters.get(f)) if f in ("n_clusters", "count", "p50_ns", "p99_ns") else None
                  for f in KDE_FIELDS])
    o = W1Out(*[_ptr(out.get(f)) for f in W1_FIELDS])
    ws = out["_workspace"]
    _check(lib().argus_w1(ctypes.byref(cl), n_ranks, n_steps, n_kernels, ctypes.byref(p), ctypes.byref(o), _ptr(ws),
                          ws.numel(), _stream(dev)), "argus_w1")
    return out


# ------------------------------------------------------------------------- L2
def alloc_l2(n_ranks: int, n_steps: int, n_events: int, n_dims: int, max_groups: int, device="cuda") -> dict:
    GO, C = n_steps * n_events * max_groups, n_ranks * n_steps * n_events
    e = lambda n, dt: torch.empty(n, dtype=dt, device=device)  # noqa: E731
    ws = lib().argus_l2_workspace(n_ranks, n_dims)
    return {"n": e(GO, torch.int32), "mean_ns": e(GO, torch.float64), "std_ns": e(GO, torch.float64),
            "cv": e(GO, torch.float64), "cls": e(GO, torch.uint8), "n_strag": e(GO, torch.int32),
            "z": e(C, torch.float32), "flags": e(C, torch.uint8), "dev_status": e(1, torch.int32),
            "_workspace": e(max(ws, 4), torch.uint8)}


def l2(count: torch.Tensor, sum_ns: torch.Tensor, n_ranks: int, n_steps: int, n_events: int, route: torch.Tensor,
       group_off: torch.Tensor, members: torch.Tensor, out: Optional[dict] = None, **params) -> dict:
    """argus_l2: group-aware CV classes and z-score straggler flags. route
    [n_events] uint8, group_off [n_dims][max_groups + 1] int32, members
    [n_dims][n_ranks] int32 (device tensors)."""
    dev = count.device
    n_dims, max_groups = group_off.shape[0], group_off.shape[1] - 1
    if out is None:
        out = alloc_l2(n_ranks, n_steps, n_events, n_dims, max_groups, dev)
    p = L2Params()
    lib().argus_l2_default(ctypes.byref(p))
    for k, v in params.items():
        setattr(p, k, v)
    g = Groups(_ptr(route), _ptr(group_off), _ptr(members), n_dims, max_groups)
    o = L2Out(*[_ptr(out.get(f)) for f in L2_FIELDS])
    ws = out["_workspace"]
    _check(lib().argus_l2(_ptr(count), _ptr(sum_ns), n_ranks, n_steps, n_events, ctypes.byref(g), ctypes.byref(p),
                          ctypes.byref(o), _ptr(ws), ws.numel(), _stream(dev)), "argus_l2")
    return out
