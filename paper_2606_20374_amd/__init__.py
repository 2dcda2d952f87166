"""MI355X-native hot path of ARGUS (arXiv 2606.20374): kernel-event trace
summarization, kernel-level cross-rank detection and L1 iteration windows,
KDE duration clusters, cross-rank W1 deviation scores and group-aware L2
CV / z-score comparison, as hand-written
gfx950 HIP kernels behind the C ABI of include/argus.h.

The Python layer only marshals arguments; see argus.py.
"""
from .argus import (ArgusError, alloc_cross_rank, alloc_iter_windows, alloc_kde, alloc_l2, alloc_summary, alloc_w1,
                    compact, cross_rank, iter_windows, kde, kde_defaults, kde_workspace_bytes, l1_defaults, l2, l2_defaults,
                    lib, summarize, summarize_noalloc, w1, w1_defaults, xr_defaults)

__all__ = ["ArgusError", "alloc_cross_rank", "alloc_iter_windows", "alloc_kde", "alloc_summary", "cross_rank",
           "iter_windows", "kde", "kde_defaults", "kde_workspace_bytes", "l1_defaults", "lib", "summarize", "summarize_noalloc",
           "xr_defaults", "alloc_w1", "w1", "w1_defaults", "alloc_l2", "l2", "l2_defaults", "compact", "run_step"]


def run_step(ev, n_ranks, n_steps, n_kernels, n_streams, bufs=None):
    """One pass of the whole hot path: summarize, cross-rank, iter windows.
    bufs: optional dict of preallocated outputs {'sum': ..., 'xr': ..., 'l1': ...}."""
    bufs = bufs or {}
    s = summarize(ev, n_ranks, n_steps, n_kernels, n_streams, out=bufs.get("sum"))
    x = cross_rank(s["count"], s["sum_ns"], n_ranks, n_steps, n_kernels, out=bufs.get("xr"))
    w = iter_windows(s["step_ns"], n_ranks, n_steps, out=bufs.get("l1"))
    return s, x, w
