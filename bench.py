"""Benchmark: one step of the ARGUS hot path on a whole simulated cluster.

A step is one pass of summarize (raw events -> per (rank, step, kernel)
summaries), cross-rank detection and L1 iteration windows over one resident
batch of synthetic events. The default workload is the cluster-scale step:
10,240 ranks x 400,000 kernel events (4.1e9 events, 98.3 GB of
structure-of-arrays input resident in HBM), 2,048 kernel ids, 16 streams.

Prints one JSON line. Timing uses HIP events on the stream the kernels run
on; the summarize kernel is also timed on its own for the roofline figure.
The CPU oracle is timed on a bounded sample of the same workload on the
host (single thread), and the GPU summaries of that sample are checked
against it before the line is printed.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
NB = 32

WORKLOADS = {
    "cluster": "cluster step: 10240 ranks x 1 step x 400000 events, 2048 kernel ids (Zipf 1.1), 16 streams, "
               "5% per-rank reordering, 10 stragglers, 50 degraded pairs",
    "production": "production step: 1024 ranks x 1 step x 400000 events, 2048 kernel ids, 16 streams",
    "medium": "medium: 256 ranks x 8 steps x 100000 events, 512 kernel ids, 8 streams",
    "skew": "skew: 4096 ranks x 4 steps x 200000 events, 8 hot Pareto ids + 8192 cold ids, 16 streams",
    "tiny": "tiny: 8 ranks x 4 steps x 20000 events, 64 kernel ids, 4 streams",
}


def algorithmic_summarize_bytes(n_events: int, present_cells: int, n_seg: int, n_streams: int) -> int:
    # read every event once (24 B: kid 4, stream 4, start 8, end 8); write each
    # present cell once (count 4, sum 8, min 8, max 8, hist 128 = 156 B) and
    # each rank-step's aggregates (48 B + 8 B per stream)
    return 24 * n_events + 156 * present_cells + (48 + 8 * n_streams) * n_seg


def measured_traffic(config: str):
    """HBM bytes per summarize launch from the committed rocprofv3 counter
    summary, or None when the kernel source changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"summarize_{config}.md")
    src = os.path.join(ROOT, "paper_2606_20374_amd", "csrc", "summarize.hip")
    if not os.path.exists(path):
        return None
    sha, traffic = None, None
    for line in open(path):
        if line.startswith("kernel-source:"):
            sha = line.split()[-1]
        elif line.startswith("traffic_bytes_per_launch:"):
            traffic = int(line.split()[-1])
    cur = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
    return traffic if sha == cur else None


def host_record() -> dict:
    """The host the CPU baselines ran on: usable cores, CPU model, RAM."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    ram = None
    try:
        for line in open("/proc/meminfo"):
            if line.startswith("MemTotal:"):
                ram = round(int(line.split()[1]) * 1024 / 2**30, 1)
                break
    except OSError:
        pass
    return {"nproc": len(os.sched_getaffinity(0)), "cpu_count": os.cpu_count(), "cpu_model": model,
            "ram_gib": ram}


class pinned_to_one_core:
    """Pins the calling thread to one of its allowed cores for the duration
    of a with-block (in-process; the oracle runs in the calling thread)."""

    def __enter__(self):
        self.old = os.sched_getaffinity(0)
        self.core = max(self.old)
        os.sched_setaffinity(0, {self.core})
        return self

    def __exit__(self, *exc):
        os.sched_setaffinity(0, self.old)


def cpu_baseline(trace, sample_ranks: int, gpu_sum: dict) -> dict:
    """Oracle (single-threaded, as it stands, pinned to one core) on the
    first sample_ranks ranks of the same workload; also checks the GPU
    summaries of those ranks."""
    import oracle
    cfg = trace.cfg
    K, NS, S = cfg.n_kernels, cfg.n_streams, cfg.n_steps
    g_end = sample_ranks * S
    chunk = max(S, 64 // S * S)
    t_oracle = 0.0
    counts, sums, steps = [], [], []
    n_ev = 0
    mismatches = 0
    for g0 in range(0, g_end, chunk):
        g1 = min(g_end, g0 + chunk)
        ev = trace.fill_host(g0, g1, n_threads=os.cpu_count() or 1)
        n_ev += len(ev["kernel_id"])
        with pinned_to_one_core() as pin:
            t0 = time.perf_counter()
            o = oracle.summarize(ev, K, NS)
            t_oracle += time.perf_counter() - t0
        pres = np.asarray(o["count"]).reshape(-1) > 0
        for f in ("count", "sum_ns", "min_ns", "max_ns", "hist"):
            per = NB if f == "hist" else 1
            ref = np.asarray(o[f]).reshape(-1)
            got = gpu_sum[f][g0 * K * per:g1 * K * per].view(ref.dtype)
            if f != "count":  # argus_summarize writes these for present cells only
                keep = np.repeat(pres, per)
                ref, got = ref[keep], got[keep]
            mismatches += int(np.count_nonzero(got != ref))
        for f in ("n_valid", "n_invalid", "step_ns", "busy_ns"):
            ref = np.asarray(o[f]).reshape(-1)
            mismatches += int(np.count_nonzero(gpu_sum[f][g0:g1].view(ref.dtype) != ref))
        counts.append(o["count"])
        sums.append(o["sum_ns"])
        steps.append(o["step_ns"])
    cnt, sm, st = np.concatenate(counts), np.concatenate(sums), np.concatenate(steps)
    with pinned_to_one_core() as pin:
        t0 = time.perf_counter()
        oracle.cross_rank(cnt, sm, sample_ranks, S, K)
        oracle.iter_windows(st, sample_ranks, S)
        t_oracle += time.perf_counter() - t0
    return {"value": n_ev / t_oracle, "unit": "events/s", "cores": 1, "kind": "oracle",
            "sample": f"first {sample_ranks} ranks of the same workload ({n_ev} events): oracle summarize + "
                      f"cross-rank + iter windows over the sample, single thread pinned to core {pin.core}, "
                      f"generation excluded",
            "seconds": round(t_oracle, 3), "host": host_record(), "_mismatches": mismatches}


def cpu_baseline_sharded(trace, n_workers: int, seg_per_shard: int = 64) -> dict:
    """The same single-threaded oracle summarize, unmodified, run on disjoint
    segment shards in n_workers threads at once (ctypes releases the GIL
    during each call); shards are generated beforehand, outside the timing."""
    import oracle
    from concurrent.futures import ThreadPoolExecutor
    cfg = trace.cfg
    G = cfg.n_ranks * cfg.n_steps
    n = max(1, min(n_workers, G // seg_per_shard))
    shards = [trace.fill_host(i * seg_per_shard, (i + 1) * seg_per_shard, n_threads=os.cpu_count() or 1)
              for i in range(n)]
    n_ev = sum(len(e["kernel_id"]) for e in shards)
    with ThreadPoolExecutor(max_workers=n) as ex:
        list(ex.map(lambda e: oracle.summarize(e, cfg.n_kernels, cfg.n_streams), shards[:1]))  # warm-up
        t0 = time.perf_counter()
        list(ex.map(lambda e: oracle.summarize(e, cfg.n_kernels, cfg.n_streams), shards))
        dt = time.perf_counter() - t0
    return {"value": n_ev / dt, "unit": "events/s", "cores": n, "kind": "oracle",
            "sample": f"{n} disjoint shards of {seg_per_shard} rank-steps ({n_ev} events) of the same workload, "
                      f"oracle summarize on each shard in its own thread at once, generation excluded",
            "seconds": round(dt, 3), "host": host_record()}


def timed_calls(fn, reps: int, stream) -> list:
    """Per-call times (ms) of reps back-to-back calls, from HIP events
    recorded on the stream the calls launch on."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
    ev[0].record(stream)
    for i in range(reps):
        fn()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    return [ev[i].elapsed_time(ev[i + 1]) for i in range(reps)]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="cluster", choices=sorted(WORKLOADS))
    ap.add_argument("--cpu-sample-ranks", type=int, default=2560)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES bytes (counter calibration)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kde-reps", type=int, default=5, help="timed argus_kde calls (0: skip the KDE and W1 legs)")
    ap.add_argument("--w1-reps", type=int, default=5, help="timed argus_w1 calls (0: skip the W1 leg)")
    ap.add_argument("--l2-reps", type=int, default=5, help="timed argus_l2 calls (0: skip the L2 leg)")
    ap.add_argument("--compact-reps", type=int, default=5, help="timed argus_compact calls (0: skip that leg)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only: libargus has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2606_20374_amd as pa
    import tracegen

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration:
        # a plain copy of known size: reads and writes exactly BYTES each,
        # the reference for scaling FETCH_SIZE / WRITE_SIZE counters
        n = args.copy_calibration // 8
        src = torch.ones(n, dtype=torch.int64, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n * 8}))
        return
    trace = tracegen.make(args.config)
    cfg = trace.cfg
    R, S, K, NS = cfg.n_ranks, cfg.n_steps, cfg.n_kernels, cfg.n_streams
    G = R * S
    print(f"[bench] workload {args.config}: {trace.n_events} events, generating on device", file=sys.stderr,
          flush=True)
    ev = trace.fill_device(device=dev)
    torch.cuda.synchronize()
    cs_dev = trace.checksum_device(ev, 0, min(G, 64))
    bufs = {"sum": pa.alloc_summary(R, S, K, NS, dev), "xr": pa.alloc_cross_rank(R, S, K, dev),
            "l1": pa.alloc_iter_windows(R, S, dev)}
    stream = torch.cuda.current_stream(dev)

    def step(ev_marks=None):
        if ev_marks:
            ev_marks[0].record(stream)
        s = pa.summarize(ev, R, S, K, NS, out=bufs["sum"])
        if ev_marks:
            ev_marks[1].record(stream)
        pa.cross_rank(s["count"], s["sum_ns"], R, S, K, out=bufs["xr"])
        if ev_marks:
            ev_marks[2].record(stream)
        pa.iter_windows(s["step_ns"], R, S, out=bufs["l1"])
        if ev_marks:
            ev_marks[3].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] warmup done, timing {args.steps} steps", file=sys.stderr, flush=True)

    marks = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(args.steps):
        step(marks[i])
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_per_step = total_ms / args.steps
    sum_ms = [m[0].elapsed_time(m[1]) for m in marks]
    xr_ms = [m[1].elapsed_time(m[2]) for m in marks]
    l1_ms = [m[2].elapsed_time(m[3]) for m in marks]

    s, x = bufs["sum"], bufs["xr"]
    count_h = s["count"].cpu().numpy().view(np.uint32)
    present = int(np.count_nonzero(count_h))
    alg_bytes = algorithmic_summarize_bytes(trace.n_events, present, G, NS)
    sum_avg_ms = float(np.mean(sum_ms))
    sum_med_ms = float(np.median(sum_ms))
    achieved = alg_bytes / (sum_avg_ms * 1e-3) / 1e9
    assert int(s["dev_status"].item()) == 0

    # detection outcome against the planted ground truth
    truth = trace.truth()
    strag = x["straggler"].cpu().numpy().reshape(R, S)
    flags = x["flags"].cpu().numpy().reshape(R, S, K)
    strag_ok = all(set(np.nonzero(strag[:, t])[0].tolist()) == truth["stragglers"] for t in range(S))
    pairs_ok = all({(int(r), int(k)) for r, k in zip(*np.nonzero(flags[:, t, :] & 8))} == truth["pairs"]
                   for t in range(S))

    result = {
        "metric": "kernel events summarized/sec + % of HBM peak; cross-rank detect ms/step",
        "value": trace.n_events / (ms_per_step * 1e-3),
        "unit": "events/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "int64", "data": "synthetic (seeded counter-based generator, resident in HBM)",
        "config": {"workload": WORKLOADS[args.config], "n_ranks": R, "n_steps": S, "events": trace.n_events,
                   "n_kernels": K, "n_streams": NS, "input_bytes": 24 * trace.n_events},
        "ms_per_step_median": float(np.median([a + b + c for a, b, c in zip(sum_ms, xr_ms, l1_ms)])),
        "summarize_ms": sum_avg_ms,
        "summarize_ms_median": sum_med_ms,
        "summarize_events_per_s": trace.n_events / (sum_avg_ms * 1e-3),
        "hbm_frac_summarize": achieved / HBM_PEAK_GBS,
        "hbm_frac_summarize_median": alg_bytes / (sum_med_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "cross_rank_ms_per_step": float(np.mean(xr_ms)) / S,
        "cross_rank_ms_per_step_median": float(np.median(xr_ms)) / S,
        "iter_windows_ms": float(np.mean(l1_ms)),
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": measured_traffic(args.config),
                     "kernel": "summarize_kernel", "algorithmic_bytes_per_launch": alg_bytes},
        "detection": {"stragglers_recovered": strag_ok, "pairs_recovered": pairs_ok,
                      "n_flagged_ranks": int(strag.sum())},
    }
    # L1 iteration windows on a long series: 10,240 ranks x 1,000 steps of
    # step times (seeded: 4% noise, a 1.5x regression on every 7th rank from
    # step 600, a 3x spike on every 11th rank at step 300)
    y = tracegen.l1_series(10_240, 1000)
    y_d = torch.from_numpy(y.reshape(-1)).to(dev)
    l1_out = pa.alloc_iter_windows(10_240, 1000, dev)
    for _ in range(2):
        pa.iter_windows(y_d, 10_240, 1000, out=l1_out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(5):
        pa.iter_windows(y_d, 10_240, 1000, out=l1_out)
    e1.record(stream)
    torch.cuda.synchronize()
    result["iter_windows_10240x1000_ms"] = e0.elapsed_time(e1) / 5

    if args.compact_reps > 0:
        # the uploaded record stream of the step's summaries (section 5.2,
        # sizes of section 8.3): sized once, then timed into a preallocated
        # buffer
        comp = pa.compact(s, R, S, K, 0)
        total = int(comp["seg_byte_off"][-1].item())
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.compact_reps):
            pa.compact(s, R, S, K, 0, out=comp["bytes"])
        e1.record(stream)
        torch.cuda.synchronize()
        c_ms = e0.elapsed_time(e1) / args.compact_reps
        assert int(comp["dev_status"].item()) == 0
        # read: count of every cell, hist of the present ones, sum / min /
        # max of the present ones (twice: sizing and writing); written: the
        # records and the segment offsets
        c_bytes = 4 * G * K * 2 + present * (128 * 2 + 24) + total + 16 * G
        result["compact"] = {
            "ms": c_ms, "bytes": total, "bytes_per_rank_step": total / G,
            "raw_bytes_per_rank_step": 24 * trace.n_events / G,
            "compression_ratio": 24 * trace.n_events / max(1, total),
            "algorithmic_bytes": c_bytes, "achieved_GBps": c_bytes / (c_ms * 1e-3) / 1e9,
        }
        del comp
        torch.cuda.empty_cache()

    if args.l2_reps > 0:
        # group-aware L2 (section 6.1 routing, Appendix B) over the step's
        # summaries, with the workload's TP / PP / DP / EP layout
        route, goff, gmem = tracegen.workload_groups(args.config, R, K)
        tt = lambda a, dt: torch.from_numpy(np.ascontiguousarray(a.astype(dt))).to(dev)  # noqa: E731
        route_d, goff_d, gmem_d = tt(route, np.uint8), tt(goff, np.int32), tt(gmem, np.int32)
        l2_out = pa.alloc_l2(R, S, K, goff.shape[0], goff.shape[1] - 1, dev)
        pa.l2(s["count"], s["sum_ns"], R, S, K, route_d, goff_d, gmem_d, out=l2_out)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(args.l2_reps):
            pa.l2(s["count"], s["sum_ns"], R, S, K, route_d, goff_d, gmem_d, out=l2_out)
        e1.record(stream)
        torch.cuda.synchronize()
        l2_ms = e0.elapsed_time(e1) / args.l2_reps
        assert int(l2_out["dev_status"].item()) == 0
        lf = l2_out["flags"].cpu().numpy().reshape(R, S, K)
        cls = l2_out["cls"].cpu().numpy()
        strag = sorted(truth["stragglers"])
        others = np.setdiff1d(np.arange(R), strag)
        ev_cells = (lf & 1) > 0
        result["l2"] = {
            "ms": l2_ms, "ms_per_step": l2_ms / S, "layout_tp_pp_ep": list(tracegen.LAYOUTS[args.config]),
            "groups_evaluated": int((cls != 0xFF).sum()),
            "groups_by_class": [int((cls == c).sum()) for c in (0, 1, 2)],
            "straggler_cells_flagged_frac": float(((lf[strag] & 2) > 0).sum() / max(1, ev_cells[strag].sum())),
            "other_cells_flagged_frac": float(((lf[others] & 2) > 0).sum() / max(1, ev_cells[others].sum())),
        }
        del l2_out
        torch.cuda.empty_cache()

    if args.kde_reps > 0:
        # KDE valley clustering of every (rank, step, kernel) group (section
        # 5.2): bucketing scatter + per-cell density, valleys, filters, exact
        # p50 / p99, over the summaries of the last step
        kde_out = pa.alloc_kde(trace.n_events, R, S, K, dev)
        for _ in range(2):
            pa.kde(ev, s, R, S, K, NS, out=kde_out)
        torch.cuda.synchronize()
        kde_calls = timed_calls(lambda: pa.kde(ev, s, R, S, K, NS, out=kde_out), args.kde_reps, stream)
        kde_ms = float(np.mean(kde_calls))
        assert int(kde_out["dev_status"].item()) == 0
        ncl = kde_out["n_clusters"].cpu().numpy()
        n_valid = int(s["n_valid"].cpu().numpy().view(np.uint32).astype(np.int64).sum())
        # summary record per present cell: kernel id 4 B + cluster count 1 B,
        # then (count 4, p50 8, p99 8) per cluster
        wire = int(5 * np.count_nonzero(ncl) + 20 * ncl.astype(np.int64).sum())
        # algorithmic bytes: every event's kernel id, start and end read once
        # (20 B) and its stream (4 B) where validity is not known from the
        # summary (a rank-step with invalid events, or id spaces beyond 2,048,
        # whose scatter reads every field); each rank-step's n_invalid (4 B);
        # each cell's count / min / max read (20 B) and its record written
        # (n_clusters 1, count 16, p50 32, p99 32, bw 4 = 85 B). The bucketed
        # durations the kernels write and re-read are the design's, not the
        # operation's.
        seg_events = torch.diff(ev["seg_off"]).to(torch.int64)
        inv = (s["n_invalid"].to(torch.int64) & 0xFFFFFFFF) > 0
        stream_events = trace.n_events if K > 2048 else int(seg_events[inv].sum().item())
        ev_bytes = 20 * trace.n_events + 4 * stream_events + 4 * G
        kde_alg = ev_bytes + (20 + 85) * G * K
        # the scatter writes each valid duration once, in 4 bytes where every
        # present cell of its rank-step has a maximum below 2^31 ns, else 8
        wide = ((s["max_ns"] >= 2**31) & (s["count"] > 0)).view(G, K).any(dim=1)
        nv_seg = s["n_valid"].to(torch.int64) & 0xFFFFFFFF
        rec_bytes = int((nv_seg * torch.where(wide, 8, 4)).sum().item())
        result["kde"] = {
            "ms": kde_ms, "ms_median": float(np.median(kde_calls)), "events_per_s": trace.n_events / (kde_ms * 1e-3),
            "roofline": {"bound": "hbm", "achieved": kde_alg / (kde_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": kde_alg / (kde_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                         "algorithmic_bytes_per_call": kde_alg},
            "scatter_algorithmic_bytes": ev_bytes + rec_bytes + 8 * G * K,
            "cells": G * K, "present_cells": int(np.count_nonzero(ncl)),
            "mean_clusters_per_present_cell": float(ncl[ncl > 0].mean()) if (ncl > 0).any() else 0.0,
            "cells_with_several_clusters": int((ncl > 1).sum()),
            "summary_bytes_per_rank_step": wire / G,
            "raw_bytes_per_rank_step": 24 * trace.n_events / G,
        }
        if args.w1_reps > 0:
            # cross-rank W1 deviation scores over those clusters (section 6.2,
            # Eq. 2 - 4): 64-point log grid, IQR fence alpha 1.5
            w1_out = pa.alloc_w1(R, S, K, 64, dev)
            pa.w1(kde_out, R, S, K, out=w1_out)
            torch.cuda.synchronize()
            w1_calls = timed_calls(lambda: pa.w1(kde_out, R, S, K, out=w1_out), args.w1_reps, stream)
            w1_ms = float(np.mean(w1_calls))
            assert int(w1_out["dev_status"].item()) == 0
            wf = w1_out["flag"].cpu().numpy().reshape(R, S, K).astype(bool)
            pres = ncl.reshape(R, S, K) > 0
            strag = sorted(truth["stragglers"])
            others = np.setdiff1d(np.arange(R), strag)
            # algorithmic bytes: each cell's cluster record read (81 B) and its
            # score and flag written (9 B); per (step, kernel) 64 B of
            # statistics. The 16-bit CDF table in the workspace is the design's.
            w1_alg = 90 * G * K + 64 * S * K
            result["w1"] = {
                "ms": w1_ms, "ms_median": float(np.median(w1_calls)), "ms_per_step": w1_ms / S, "grid": 64,
                "roofline": {"bound": "hbm", "achieved": w1_alg / (w1_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS,
                             "unit": "GB/s", "frac": w1_alg / (w1_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                             "algorithmic_bytes_per_call": w1_alg},
                "kernel_steps": S * K, "present_cells": int(pres.sum()),
                "straggler_cells_flagged_frac": float(wf[strag].sum() / max(1, pres[strag].sum())),
                "other_cells_flagged_frac": float(wf[others].sum() / max(1, pres[others].sum())),
            }
            del w1_out
        del kde_out
        torch.cuda.empty_cache()

    if not args.no_cpu_baseline:
        sample = min(args.cpu_sample_ranks, R)
        gs = sample * S
        g_h = {f: s[f][:gs * K * (NB if f == "hist" else 1)].cpu().numpy()
               for f in ("count", "sum_ns", "min_ns", "max_ns", "hist")}
        g_h.update({f: s[f][:gs].cpu().numpy() for f in ("n_valid", "n_invalid", "step_ns", "busy_ns")})
        ev_h = trace.fill_host(0, min(G, 64))
        assert np.array_equal(trace.checksum_host(ev_h, 0, min(G, 64)), cs_dev), "device/host trace mismatch"
        print(f"[bench] cpu baseline: oracle on {sample} ranks", file=sys.stderr, flush=True)
        cb = cpu_baseline(trace, sample, g_h)
        mism = cb.pop("_mismatches")
        result["cpu_baseline"] = cb
        result["parity_sample"] = {"segments": sample * S, "mismatches": mism}
        workers = min(16, os.cpu_count() or 1)
        print(f"[bench] sharded cpu baseline: {workers} threads", file=sys.stderr, flush=True)
        result["cpu_baseline_sharded"] = cpu_baseline_sharded(trace, workers)
        if mism:
            print(json.dumps(result))
            raise SystemExit(f"parity failure on the sampled segments: {mism} mismatching elements")
    print(json.dumps(result))


if __name__ == "__main__":
    main()
