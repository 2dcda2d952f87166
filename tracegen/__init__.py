"""Seeded synthetic kernel-event traces for the summarizer and detectors.

The paper measures on proprietary production traces (section 8.3, Table
"data-volume"; section 9 case studies), so every workload here is synthetic.
This module builds, per workload, the tables that the per-event rule in
``tg_event.h`` reads, the ground truth of what was injected, and fills the
structure-of-arrays event buffers on the host (numpy) or on the device
(torch tensors, filled by a HIP kernel from the same per-event rule).

Workload shapes:
* each rank-step repeats one per-job template of ``tmpl_len`` kernel launches
  ``events_per_seg / tmpl_len`` times (the repetitive per-stream patterns of
  section 5.2); stream = kernel id mod n_streams;
* durations are lognormal around a per-kernel base (log of the base uniform
  over [ln 2 us, ln 5 ms], sigma 0.1 in ln), or Pareto(alpha 1.5, x_m 10 us)
  for the "hot" communication-like ids of the skew workload; a share of the
  lognormal ids runs at 2 or 3 scales (x1, x3, x9) depending on the template
  position, the multimodal per-kernel durations of section 5.2;
* injected faults follow the case-study shapes: whole-rank slowdowns
  (stragglers, section 9.1), single degraded (rank, kernel) pairs (Appendix D
  table), host stalls that stretch one step without slowing any kernel
  (section 9.4), and a straggler masked by inflated communication on its
  peers (section 9.5).

No part of the summarization or detection method is computed here.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os
from typing import Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtracegen.so")

EPOCH_NS = 1_764_000_000_000_000_000  # > 2**60: no float64 shortcut survives it
LN_SIGMA = 0.1
PARETO_ALPHA = 1.5
PARETO_XM_NS = 10_000
NO_STALL = 2**31 - 1


@dataclasses.dataclass(frozen=True)
class TraceConfig:
    name: str
    seed: int
    n_ranks: int
    n_steps: int
    events_per_seg: int
    n_kernels: int
    n_streams: int
    tmpl_len: int
    ids: str = "uniform"          # "uniform" | "zipf" | "skew"
    zipf_s: float = 1.1
    n_hot: int = 0                 # skew: ids [0, n_hot) are hot (Pareto durations)
    hot_pm: int = 900              # skew: permille of template positions that are hot
    swap_pm: int = 0               # per-rank template pair swaps (permille)
    invalid_ppm: int = 0           # corrupted records (ppm), edge-case tests only
    n_stragglers: int = 0
    straggler_pm: tuple = (1000, 1000)
    n_pairs: int = 0
    pair_pm: tuple = (1000, 1000)
    n_anomalous: int = 0           # host-stalled (rank, step) segments
    masked_straggler: bool = False  # skew: one rank slow on cold ids, peers slow on hot ids
    modal_pm: int = 300            # permille of lognormal ids whose positions run at several scales

    @property
    def n_segments(self) -> int:
        return self.n_ranks * self.n_steps

    @property
    def n_events(self) -> int:
        return self.n_segments * self.events_per_seg


# The five workloads (tiny, medium, production-shaped step, cluster-scale
# step, skew/contention stress).
CONFIGS = {
    "tiny": TraceConfig("tiny", seed=1, n_ranks=8, n_steps=4, events_per_seg=20_000, n_kernels=64,
                        n_streams=4, tmpl_len=2_000, ids="uniform", n_stragglers=1,
                        straggler_pm=(1300, 1300), n_pairs=1, pair_pm=(2000, 2000)),
    "medium": TraceConfig("medium", seed=2, n_ranks=256, n_steps=8, events_per_seg=100_000, n_kernels=512,
                          n_streams=8, tmpl_len=10_000, ids="zipf", n_stragglers=3,
                          straggler_pm=(1150, 1500), n_pairs=5, pair_pm=(1500, 3000), n_anomalous=2),
    "production": TraceConfig("production", seed=3, n_ranks=1024, n_steps=1, events_per_seg=400_000,
                              n_kernels=2048, n_streams=16, tmpl_len=40_000, ids="zipf", n_stragglers=5,
                              straggler_pm=(1050, 1500)),
    "cluster": TraceConfig("cluster", seed=4, n_ranks=10_240, n_steps=1, events_per_seg=400_000,
                           n_kernels=2048, n_streams=16, tmpl_len=40_000, ids="zipf", swap_pm=50,
                           n_stragglers=10, straggler_pm=(1050, 1500), n_pairs=50, pair_pm=(1500, 3000)),
    "skew": TraceConfig("skew", seed=5, n_ranks=4096, n_steps=4, events_per_seg=200_000, n_kernels=8200,
                        n_streams=16, tmpl_len=20_000, ids="skew", n_hot=8, hot_pm=900,
                        masked_straggler=True),
}


def config(name: str, **overrides) -> TraceConfig:
    return dataclasses.replace(CONFIGS[name], **overrides)


class _Params(ctypes.Structure):
    _fields_ = [
        ("seed", ctypes.c_uint64),
        ("n_ranks", ctypes.c_int32), ("n_steps", ctypes.c_int32),
        ("n_kernels", ctypes.c_int32), ("n_streams", ctypes.c_int32),
        ("tmpl_len", ctypes.c_int32), ("n_hot", ctypes.c_int32),
        ("swap_pm", ctypes.c_int32), ("invalid_ppm", ctypes.c_int32),
        ("epoch_ns", ctypes.c_int64), ("step_period_ns", ctypes.c_int64),
        ("t_span_ns", ctypes.c_int64),
    ]


_TABLE_FIELDS = ["tmpl_kid", "tmpl_off", "tmpl_base_ns", "ln_q24", "pareto_ns", "mult_hot_pm", "mult_cold_pm",
                 "pair_off", "pair_kid", "pair_pm", "stall_rep", "stall_ns"]


class _Tables(ctypes.Structure):
    _fields_ = [(f, ctypes.c_void_p) for f in _TABLE_FIELDS]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        P, V = ctypes.POINTER, ctypes.c_void_p
        L.tg_fill_host.argtypes = [P(_Params), P(_Tables), V, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                   V, V, V, V, ctypes.c_int32]
        L.tg_checksum_host.argtypes = [P(_Params), V, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64,
                                       V, V, V, V, V]
        L.tg_fill_device.argtypes = [P(_Params), P(_Tables), V, ctypes.c_int32, ctypes.c_int32,
                                     ctypes.c_int64, V, V, V, V, V]
        L.tg_checksum_device.argtypes = [V, ctypes.c_int32, ctypes.c_int32, ctypes.c_int64, V, V, V, V, V, V]
        for f in (L.tg_fill_host, L.tg_checksum_host, L.tg_fill_device, L.tg_checksum_device):
            f.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


def _phi_inv(p: np.ndarray) -> np.ndarray:
    # Standard normal quantile (Cephes ndtri via scipy).
    from scipy.special import ndtri
    return ndtri(p)


def build_ln_table() -> np.ndarray:
    j = np.arange(65536, dtype=np.float64)
    z = _phi_inv((j + 0.5) / 65536.0)
    return np.rint(np.exp(LN_SIGMA * z) * 2.0**24).astype(np.uint32)


def build_pareto_table() -> np.ndarray:
    j = np.arange(65536, dtype=np.float64)
    q = PARETO_XM_NS * ((j + 0.5) / 65536.0) ** (-1.0 / PARETO_ALPHA)
    return np.rint(q).astype(np.uint32)


class Trace:
    """One synthetic workload: tables, segment offsets and ground truth."""

    def __init__(self, cfg: TraceConfig, seg_lengths: Optional[Sequence[int]] = None):
        self.cfg = cfg
        R, S, K, NS, T = cfg.n_ranks, cfg.n_steps, cfg.n_kernels, cfg.n_streams, cfg.tmpl_len
        G = R * S
        rng = np.random.default_rng([cfg.seed, 0x7A61])
        if seg_lengths is None:
            lens = np.full(G, cfg.events_per_seg, dtype=np.int64)
        else:
            lens = np.asarray(seg_lengths, dtype=np.int64)
            assert lens.shape == (G,) and (lens >= 0).all()
        self.seg_off = np.zeros(G + 1, dtype=np.int64)
        np.cumsum(lens, out=self.seg_off[1:])
        self.n_events = int(self.seg_off[-1])

        # per-kernel nominal durations: log uniform over [ln 2 us, ln 5 ms]
        self.base_ns = np.rint(np.exp(rng.uniform(math.log(2e3), math.log(5e6), size=K))).astype(np.int64)
        self.ln_q24 = build_ln_table()
        self.pareto_ns = build_pareto_table()

        # template kernel ids
        if cfg.ids == "uniform":
            kid = rng.integers(0, K, size=T).astype(np.int32)
            m = min(T, K)
            kid[:m] = np.arange(m, dtype=np.int32)
        elif cfg.ids == "zipf":
            w = (np.arange(1, K + 1, dtype=np.float64)) ** (-cfg.zipf_s)
            kid = rng.choice(K, size=T, p=w / w.sum()).astype(np.int32)
        elif cfg.ids == "skew":
            hot = rng.random(T) < cfg.hot_pm / 1000.0
            kid = np.where(hot, rng.integers(0, cfg.n_hot, size=T),
                           rng.integers(cfg.n_hot, K, size=T)).astype(np.int32)
        else:
            raise ValueError(cfg.ids)
        self.tmpl_kid = kid
        # multimodal ids: the same kernel at different template positions runs
        # at different scales (section 5.2: one collective at two positions
        # moving different volumes). Half of the chosen ids are bimodal
        # (x1, x3), half trimodal (x1, x3, x9); each position draws its scale
        # uniformly from its id's set. Drawn from a stream of its own so the
        # injections below do not depend on it.
        mrng = np.random.default_rng([cfg.seed, 0x4D4F4445])
        modal = (mrng.random(K) < cfg.modal_pm / 1000.0) & (np.arange(K) >= cfg.n_hot)
        n_modes = np.where(modal, np.where(mrng.random(K) < 0.5, 2, 3), 1)
        mode = (mrng.random(T) * n_modes[kid]).astype(np.int64)
        self.tmpl_mode_pm = (1000 * 3 ** mode).astype(np.int64)
        self.n_modes = n_modes
        self.tmpl_base_ns = np.where(kid < cfg.n_hot, 0, self.base_ns[kid] * self.tmpl_mode_pm // 1000)
        # per-stream cursors: each stream runs its template launches back to
        # back with 1-20 us gaps
        nominal = np.where(kid < cfg.n_hot, 3 * PARETO_XM_NS, self.tmpl_base_ns)
        gaps = rng.integers(1_000, 20_001, size=T)
        cursor = np.zeros(NS, dtype=np.int64)
        off = np.zeros(T, dtype=np.int64)
        for p in range(T):
            st = kid[p] % NS
            cursor[st] += gaps[p]
            off[p] = cursor[st]
            cursor[st] += nominal[p]
        self.tmpl_off = off
        self.t_span_ns = int(cursor.max()) + 20_000
        reps_max = max(1, -(-int(lens.max(initial=0)) // T))
        self.step_period_ns = 4 * reps_max * self.t_span_ns

        # injections (ground truth)
        mult_hot = np.full(R, 1000, dtype=np.int32)
        mult_cold = np.full(R, 1000, dtype=np.int32)
        strag = rng.choice(R, size=cfg.n_stragglers, replace=False) if cfg.n_stragglers else np.zeros(0, int)
        strag_pm = rng.integers(cfg.straggler_pm[0], cfg.straggler_pm[1] + 1, size=len(strag))
        for r, m in zip(strag, strag_pm):
            mult_hot[r] = m
            mult_cold[r] = m
        self.stragglers = {int(r): int(m) for r, m in zip(strag, strag_pm)}
        self.masked_straggler = None
        if cfg.masked_straggler:
            ms = int(rng.integers(0, R))
            mult_hot[:] = 1500
            mult_hot[ms] = 1000
            mult_cold[ms] = 1300
            self.masked_straggler = ms
        normal = np.setdiff1d(np.arange(R), strag)
        if self.masked_straggler is not None:
            normal = np.setdiff1d(normal, [self.masked_straggler])
        present = np.unique(kid[kid >= cfg.n_hot])
        pairs = {}
        while len(pairs) < cfg.n_pairs:
            r = int(rng.choice(normal))
            k = int(rng.choice(present))
            if (r, k) not in pairs:
                pairs[(r, k)] = int(rng.integers(cfg.pair_pm[0], cfg.pair_pm[1] + 1))
        self.pairs = pairs
        pair_off = np.zeros(R + 1, dtype=np.int32)
        by_rank = sorted(pairs.items())
        for (r, _), _m in by_rank:
            pair_off[r + 1] += 1
        np.cumsum(pair_off, out=pair_off)
        self.pair_off = pair_off
        self.pair_kid = np.array([k for (r, k), _ in by_rank] or [0], dtype=np.int32)
        self.pair_pm = np.array([m for _, m in by_rank] or [1000], dtype=np.int32)
        self.mult_hot_pm, self.mult_cold_pm = mult_hot, mult_cold

        stall_rep = np.full(G, NO_STALL, dtype=np.int32)
        stall_ns = np.zeros(G, dtype=np.int64)
        anomalous = []
        if cfg.n_anomalous:
            assert S >= 3, "anomalous steps need an interior step"
            cand = np.setdiff1d(normal, [r for (r, _) in pairs])
            ranks = rng.choice(cand, size=cfg.n_anomalous, replace=False)
            for r in ranks:
                s = int(rng.integers(1, S - 1))
                g = int(r) * S + s
                reps = max(1, int(lens[g]) // T)
                stall_rep[g] = reps // 2
                stall_ns[g] = reps * self.t_span_ns
                anomalous.append((int(r), s))
        self.anomalous = anomalous
        self.stall_rep, self.stall_ns = stall_rep, stall_ns

        self._params = _Params(cfg.seed, R, S, K, NS, T, cfg.n_hot, cfg.swap_pm, cfg.invalid_ppm,
                               EPOCH_NS, self.step_period_ns, self.t_span_ns)
        self._host_tables = {
            "tmpl_kid": self.tmpl_kid, "tmpl_off": self.tmpl_off, "tmpl_base_ns": self.tmpl_base_ns,
            "ln_q24": self.ln_q24, "pareto_ns": self.pareto_ns, "mult_hot_pm": self.mult_hot_pm,
            "mult_cold_pm": self.mult_cold_pm, "pair_off": self.pair_off, "pair_kid": self.pair_kid,
            "pair_pm": self.pair_pm, "stall_rep": self.stall_rep, "stall_ns": self.stall_ns,
        }
        for k, v in self._host_tables.items():
            self._host_tables[k] = np.ascontiguousarray(v)
        self._dev_tables = None

    # ------------------------------------------------------------------ host
    def fill_host(self, g_begin: int = 0, g_end: Optional[int] = None, n_threads: int = 8) -> dict:
        """Events of segments [g_begin, g_end) as numpy SoA plus local seg_off."""
        G = self.cfg.n_segments
        g_end = G if g_end is None else g_end
        base = int(self.seg_off[g_begin])
        n = int(self.seg_off[g_end]) - base
        out = {
            "kernel_id": np.empty(n, np.int32), "stream": np.empty(n, np.int32),
            "start_ns": np.empty(n, np.int64), "end_ns": np.empty(n, np.int64),
        }
        tb = _Tables(*[_ptr(self._host_tables[f]) for f in _TABLE_FIELDS])
        rc = lib().tg_fill_host(ctypes.byref(self._params), ctypes.byref(tb), _ptr(self.seg_off), g_begin,
                                g_end, base, _ptr(out["kernel_id"]), _ptr(out["stream"]),
                                _ptr(out["start_ns"]), _ptr(out["end_ns"]), n_threads)
        assert rc == 0, rc
        out["seg_off"] = np.ascontiguousarray(self.seg_off[g_begin:g_end + 1] - base)
        return out

    def checksum_host(self, ev: dict, g_begin: int = 0, g_end: Optional[int] = None) -> np.ndarray:
        g_end = self.cfg.n_segments if g_end is None else g_end
        base = int(self.seg_off[g_begin])
        sums = np.zeros(g_end - g_begin, dtype=np.uint64)
        rc = lib().tg_checksum_host(ctypes.byref(self._params), _ptr(self.seg_off), g_begin, g_end, base,
                                    _ptr(ev["kernel_id"]), _ptr(ev["stream"]), _ptr(ev["start_ns"]),
                                    _ptr(ev["end_ns"]), _ptr(sums))
        assert rc == 0, rc
        return sums

    # ---------------------------------------------------------------- device
    def _device_tables(self, device):
        import torch
        if self._dev_tables is None:
            self._dev_tables = {k: torch.from_numpy(v).to(device) for k, v in self._host_tables.items()}
            self._dev_seg_off = torch.from_numpy(self.seg_off).to(device)
        return self._dev_tables

    def alloc_device(self, device="cuda"):
        import torch
        n = self.n_events
        return {
            "kernel_id": torch.empty(n, dtype=torch.int32, device=device),
            "stream": torch.empty(n, dtype=torch.int32, device=device),
            "start_ns": torch.empty(n, dtype=torch.int64, device=device),
            "end_ns": torch.empty(n, dtype=torch.int64, device=device),
        }

    def fill_device(self, ev: Optional[dict] = None, device="cuda", chunk_segments: int = 4096) -> dict:
        """Fill every segment on the device; returns SoA torch tensors + seg_off."""
        import torch
        if ev is None:
            ev = self.alloc_device(device)
        dt = self._device_tables(device)
        tb = _Tables(*[dt[f].data_ptr() for f in _TABLE_FIELDS])
        stream = torch.cuda.current_stream(device).cuda_stream
        G = self.cfg.n_segments
        for g0 in range(0, G, chunk_segments):
            g1 = min(G, g0 + chunk_segments)
            rc = lib().tg_fill_device(ctypes.byref(self._params), ctypes.byref(tb), self._dev_seg_off.data_ptr(),
                                      g0, g1, 0, ev["kernel_id"].data_ptr(), ev["stream"].data_ptr(),
                                      ev["start_ns"].data_ptr(), ev["end_ns"].data_ptr(), stream)
            assert rc == 0, rc
        ev["seg_off"] = self._dev_seg_off
        return ev

    def checksum_device(self, ev: dict, g_begin: int = 0, g_end: Optional[int] = None) -> np.ndarray:
        import torch
        g_end = self.cfg.n_segments if g_end is None else g_end
        self._device_tables(ev["kernel_id"].device)
        sums = torch.zeros(g_end - g_begin, dtype=torch.int64, device=ev["kernel_id"].device)
        stream = torch.cuda.current_stream(ev["kernel_id"].device).cuda_stream
        rc = lib().tg_checksum_device(self._dev_seg_off.data_ptr(), g_begin, g_end, 0,
                                      ev["kernel_id"].data_ptr(), ev["stream"].data_ptr(),
                                      ev["start_ns"].data_ptr(), ev["end_ns"].data_ptr(), sums.data_ptr(), stream)
        assert rc == 0, rc
        return sums.cpu().numpy().view(np.uint64)

    # ----------------------------------------------------------------- truth
    def truth(self) -> dict:
        return {
            "stragglers": set(self.stragglers) | ({self.masked_straggler} if self.masked_straggler is not None
                                                  else set()),
            "pairs": set(self.pairs),
            "anomalous": set(self.anomalous),
            "masked_straggler": self.masked_straggler,
        }


def make(name: str, seg_lengths=None, **overrides) -> Trace:
    return Trace(config(name, **overrides), seg_lengths=seg_lengths)


# ---------------------------------------------------------------------------
# Parallelism groups and the event routing table (inputs of the L2 step).
# Ranks follow the usual tensor-major layout r = t + TP (p + PP d) with
# tensor index t, pipeline stage p and data-parallel index d; expert-parallel
# groups split each data-parallel group into chunks of EP consecutive d.
DIMS = ("tp", "pp", "dp", "ep")


def parallel_groups(n_ranks: int, tp: int, pp: int, ep: int = 1):
    """Group lists of the four parallelism dimensions: (group_off
    [4][max_groups + 1] int32, members [4][n_ranks] int32, n_groups [4])."""
    assert n_ranks % (tp * pp) == 0
    dp = n_ranks // (tp * pp)
    assert dp % ep == 0
    r = np.arange(n_ranks)
    t, p, d = r % tp, (r // tp) % pp, r // (tp * pp)
    keys = [d * pp + p,                      # TP group: ranks sharing (p, d)
            d * tp + t,                      # PP group: ranks sharing (t, d)
            p * tp + t,                      # DP group: ranks sharing (t, p)
            ((d // ep) * pp + p) * tp + t]   # EP group: (t, p) and a chunk of ep consecutive d
    n_groups = [n_ranks // tp, n_ranks // pp, tp * pp, n_ranks // ep]
    G = max(n_groups)
    off = np.zeros((4, G + 1), np.int32)
    mem = np.zeros((4, n_ranks), np.int32)
    for i, key in enumerate(keys):
        order = np.argsort(key, kind="stable")
        mem[i] = order
        cnt = np.bincount(key, minlength=G)
        off[i, 1:] = np.cumsum(cnt)
    return off, mem, n_groups


def event_routes(n_events: int, seed: int = 0, shares=(150, 100, 500, 250)) -> np.ndarray:
    """A seeded routing table: each event id is compared in one dimension
    (TP, PP, DP, EP), drawn with the given permille shares."""
    rng = np.random.default_rng([seed, 0x12A7])
    w = np.asarray(shares, np.float64)
    return rng.choice(4, size=n_events, p=w / w.sum()).astype(np.uint8)


# Parallel layout (tensor, pipeline, expert degrees) of each workload; the
# data-parallel degree is what remains of the rank count.
LAYOUTS = {"tiny": (2, 2, 2), "medium": (2, 4, 4), "production": (8, 4, 8), "cluster": (8, 8, 8),
           "skew": (8, 4, 8)}


def workload_groups(name: str, n_ranks: int, n_events: int, seed: int = 0):
    """(route, group_off, members) of a workload's parallel layout."""
    tp, pp, ep = LAYOUTS[name]
    off, mem, _ = parallel_groups(n_ranks, tp, pp, ep)
    return event_routes(n_events, seed), off, mem


def l1_series(n_ranks: int = 10_240, n_steps: int = 1000, seed: int = 7) -> np.ndarray:
    """Seeded per-rank step times [n_ranks][n_steps] (int64 ns) for the L1
    iteration-window path at long series: 1 s steps with 4% Gaussian noise,
    a 1.5x regression from step 600 on every 7th rank, a 3x spike at step 300
    on every 11th rank."""
    rng = np.random.default_rng(seed)
    y = (10**9 * (1 + 0.04 * rng.standard_normal((n_ranks, n_steps)))).astype(np.int64)
    if n_steps > 600:
        y[::7, 600:] = y[::7, 600:] * 3 // 2
    if n_steps > 300:
        y[::11, 300] *= 3
    return y
