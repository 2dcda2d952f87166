"""The KDE's floating-point steps on the device against the oracle's (the host
C library), over their whole reachable domain.

argus_kde's integer outputs (grids, bandwidths, densities, valleys,
clusters, percentiles) follow exactly from three floating-point results: the
Gaussian weights floor(65536 exp(-32768 t^2 / H^2) + 0.5), n^(-1/5) (the
double nearest to the real value, decided by exact integer comparisons on
both sides; a table of it below 65,536 durations) and the bandwidth H =
floor(256 * 1.06 sqrt(var) n^(-1/5) + 0.5). A probe library evaluates the
device's ones through the same inline functions the cell kernels call, and
they must equal the oracle's bit for bit:

* weights: every bandwidth H = 1 .. 2^17 (h up to 512 grid steps, 8 octaves)
  and every t up to the kernels' table bound floor(0.019 H) + 2, at which the
  weight must already be 0 (163 million weights);
* n^(-1/5): every n from 1 to 2^22 and 2^20 random n up to 2^33;
* H: 2^22 random (var, n) pairs, var from exact integer moment quotients as
  the kernels form them and log-uniform doubles.
The grid index of a duration (an integer result that a hardware log2
estimate only starts) must equal the oracle's exact one for every duration
below 2^20, every threshold of every octave and its two neighbours, and 2^22
log-uniform random durations; so must the 32-bit form the kernels use for
4-byte records, on every one of those durations below 2^32.
The full-size KDE parity tests compare the bandwidth and clusters of every
cell of the benchmarked workloads on top of this.
"""
import ctypes
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from tests import parity as P

pytestmark = pytest.mark.gpu
DEV = "cuda"
PROBE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "probe", "libkdemathprobe.so")
POW_TABLE = 65536


def _probe():
    assert os.path.exists(PROBE), f"{PROBE} is not built (__graft_entry__.build())"
    L = ctypes.CDLL(PROBE)
    V = ctypes.c_void_p
    L.probe_kde_weights.argtypes = [V, V, ctypes.c_int32, V, V]
    L.probe_kde_root5.argtypes = [V, ctypes.c_int64, V, V]
    L.probe_kde_bw_q8.argtypes = [V, V, V, ctypes.c_int64, V, V]
    L.probe_kde_grid.argtypes = [V, ctypes.c_int64, V, V]
    L.probe_kde_grid32.argtypes = [V, ctypes.c_int64, V, V]
    return L


def _dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).to(DEV)


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def test_weights_match_the_host_for_every_bandwidth_up_to_2_17():
    print("\n[gpu-case] kde weights: H = 1 .. 2^17, every t to the table bound", flush=True)
    L = _probe()
    n_diff = n_tot = 0
    chunks = np.array_split(np.arange(1, (1 << 17) + 1, dtype=np.int64), 16)

    def host(Hs):
        nt = Hs * 19 // 1000 + 3  # t = 0 .. floor(0.019 H) + 2
        off = np.concatenate([[0], np.cumsum(nt)]).astype(np.int64)
        return off, oracle.kde_weights_many(Hs, off)

    with ThreadPoolExecutor(P.host_threads()) as ex:
        hosts = list(ex.map(host, chunks))
    for Hs, (off, want) in zip(chunks, hosts):
        w = torch.empty(int(off[-1]), dtype=torch.int32, device=DEV)
        assert L.probe_kde_weights(_dev(Hs).data_ptr(), _dev(off).data_ptr(), len(Hs), w.data_ptr(), _stream()) == 0
        got = w.cpu().numpy().view(np.uint32)
        n_diff += int(np.count_nonzero(got != want))
        n_tot += got.size
        # the kernels size their weight tables by this bound
        assert (want[off[1:] - 1] == 0).all(), "a weight beyond floor(0.019 H) + 2 is nonzero"
    assert n_tot > 1.6e8
    assert n_diff == 0, f"{n_diff} of {n_tot} device weights differ from the host's"


def test_fifth_root_matches_the_oracle():
    print("\n[gpu-case] kde n^(-1/5): n = 1 .. 2^22 and random n to 2^33", flush=True)
    L = _probe()
    rng = np.random.default_rng(7)
    n = np.concatenate([np.arange(1, 1 << 22, dtype=np.int64),
                        rng.integers(1 << 22, 1 << 33, size=1 << 20, dtype=np.int64)])
    out = torch.empty(n.size, dtype=torch.float64, device=DEV)
    assert L.probe_kde_root5(_dev(n).data_ptr(), n.size, out.data_ptr(), _stream()) == 0
    got = out.cpu().numpy()
    want = oracle.kde_root5_many(n)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (bad.size, n[bad[:5]], got[bad[:5]], want[bad[:5]])


def test_bandwidth_matches_the_host():
    print("\n[gpu-case] kde bandwidth: 2^22 random (var, n)", flush=True)
    L = _probe()
    rng = np.random.default_rng(8)
    m = 1 << 21
    n = np.exp(rng.uniform(np.log(2), np.log(2.0**33), size=2 * m)).astype(np.int64)
    # the kernels' var: an exact integer n s2 - s1^2 over n (n - 1), grid spans
    # up to 4,096 points
    span = rng.integers(1, 4096, size=m).astype(np.float64)
    V = np.floor(rng.random(m) * (n[:m].astype(np.float64) ** 2) * span * span / 4)
    var = np.concatenate([V / (n[:m].astype(np.float64) * (n[:m] - 1).astype(np.float64)),
                          np.exp(rng.uniform(np.log(1e-6), np.log(1e7), size=m))])
    pw_small = np.where(n < POW_TABLE, oracle.kde_root5_many(np.maximum(n, 1)), 0.0)
    out = torch.empty(n.size, dtype=torch.int64, device=DEV)
    assert L.probe_kde_bw_q8(_dev(var).data_ptr(), _dev(n).data_ptr(), _dev(pw_small).data_ptr(), n.size,
                             out.data_ptr(), _stream()) == 0
    got = out.cpu().numpy()
    want = oracle.kde_bw_q8_many(var, n)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, (bad.size, var[bad[:5]], n[bad[:5]], got[bad[:5]], want[bad[:5]])


def test_grid_index_matches_the_oracle():
    print("\n[gpu-case] kde grid index (64- and 32-bit forms): d < 2^20, every threshold of every octave +-1, 2^22 random", flush=True)
    th = oracle.kde_thresholds().astype(np.uint64)
    parts = [np.arange(1 << 20, dtype=np.uint64)]
    # every threshold of every octave and its neighbours: for octaves below
    # 2^23 the threshold's duration is the smallest d whose shifted mantissa
    # reaches it
    for e in range(20, 63):
        if e >= 23:
            b = th << np.uint64(e - 23)
        else:
            sh = np.uint64(23 - e)
            b = (th + (np.uint64(1) << sh) - np.uint64(1)) >> sh
        parts += [b - np.uint64(1), b, b + np.uint64(1)]
    rng = np.random.default_rng(17)
    parts.append(np.exp2(rng.uniform(1.0, 62.99, 1 << 22)).astype(np.uint64))
    parts.append(np.array([2**63 - 1, 2**63 - 2, 2**62, 2**62 - 1], np.uint64))
    d = np.unique(np.concatenate(parts))
    want = oracle.kde_bin_many(d)
    out = torch.empty(d.size, dtype=torch.int32, device=DEV)
    assert _probe().probe_kde_grid(_dev(d.view(np.int64)).data_ptr(), d.size, out.data_ptr(), _stream()) == 0
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, (bad.size, d[bad[:5]], got[bad[:5]], want[bad[:5]])
    # the 32-bit form (4-byte records) on every sampled duration below 2^32
    sel = d < np.uint64(1 << 32)
    d32, want32 = d[sel].astype(np.uint32), want[sel]
    assert d32.size > (1 << 20) and int(d32.max()) > (1 << 31)
    out32 = torch.empty(d32.size, dtype=torch.int32, device=DEV)
    assert _probe().probe_kde_grid32(_dev(d32.view(np.int32)).data_ptr(), d32.size, out32.data_ptr(), _stream()) == 0
    torch.cuda.synchronize()
    got32 = out32.cpu().numpy()
    bad = np.flatnonzero(got32 != want32)
    assert bad.size == 0, (bad.size, d32[bad[:5]], got32[bad[:5]], want32[bad[:5]])
