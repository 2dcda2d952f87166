"""Pins of the oracle's KDE valley clustering (section 5.2, Eq. 1) against
values fixed by mathematics and by construction, not by the oracle itself:

* the grid's mantissa thresholds and grid values against exact big-integer
  logarithms (floor(log2 N) = N.bit_length() - 1);
* the bandwidth against the closed-form variance of two-spike data;
* hand-worked spike patterns whose outcome follows from the filter rules
  (size threshold, spacing threshold, the cluster cap and its tie rule);
* single-mode groups: one cluster whose p50 / p99 equal the standard
  library's lower median and numpy's inverted-CDF 0.99 quantile;
* lognormal mixtures whose components cannot overlap: every component is
  recovered with its exact count, lower median and nearest-rank p99;
* the trace generator's planted per-position duration scales.
"""
import math
import statistics

import numpy as np
import pytest

import oracle
import tracegen

P = oracle.KDE_DEFAULTS


def exact_theta(t: int) -> int:
    """Smallest m with floor(64 log2 m) >= 1472 + t, i.e. ceil(2^(23 + t/64))."""
    m = int(math.ceil(2.0 ** (23 + t / 64.0))) - 2
    while ((m ** 64).bit_length() - 1) < 1472 + t:
        m += 1
    return m


def exact_bin(d: int, s: int) -> int:
    """floor(2^s log2 d') with d' = d truncated to 24 significant bits."""
    if d < 2:
        return 0
    e = d.bit_length() - 1
    if e > 23:
        d = (d >> (e - 23)) << (e - 23)
    return (d ** (1 << s)).bit_length() - 1


def test_thresholds_exact():
    th = oracle.kde_thresholds()
    assert [int(x) for x in th] == [exact_theta(t) for t in range(64)]


def test_grid_values_exact():
    th = [exact_theta(t) for t in range(64)]
    vals = set(range(0, 4100))
    for e in range(0, 63):
        for t in range(64):
            # smallest duration of octave e whose 24-bit mantissa reaches th[t]
            b = th[t] << (e - 23) if e >= 23 else -(-th[t] >> (23 - e))
            for dd in (-1, 0, 1):
                if 0 <= b + dd < 2**63:
                    vals.add(b + dd)
    rng = np.random.default_rng(5)
    vals.update(int(x) for x in rng.integers(0, 2**63 - 1, size=2000, dtype=np.int64))
    vals.add(2**63 - 1)
    for d in sorted(vals):
        assert oracle.kde_bin(d, 6) == exact_bin(d, 6), d
    for s in (1, 3, 5):
        for d in sorted(vals)[::7]:
            assert oracle.kde_bin(d, s) == exact_bin(d, s), (d, s)


def _spikes(*pairs):
    out = []
    for d, n in pairs:
        out += [d] * n
    rng = np.random.default_rng(len(out))
    out = np.array(out, dtype=np.uint64)
    rng.shuffle(out)
    return out


def nearest_fifth_root_recip(n: int) -> float:
    """The double nearest to n^(-1/5), from 60-digit decimal arithmetic
    (Decimal -> float rounds to nearest)."""
    from decimal import Decimal, localcontext
    with localcontext() as ctx:
        ctx.prec = 60
        return float(Decimal(n) ** (Decimal(-1) / Decimal(5)))


def test_fifth_root_is_the_nearest_double():
    # the bandwidth's n^(-1/5): every n to 20,000, random n to 2^33, perfect
    # fifth powers and powers of two, against exact decimal arithmetic
    rng = np.random.default_rng(9)
    ns = np.concatenate([np.arange(1, 20_001), rng.integers(20_001, 2**33, size=5000),
                         np.array([k**5 for k in range(2, 80)] + [2**k for k in range(33)])]).astype(np.int64)
    got = oracle.kde_root5_many(ns)
    want = np.array([nearest_fifth_root_recip(int(n)) for n in ns])
    assert np.array_equal(got, want), ns[got != want][:5]


@pytest.mark.parametrize("na,nb,octaves", [(100, 100, 2), (1000, 300, 5), (7, 9, 3)])
def test_bandwidth_two_spikes(na, nb, octaves):
    # grid values 64*20 and 64*(20 + octaves): exact powers of two
    D = 64 * octaves
    r = oracle.kde_group(_spikes((2**20, na), (2**(20 + octaves), nb)))
    n = na + nb
    var = na * nb * D * D / (n * (n - 1))  # closed form of the sample variance
    h = 1.06 * math.sqrt(var) * nearest_fifth_root_recip(n)
    assert r["bw_q8"] == math.floor(h * 256 + 0.5)


def test_single_value_and_empty():
    r = oracle.kde_group([])
    assert r["n_clusters"] == 0 and r["count"].sum() == 0
    r = oracle.kde_group([12345])
    assert r["n_clusters"] == 1 and r["count"][0] == 1 and r["p50_ns"][0] == r["p99_ns"][0] == 12345
    r = oracle.kde_group([777] * 50)
    assert r["n_clusters"] == 1 and r["count"][0] == 50 and r["p50_ns"][0] == 777 and r["bw_q8"] == 0
    r = oracle.kde_group([0, 1, 1, 0])
    assert r["n_clusters"] == 1 and r["p50_ns"][0] == 0 and r["p99_ns"][0] == 1


def test_two_far_spikes():
    r = oracle.kde_group(_spikes((10_000, 1000), (1_000_000, 500)))
    assert r["n_clusters"] == 2
    assert list(r["count"]) == [1000, 500, 0, 0]
    assert list(r["p50_ns"][:2]) == [10_000, 1_000_000] and list(r["p99_ns"][:2]) == [10_000, 1_000_000]


def _lb(b: int) -> int:
    """Smallest duration with grid value >= b (s = 6)."""
    e, t = divmod(b, 64)
    th = exact_theta(t)
    return th << (e - 23) if e >= 23 else -(-th >> (23 - e))


@pytest.mark.parametrize("D,expect", [(96, 2), (95, 1), (120, 2), (60, 1)])
def test_spacing_filter_threshold(D, expect):
    # two equal spikes D grid steps apart: by symmetry the valley sits at
    # floor(D/2); it survives only if it is >= gap = 48 steps from both
    # extremes, i.e. D >= 96
    b0 = 64 * 25
    r = oracle.kde_group(_spikes((_lb(b0), 2000), (_lb(b0 + D), 2000)))
    assert oracle.kde_bin(_lb(b0 + D)) - oracle.kde_bin(_lb(b0)) == D
    assert r["n_cand"] >= 1
    assert r["n_clusters"] == expect
    if expect == 2:
        assert list(r["count"][:2]) == [2000, 2000]
    else:
        assert r["count"][0] == 4000


@pytest.mark.parametrize("nb,expect", [(52, 1), (53, 2)])
def test_cluster_size_threshold(nb, expect):
    # 1000 + nb samples: each side needs ceil(0.05 n) = 53 samples
    r = oracle.kde_group(_spikes((2**14, 1000), (2**19, nb)))
    assert r["n_clusters"] == expect
    if expect == 2:
        assert list(r["count"][:2]) == [1000, nb] and r["p50_ns"][1] == 2**19
    else:
        assert r["count"][0] == 1000 + nb and r["p99_ns"][0] == 2**19


@pytest.mark.parametrize("na,nb,expect", [(3, 3, 2), (3, 2, 1), (2, 3, 1)])
def test_min_count(na, nb, expect):
    r = oracle.kde_group(_spikes((2**10, na), (2**20, nb)))
    assert r["n_clusters"] == expect


def test_cluster_cap_drops_upper_valleys_on_ties():
    # six equal spikes 10 octaves apart: every valley is a zero plateau (the
    # bandwidth is ~60 steps, weights vanish beyond ~300 < 320 steps), so all
    # five valleys tie and the cap of four clusters drops the upper two
    N = 400_000
    d = _spikes(*[(2 ** (5 + 10 * i), N) for i in range(6)])
    r = oracle.kde_group(d)
    assert r["n_cand"] >= 5
    assert r["n_clusters"] == oracle.KDE_MAXC == 4
    assert list(r["count"]) == [N, N, N, 3 * N]
    assert list(r["p50_ns"]) == [2**5, 2**15, 2**25, 2**45]
    assert list(r["p99_ns"]) == [2**5, 2**15, 2**25, 2**55]


def _nearest_rank_p99(x):
    return int(np.quantile(np.asarray(x, dtype=np.float64), 0.99, method="inverted_cdf"))


@pytest.mark.parametrize("n", [2, 5, 20, 100, 1000, 20000])
def test_unimodal_lognormal_is_one_cluster(n):
    rng = np.random.default_rng(n)
    for rep in range(5):
        x = np.exp(rng.normal(math.log(80_000), 0.1, n)).astype(np.uint64)
        r = oracle.kde_group(x)
        assert r["n_clusters"] == 1, (n, rep)
        assert r["count"][0] == n
        assert r["p50_ns"][0] == statistics.median_low(x.tolist())
        assert r["p99_ns"][0] == _nearest_rank_p99(x)


@pytest.mark.parametrize("sizes", [(500, 200, 50), (60, 60, 60), (1000, 2000), (300, 400, 4000, 400)])
def test_lognormal_mixture_recovered(sizes):
    # components 2 octaves apart, each truncated to +-4 sigma (0.58 octave):
    # no sample of one component can fall inside another's range
    rng = np.random.default_rng(sum(sizes))
    comps = []
    for i, m in enumerate(sizes):
        z = np.clip(rng.normal(0, 1, m), -4, 4)
        comps.append(np.exp(math.log(30_000 * 4**i) + 0.1 * z).astype(np.uint64))
    r = oracle.kde_group(np.concatenate(comps))
    assert r["n_clusters"] == len(sizes)
    for i, c in enumerate(comps):
        assert r["count"][i] == len(c)
        assert r["p50_ns"][i] == statistics.median_low(c.tolist())
        assert r["p99_ns"][i] == _nearest_rank_p99(c)


def test_generator_modes_recovered():
    """Every (rank, step, kernel) group of the tiny trace whose duration
    scales each hold >= 10% of its events comes out as one cluster per scale,
    with the exact number of events at that scale."""
    trace = tracegen.make("tiny")
    cfg = trace.cfg
    ev = trace.fill_host()
    r = oracle.kde(ev, cfg.n_kernels, cfg.n_streams)
    assert r["bad_segments"] == 0
    T, K = cfg.tmpl_len, cfg.n_kernels
    reps = cfg.events_per_seg // T
    checked = multi = 0
    for k in range(K):
        modes, counts = np.unique(trace.tmpl_mode_pm[trace.tmpl_kid == k], return_counts=True)
        counts = counts * reps
        if counts.size == 0 or counts.min() * 10 < counts.sum():
            continue
        for g in range(cfg.n_segments):
            c = g * K + k
            assert r["n_clusters"][c] == len(modes), (g, k, modes, counts)
            assert list(r["count"][c][:len(modes)]) == counts.tolist(), (g, k)
            checked += 1
            multi += len(modes) > 1
    assert checked >= 32 * 40 and multi >= 32 * 8, (checked, multi)


def test_density_is_the_scaled_gaussian():
    # two spikes 10 octaves apart: near the lower one only its own kernel
    # contributes, so f(t) = N * round(65536 * phi(t / h) / phi(0)) with phi
    # the normal density (scipy) and h the reported quantised bandwidth
    from scipy.stats import norm
    N = 100_000
    r = oracle.kde_group(_spikes((2**20, N), (2**30, N)), debug=True)
    hq = r["bw_q8"] / 256.0
    T = int(hq * math.sqrt(2 * math.log(131072)))
    assert 640 > 2 * T + 2  # a zero plateau separates the spikes
    for t in range(0, T + 1):
        w = math.floor(65536 * norm.pdf(t, scale=hq) / norm.pdf(0, scale=hq) + 0.5)
        assert int(r["f"][t]) == N * w, t
    assert int(r["f"][T + 2]) == 0


def _brute_valleys(f):
    """Middle (rounded down) of every maximal run of equal values that is
    strictly below both neighbouring runs, inside the grid."""
    runs, j = [], 0
    f = [int(x) for x in f]
    while j < len(f):
        k = j
        while k + 1 < len(f) and f[k + 1] == f[j]:
            k += 1
        runs.append((j, k))
        j = k + 1
    out = []
    for i in range(1, len(runs) - 1):
        a, b = runs[i]
        if f[runs[i - 1][0]] > f[a] and f[runs[i + 1][0]] > f[a]:
            out.append((a + b) // 2)
    return out


@pytest.mark.parametrize("seed", range(6))
def test_valleys_are_strict_run_minima(seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(3, 400))
    k = int(rng.integers(1, 4))
    x = np.concatenate([np.exp(rng.normal(math.log(20_000 * 3**i), 0.3, n)) for i in range(k)]).astype(np.uint64)
    x = x[: max(3, len(x) - int(rng.integers(0, n)))]
    r = oracle.kde_group(x, debug=True)
    assert list(r["cand"]) == _brute_valleys(r["f"])


def test_plateau_valley_sits_mid_plateau():
    # 1e6 samples per spike: h ~ 5.6 steps, so the density is exactly zero on
    # most of the 200 steps between the spikes; the valley is the middle of
    # that zero run (100 steps from each extreme), which passes the spacing
    # filter, while the run's start (~28 steps in) would not
    N = 1_000_000
    r = oracle.kde_group(_spikes((2**20, N), (_lb(64 * 20 + 200), N)), debug=True)
    assert 100 in list(r["cand"])
    # the integer weights make terraces on the density's flanks; none of
    # them is a valley
    assert list(r["cand"]) == _brute_valleys(r["f"])
    assert r["n_clusters"] == 2 and list(r["count"][:2]) == [N, N]


def test_samples_on_the_valley_belong_to_the_lower_cluster():
    # equal spikes 100 steps apart plus two samples exactly halfway: the
    # density stays symmetric with its minimum on those samples' grid point
    b0 = 64 * 20
    r = oracle.kde_group(_spikes((_lb(b0), 20), (_lb(b0 + 50), 2), (_lb(b0 + 100), 20)), debug=True)
    assert list(r["cand"]) == [50]
    assert r["n_clusters"] == 2 and list(r["count"][:2]) == [22, 20]
    assert r["p99_ns"][0] == _lb(b0 + 50)


def test_spacing_filter_drops_the_shallower_of_two_close_valleys():
    # spikes at grid offsets 0, 400, 500, 600, 1000 with counts 2.5e5, 5e5,
    # 7.5e4, 2.5e5, 2.5e5 (h ~ 19 steps). The valleys around the small middle
    # spike lie ~90 steps apart (< gap 120); the one next to the larger
    # neighbour (offset 400) carries more of that neighbour's tail, so it is
    # the shallower and is dropped: the middle spike joins the 400 spike.
    # All other boundary distances are >= 200.
    b0 = 64 * 12
    counts = [250_000, 500_000, 75_000, 250_000, 250_000]
    offs = [0, 400, 500, 600, 1000]
    r = oracle.kde_group(_spikes(*[(_lb(b0 + o), c) for o, c in zip(offs, counts)]), gap=120)
    assert r["n_clusters"] == 4
    assert list(r["count"]) == [250_000, 575_000, 250_000, 250_000]
    assert list(r["p50_ns"]) == [_lb(b0), _lb(b0 + 400), _lb(b0 + 600), _lb(b0 + 1000)]
    assert r["p99_ns"][1] == _lb(b0 + 500)


def test_size_filter_small_cluster_between_equal_valleys_joins_the_upper():
    # zero-density valleys on both sides of a 4,000-sample spike (< 5% of
    # 204,000): both valleys have f = 0, the tie goes to the upper valley
    N = 100_000
    b0 = 64 * 12
    r = oracle.kde_group(_spikes((_lb(b0), N), (_lb(b0 + 300), 4000), (_lb(b0 + 600), N)), debug=True)
    assert r["f"][150] == 0 and r["f"][450] == 0
    assert r["n_clusters"] == 2 and list(r["count"][:2]) == [N, N + 4000]
    assert r["p50_ns"][1] == _lb(b0 + 600) and r["p50_ns"][0] == _lb(b0)


def test_size_filter_merges_the_first_of_equal_small_clusters_first():
    # clusters 4,000 | 4,000 | 100,000 (need 5,400): the first small one goes
    # first, into its only neighbour, and the merged 8,000 passes; merging the
    # second one first (into the large one, across the upper of two tied
    # zero-density valleys) would leave 4,000 alone and end with one cluster
    b0 = 64 * 12
    r = oracle.kde_group(_spikes((_lb(b0), 4000), (_lb(b0 + 300), 4000), (_lb(b0 + 600), 100_000)), debug=True)
    assert r["f"][150] == 0 and r["f"][450] == 0
    assert r["n_clusters"] == 2 and list(r["count"][:2]) == [8000, 100_000]
