/*
 * ARGUS oracle, part 2: per-(rank, step, kernel) duration clustering by
 * valleys of a kernel density estimate, summarised as (count, p50, p99)
 * triples per cluster.
 *
 * TEST INFRASTRUCTURE ONLY, like the rest of liboracle: only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg load it. It shares no
 * source with the HIP kernels.
 *
 * Section 5.2 ("Online Statistical Compression of Kernel Traces"): the
 * durations of one (kernel, stream, rank) group in one window are log
 * transformed; a Gaussian KDE (Eq. 1) with bandwidth h = 1.06 sigma n^(-1/5)
 * is evaluated on an equally spaced grid; its local minima are candidate
 * cluster boundaries; a cluster-level filter (enough samples on both sides of
 * a valley) and a spacing filter (adjacent boundaries far enough apart in
 * duration) remove noise valleys; each remaining cluster reports its count,
 * median and 99th percentile. This file follows those steps in that order.
 *
 * Readings (the paper gives no grid, no filter thresholds and no tie rules):
 *  - grid: x = floor(2^s log2 d') where d' keeps the 24 leading significant
 *    bits of the duration d (exact for d < 2^24 ns) and d = 0 counts as 1;
 *    one grid point per integer x between the smallest and largest x of the
 *    group, s = 6 by default (64 points per octave);
 *  - sigma: sample standard deviation (n - 1) of the grid values x;
 *    h = (1.06 sqrt(var)) n^(-1/5) in grid steps, quantised to
 *    H = floor(256 h + 0.5) (units of 1/256 step); H = 0 means no valleys;
 *    n^(-1/5) is the double nearest to the real fifth root, decided by exact
 *    integer comparisons (a math library's pow(n, -0.2) takes the exponent
 *    as the double nearest -0.2 and rounds differently from one library to
 *    the next);
 *  - binned KDE with integer weights w(t) = floor(65536 exp(-t^2 / (2 (H/256)^2)) + 0.5)
 *    for grid distance t; f(j) = sum_b c(b) w(|j - b|) over the histogram c
 *    (the 1/(n h sqrt(2 pi)) factor does not move minima);
 *  - valley: a maximal run of equal f values, strictly lower than its two
 *    neighbours, inside the grid; its position is the middle of the run
 *    (rounded down); samples at or below a boundary go to the lower cluster;
 *  - cluster-level filter: while the smallest cluster (first one on ties) has
 *    fewer than max(min_count, ceil(frac_pm n / 1000)) samples, drop one of
 *    its bounding valleys: its only one at either end, else the shallower
 *    (larger f; the upper one on ties);
 *  - spacing filter: boundaries are the group's smallest grid value, the
 *    valleys, and its largest grid value; while two adjacent ones are fewer
 *    than gap steps apart (first such pair), drop the valley of the pair, or
 *    the shallower of two valleys (the upper one on ties);
 *  - at most KDE_MAXC clusters: drop the shallowest valley (the upper one on
 *    ties) until that holds;
 *  - p50 = lower median, p99 = nearest-rank 99th percentile (element
 *    ceil(0.99 m) of the m sorted durations) of each cluster's raw durations.
 *
 * The floored samples, the quantised bandwidth and the integer weights make
 * this an approximation of Eq. 1. Its distance from Eq. 1 as printed (float64
 * Gaussian KDE of the raw logs with the unquantised bandwidth, same valley and
 * filter rules) is measured and bounded in tests/test_oracle_kde_eq1.py: the
 * same number of clusters in every group tested, boundaries displaced only
 * across empty cells, by one grid step, or inside a valley bottom where Eq. 1
 * itself is flat to 1e-3, and at most 6.5e-4 of the samples assigned to
 * another cluster.
 *
 * Parity pins (tests/test_oracle_kde.py): the threshold table and grid
 * function against exact big-integer logarithms; bandwidth against the closed
 * form of two-spike data; hand-worked spike patterns for each filter rule and
 * the cluster cap; recovery of lognormal mixtures whose components cannot
 * overlap; and recovery of the generator's planted per-position duration
 * modes in seeded traces.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;

#define KDE_MAXC 4

/* th[t] = ceil(2^(23 + t/64)) for t in [0, 64): the smallest 24-bit mantissa
 * whose base-2 logarithm has fractional part >= t/64. */
static void kde_thresholds(uint32_t* th) {
  for (int t = 0; t < 64; t++) th[t] = (uint32_t)ceill(exp2l(23.0L + (long double)t / 64.0L));
}

void orc_kde_thresholds(uint32_t* th) { kde_thresholds(th); }

/* floor(64 log2 d') with d' the 24 leading significant bits of d. */
static int kde_bin64(uint64_t d, const uint32_t* th) {
  if (d < 2) return 0;
  int e = 63 - __builtin_clzll(d);
  uint32_t m = e >= 23 ? (uint32_t)(d >> (e - 23)) : (uint32_t)(d << (23 - e));
  int t = 0;
  while (t < 63 && m >= th[t + 1]) t++;
  return e * 64 + t;
}

int orc_kde_bin(uint64_t d, int32_t sub_bits) {
  uint32_t th[64];
  kde_thresholds(th);
  return kde_bin64(d, th) >> (6 - sub_bits);
}

/* orc_kde_bin at full resolution (64 grid points per octave) for m durations. */
void orc_kde_bin_many(const uint64_t* d, int64_t m, int32_t* out) {
  uint32_t th[64];
  kde_thresholds(th);
  for (int64_t i = 0; i < m; i++) out[i] = kde_bin64(d[i], th);
}

static int cmp_u64(const void* a, const void* b) {
  uint64_t x = *(const uint64_t*)a, y = *(const uint64_t*)b;
  return x < y ? -1 : x > y;
}

/* ---- n^(-1/5), the double nearest to the real value ----------------------
 * Whether the fifth root z = n^(-1/5) lies above or below a dyadic number
 * m = c 2^k (c odd) is decided exactly: z < m iff c^5 n > 2^(-5k). The product
 * is formed in 32-bit limbs (c < 2^55, n < 2^33: under 320 bits). */
#define MP_LIMBS 12

/* a *= m (a: MP_LIMBS little-endian 32-bit limbs) */
static void mp_mul_u32(uint32_t* a, uint32_t m) {
  uint64_t carry = 0;
  for (int i = 0; i < MP_LIMBS; i++) {
    uint64_t v = (uint64_t)a[i] * m + carry;
    a[i] = (uint32_t)v;
    carry = v >> 32;
  }
}

/* a *= m for a 64-bit m: a * lo + (a * hi) << 32 */
static void mp_mul_u64(uint32_t* a, uint64_t m) {
  uint32_t lo[MP_LIMBS], hi[MP_LIMBS];
  memcpy(lo, a, sizeof(lo));
  memcpy(hi, a, sizeof(hi));
  mp_mul_u32(lo, (uint32_t)m);
  mp_mul_u32(hi, (uint32_t)(m >> 32));
  uint64_t carry = 0;
  for (int i = 0; i < MP_LIMBS; i++) {
    uint64_t v = (uint64_t)lo[i] + (i > 0 ? hi[i - 1] : 0) + carry;
    a[i] = (uint32_t)v;
    carry = v >> 32;
  }
}

/* sign of c^5 n - 2^e: 1, 0 or -1 (c, n >= 1, 0 <= e < 32 MP_LIMBS) */
static int fifth_cmp(uint64_t c, uint64_t n, int e) {
  uint32_t a[MP_LIMBS] = {0};
  a[0] = 1;
  for (int r = 0; r < 5; r++) mp_mul_u64(a, c);
  mp_mul_u64(a, n);
  int top = MP_LIMBS - 1;
  while (top > 0 && a[top] == 0) top--;
  int bits = 32 * top + (a[top] ? 32 - __builtin_clz(a[top]) : 0);
  if (bits != e + 1) return bits > e + 1 ? 1 : -1; /* 2^e has e + 1 bits */
  for (int i = 0; i < MP_LIMBS; i++) {             /* same length: equal iff only the top bit is set */
    uint32_t want = i == e / 32 ? (1u << (e % 32)) : 0u;
    if (a[i] != want) return 1;
  }
  return 0;
}

/* The double nearest to n^(-1/5) for 1 <= n < 2^33. y = M 2^q with M in
 * [2^52, 2^53); its rounding interval is bounded by the midpoints to its
 * neighbours, (2M + 1) 2^(q-1) above and (2M - 1) 2^(q-1) below, or
 * (4M - 1) 2^(q-2) below when M = 2^52 (the neighbour below lies in the next
 * lower binade). z is irrational or a reciprocal integer, never a midpoint. */
static double kde_pw(int64_t n) {
  double y = pow((double)n, -0.2); /* a start within a few units in the last place */
  for (;;) {
    int q;
    double f = frexp(y, &q); /* y = f 2^q, f in [0.5, 1) */
    uint64_t M = (uint64_t)ldexp(f, 53);
    q -= 53;
    /* z < upper midpoint: (2M + 1)^5 n > 2^(5 (1 - q)) */
    if (fifth_cmp(2 * M + 1, (uint64_t)n, 5 * (1 - q)) <= 0) {
      y = nextafter(y, INFINITY);
      continue;
    }
    /* z > lower midpoint: (2M - 1)^5 n < 2^(5 (1 - q)), or (4M - 1)^5 n < 2^(5 (2 - q)) */
    int below = M == (1ull << 52) ? fifth_cmp(4 * M - 1, (uint64_t)n, 5 * (2 - q))
                                  : fifth_cmp(2 * M - 1, (uint64_t)n, 5 * (1 - q));
    if (below >= 0) {
      y = nextafter(y, 0.0);
      continue;
    }
    return y;
  }
}

/* Step 2's bandwidth: H = floor(256 h + 0.5) with h = 1.06 sqrt(var) n^(-1/5)
 * in grid steps, n^(-1/5) the double nearest to the real value. */
static int64_t kde_bw_q8(double var, int64_t n) {
  double h = 1.06 * sqrt(var) * kde_pw(n);
  return (int64_t)floor(h * 256.0 + 0.5);
}

/* Step 3's integer Gaussian weight of grid distance t for bandwidth H. */
static uint32_t kde_weight(int64_t t, int64_t H) {
  double a = (double)(32768LL * t * t) / (double)(H * H);
  return (uint32_t)floor(65536.0 * exp(-a) + 0.5);
}

/* Test access to the floating-point steps: the weights of t = 0 .. nt-1 for
 * bandwidth H, n^-0.2, and H from (var, n). */
void orc_kde_weights(int64_t H, int32_t nt, uint32_t* w) {
  for (int32_t t = 0; t < nt; t++) w[t] = kde_weight(t, H);
}
double orc_kde_root5(int64_t n) { return kde_pw(n); }
int64_t orc_kde_bw_q8(double var, int64_t n) { return kde_bw_q8(var, n); }

/* The same over arrays: weights of t = 0 .. off[i+1]-off[i]-1 for each H[i]
 * into w[off[i] ..]; n^-0.2 and H of (var[i], n[i]). */
void orc_kde_weights_many(const int64_t* H, const int64_t* off, int32_t nH, uint32_t* w) {
  for (int32_t i = 0; i < nH; i++)
    for (int64_t t = 0; t < off[i + 1] - off[i]; t++) w[off[i] + t] = kde_weight(t, H[i]);
}
void orc_kde_root5_many(const int64_t* n, int64_t m, double* out) {
  for (int64_t i = 0; i < m; i++) out[i] = kde_pw(n[i]);
}
void orc_kde_bw_q8_many(const double* var, const int64_t* n, int64_t m, int64_t* out) {
  for (int64_t i = 0; i < m; i++) out[i] = kde_bw_q8(var[i], n[i]);
}

/* Remove valley i from the position / value lists of length *m. */
static void drop(int32_t* pos, uint64_t* val, int32_t* m, int32_t i) {
  for (int32_t q = i; q + 1 < *m; q++) {
    pos[q] = pos[q + 1];
    val[q] = val[q + 1];
  }
  (*m)--;
}

/*
 * One group: d[0..n) sorted ascending. Writes n_clusters, and per cluster
 * count / p50 / p99 (KDE_MAXC slots, unused ones zero); bw_q8 = H; n_cand =
 * number of valleys before filtering.
 */
static void kde_group(int64_t n, const uint64_t* d, int32_t s, int32_t frac_pm, int32_t min_count, int32_t gap,
                      const uint32_t* th, uint8_t* n_clusters, uint32_t* cnt, int64_t* p50, int64_t* p99,
                      int32_t* bw_q8, int32_t* n_cand, uint64_t* f_dbg, int32_t* cand_dbg) {
  for (int q = 0; q < KDE_MAXC; q++) {
    cnt[q] = 0;
    p50[q] = 0;
    p99[q] = 0;
  }
  *bw_q8 = 0;
  *n_cand = 0;
  if (n == 0) {
    *n_clusters = 0;
    return;
  }
  /* 1. log transform onto the grid */
  int32_t lo = kde_bin64(d[0], th) >> (6 - s);
  int32_t hi = kde_bin64(d[n - 1], th) >> (6 - s);
  int32_t G = hi - lo + 1;
  uint64_t* c = calloc((size_t)G, sizeof(uint64_t));
  uint64_t s1 = 0, s2 = 0;
  for (int64_t i = 0; i < n; i++) {
    uint64_t x = (uint64_t)((kde_bin64(d[i], th) >> (6 - s)) - lo);
    c[x]++;
    s1 += x;
    s2 += x * x;
  }

  /* 2. bandwidth (Scott's rule as printed), in grid steps, quantised */
  int64_t H = 0;
  if (n >= 2) {
    u128 V = (u128)n * s2 - (u128)s1 * s1;
    double var = (double)V / ((double)n * (double)(n - 1));
    H = kde_bw_q8(var, n);
  }
  *bw_q8 = (int32_t)H;

  /* 3. density on the grid and its valleys */
  int32_t m = 0;
  int32_t* pos = NULL;
  uint64_t* val = NULL;
  if (H > 0 && G >= 3) {
    uint32_t* w = malloc((size_t)G * sizeof(uint32_t));
    int32_t T = -1;
    for (int32_t t = 0; t < G; t++) {
      uint32_t wt = kde_weight(t, H);
      if (wt == 0) break;
      w[t] = wt;
      T = t;
    }
    uint64_t* f = calloc((size_t)G, sizeof(uint64_t));
    for (int32_t j = 0; j < G; j++) {
      int32_t b0 = j - T > 0 ? j - T : 0, b1 = j + T < G - 1 ? j + T : G - 1; /* w(t) = 0 for t > T */
      for (int32_t b = b0; b <= b1; b++) f[j] += c[b] * w[j > b ? j - b : b - j];
    }
    if (f_dbg) memcpy(f_dbg, f, (size_t)G * sizeof(uint64_t));
    pos = malloc((size_t)G * sizeof(int32_t));
    val = malloc((size_t)G * sizeof(uint64_t));
    int32_t j = 1;
    while (j <= G - 2) {
      if (f[j] < f[j - 1]) {
        int32_t k = j;
        while (k + 1 < G && f[k + 1] == f[j]) k++;
        if (k + 1 < G && f[k + 1] > f[j]) {
          pos[m] = (j + k) / 2;
          val[m] = f[j];
          m++;
        }
        j = k + 1;
      } else {
        j++;
      }
    }
    free(f);
    free(w);
  }
  *n_cand = m;
  if (cand_dbg)
    for (int32_t q = 0; q < m; q++) cand_dbg[q] = pos[q];

  /* 4. cluster-level filter */
  int64_t need = ((int64_t)frac_pm * n + 999) / 1000;
  if (need < min_count) need = min_count;
  while (m > 0) {
    int32_t best = 0;
    uint64_t best_size = 0;
    for (int32_t q = 0; q <= m; q++) {
      int32_t a = q == 0 ? 0 : pos[q - 1] + 1, b = q == m ? G - 1 : pos[q];
      uint64_t sz = 0;
      for (int32_t x = a; x <= b; x++) sz += c[x];
      if (q == 0 || sz < best_size) {
        best = q;
        best_size = sz;
      }
    }
    if (best_size >= (uint64_t)need) break;
    if (best == 0)
      drop(pos, val, &m, 0);
    else if (best == m)
      drop(pos, val, &m, m - 1);
    else
      drop(pos, val, &m, val[best - 1] > val[best] ? best - 1 : best);
  }

  /* 5. spacing filter over [lowest value, valleys..., highest value] */
  while (m > 0) {
    int32_t hit = -1;
    for (int32_t q = 0; q <= m && hit < 0; q++) {
      int32_t a = q == 0 ? 0 : pos[q - 1], b = q == m ? G - 1 : pos[q];
      if (b - a < gap) hit = q;
    }
    if (hit < 0) break;
    if (hit == 0)
      drop(pos, val, &m, 0);
    else if (hit == m)
      drop(pos, val, &m, m - 1);
    else
      drop(pos, val, &m, val[hit - 1] > val[hit] ? hit - 1 : hit);
  }

  /* 6. cluster cap */
  while (m > KDE_MAXC - 1) {
    int32_t sh = 0;
    for (int32_t q = 1; q < m; q++)
      if (val[q] >= val[sh]) sh = q;
    drop(pos, val, &m, sh);
  }

  /* 7. per-cluster count and order statistics (d is sorted and the grid
   * value is monotone in d, so each cluster is a contiguous run of d) */
  int64_t first = 0;
  for (int32_t q = 0; q <= m; q++) {
    int32_t a = q == 0 ? 0 : pos[q - 1] + 1, b = q == m ? G - 1 : pos[q];
    uint64_t sz = 0;
    for (int32_t x = a; x <= b; x++) sz += c[x];
    cnt[q] = (uint32_t)sz;
    p50[q] = (int64_t)d[first + ((int64_t)sz - 1) / 2];
    p99[q] = (int64_t)d[first + (99 * (int64_t)sz + 99) / 100 - 1];
    first += (int64_t)sz;
  }
  *n_clusters = (uint8_t)(m + 1);
  free(pos);
  free(val);
  free(c);
}

/* One group given its durations in any order (hand-built test cases).
 * f_dbg (grid length) and cand_dbg (valley positions before filtering, grid
 * indices) may be NULL; they expose the density for tests. */
void orc_kde_group(int64_t n, const uint64_t* durations, int32_t sub_bits, int32_t frac_pm, int32_t min_count,
                   int32_t gap, uint8_t* n_clusters, uint32_t* cnt, int64_t* p50, int64_t* p99, int32_t* bw_q8,
                   int32_t* n_cand, uint64_t* f_dbg, int32_t* cand_dbg) {
  uint32_t th[64];
  kde_thresholds(th);
  uint64_t* d = malloc((size_t)(n > 0 ? n : 1) * sizeof(uint64_t));
  if (n > 0) {
    memcpy(d, durations, (size_t)n * sizeof(uint64_t));
    qsort(d, (size_t)n, sizeof(uint64_t), cmp_u64);
  }
  kde_group(n, d, sub_bits, frac_pm, min_count, gap, th, n_clusters, cnt, p50, p99, bw_q8, n_cand, f_dbg,
            cand_dbg);
  free(d);
}

/*
 * Every (segment, kernel) group of a raw event trace. Validity of a record
 * is the summarizer's rule (known kernel id and stream, start >= 0,
 * end >= start); d = end - start. Outputs are [n_seg][K] and
 * [n_seg][K][KDE_MAXC]. Returns the number of malformed segments (treated as
 * empty).
 */
int64_t orc_kde(int64_t n_seg, int32_t K, int32_t NS, int64_t n_events, const int32_t* kid, const int32_t* stream,
                const int64_t* start, const int64_t* end, const int64_t* seg_off, int32_t sub_bits,
                int32_t frac_pm, int32_t min_count, int32_t gap, uint8_t* n_clusters, uint32_t* cnt,
                int64_t* p50, int64_t* p99, int32_t* bw_q8) {
  uint32_t th[64];
  kde_thresholds(th);
  int64_t bad = 0;
  for (int64_t g = 0; g < n_seg; g++) {
    int64_t lo = seg_off[g], hi = seg_off[g + 1];
    if (!(lo >= 0 && lo <= hi && hi <= n_events && (hi - lo) <= (int64_t)UINT32_MAX)) {
      bad++;
      lo = hi = 0;
    }
    /* group the segment's valid durations by kernel id (counting sort) */
    int64_t* off = calloc((size_t)K + 1, sizeof(int64_t));
    for (int64_t i = lo; i < hi; i++) {
      int valid = kid[i] >= 0 && kid[i] < K && stream[i] >= 0 && stream[i] < NS && start[i] >= 0 &&
                  end[i] >= start[i];
      if (valid) off[kid[i] + 1]++;
    }
    for (int32_t k = 0; k < K; k++) off[k + 1] += off[k];
    uint64_t* d = malloc((size_t)(off[K] > 0 ? off[K] : 1) * sizeof(uint64_t));
    int64_t* fill = malloc((size_t)K * sizeof(int64_t));
    memcpy(fill, off, (size_t)K * sizeof(int64_t));
    for (int64_t i = lo; i < hi; i++) {
      int valid = kid[i] >= 0 && kid[i] < K && stream[i] >= 0 && stream[i] < NS && start[i] >= 0 &&
                  end[i] >= start[i];
      if (valid) d[fill[kid[i]]++] = (uint64_t)end[i] - (uint64_t)start[i];
    }
    for (int32_t k = 0; k < K; k++) {
      int64_t c = g * K + k, n = off[k + 1] - off[k];
      int32_t n_cand;
      qsort(d + off[k], (size_t)n, sizeof(uint64_t), cmp_u64);
      kde_group(n, d + off[k], sub_bits, frac_pm, min_count, gap, th, n_clusters + c, cnt + c * KDE_MAXC,
                p50 + c * KDE_MAXC, p99 + c * KDE_MAXC, bw_q8 + c, &n_cand, NULL, NULL);
    }
    free(fill);
    free(d);
    free(off);
  }
  return bad;
}
