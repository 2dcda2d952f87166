/*
 * ARGUS oracle, part 3: cross-rank Wasserstein-1 deviation scores over the
 * per-cell duration clusters, and the IQR upper fence on those scores.
 *
 * TEST INFRASTRUCTURE ONLY, like the rest of liboracle: only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg load it. It shares no
 * source with the HIP kernels.
 *
 * Section 6.2 ("CDF reconstruction", "Wasserstein-1 distance and anomaly
 * identification", "Cross-rank IQR anomaly determination"), Eq. 2 - 4, for
 * every (step, kernel) over the ranks where the kernel has clusters:
 *   - each cluster c of rank r is a lognormal with mu = ln p50 and
 *     sigma = (ln p99 - ln p50) / 2.326; the rank's CDF is the count-weighted
 *     mixture F_r(x) = sum_c w_c Phi((ln x - mu_c) / sigma_c) (Eq. 2);
 *   - W1(F_a, F_b) = integral of |F_a - F_b| dx (Eq. 3) by the trapezoid rule
 *     on a log-uniform grid;
 *   - the deviation score of rank a is its mean W1 to the other ranks;
 *   - ranks whose score exceeds Q3 + alpha (Q3 - Q1) are flagged (Eq. 4).
 *
 * Readings (the paper fixes no grid, no quartile rule and no handling of
 * degenerate clusters):
 *   - durations below 1 ns count as 1 ns (p' = max(p, 1)); a cluster with
 *     p99 = p50 is a point mass (Phi becomes the unit step at p50);
 *   - grid: G points x_i = exp(ln lo + i (ln hi - ln lo) / (G - 1)) with
 *     lo = max(1, min floor(p50^2 / p99)) and hi = max ceil(p99^2 / p50) over
 *     all clusters of the present ranks (the lognormal's mirror of its 99th
 *     percentile below the median, and its 99.99th percentile); |F_a - F_b|
 *     is taken as 0 outside [lo, hi];
 *   - trapezoid weights w_i = (x_{i+1} - x_{i-1}) / 2 with x_{-1} = x_0 and
 *     x_G = x_{G-1};
 *   - CDF values are taken to 16-bit fixed point, q = min(65535,
 *     floor(65536 F)), before differencing, so the per-point sums of |q_a -
 *     q_b| are exact integers; score_a = sum_i w_i S_ai / (65536 (n - 1)),
 *     accumulated in ascending i, S_ai = sum_b |q_ai - q_bi|;
 *   - Q1, Q3 = lower nearest-rank quartiles v[(n-1)/4], v[3(n-1)/4] of the
 *     sorted scores (the same rule as the cross-rank step); no scores when
 *     fewer than min_ranks ranks are present.
 *   - a cell takes part ("is present") iff it has 1 to W1_MAXC clusters whose
 *     counts sum to at least 1; a cell with more than W1_MAXC clusters, or
 *     with clusters of total count 0, is a malformed record: it is left out
 *     like an absent cell and counted in the return value.
 *
 * Parity pins (tests/test_oracle_w1.py): the CDF at p50 and p99 against the
 * normal distribution; W1 of two equal-shape lognormals against the closed
 * form (difference of means); the score relation of one outlier among equal
 * ranks; hand-worked quartile / fence cases; brute-force recomputation on
 * tiny inputs; recovery of planted stragglers through oracle clusters.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;

#define W1_MAXC 4
#define W1_Z99 2.326

static int cmp_f64(const void* a, const void* b) {
  double x = *(const double*)a, y = *(const double*)b;
  return x < y ? -1 : x > y;
}

/* Fixed-point CDF of one rank's mixture at log-duration u. */
static uint32_t mixture_q(int ncl, const uint32_t* count, const int64_t* p50, const int64_t* p99, double u) {
  uint64_t tot = 0;
  for (int c = 0; c < ncl; c++) tot += count[c];
  double F = 0.0;
  for (int c = 0; c < ncl; c++) {
    double a = p50[c] > 1 ? (double)p50[c] : 1.0;
    double b = p99[c] > 1 ? (double)p99[c] : 1.0;
    if (b < a) b = a;
    double mu = log(a);
    double sigma = (log(b) - mu) / W1_Z99;
    double phi;
    if (sigma > 0.0)
      phi = 0.5 * erfc((mu - u) / (sigma * M_SQRT2));
    else
      phi = u >= mu ? 1.0 : 0.0;
    F += ((double)count[c] / (double)tot) * phi;
  }
  double v = floor(F * 65536.0);
  return v >= 65535.0 ? 65535u : (uint32_t)v;
}

/* floor(a^2 / b) and ceil(b^2 / a) for 1 <= a <= b, exact (the latter capped
 * at 2^63 - 1). */
static uint64_t lo_bound(uint64_t a, uint64_t b) { return (uint64_t)(((u128)a * a) / b); }
static uint64_t hi_bound(uint64_t a, uint64_t b) {
  u128 num = (u128)b * b;
  u128 q = (num + a - 1) / a;
  return q > (u128)INT64_MAX ? (uint64_t)INT64_MAX : (uint64_t)q;
}

/* 1 if the cell's cluster record is usable, 0 if absent, -1 if malformed. */
static int cell_state(uint8_t ncl, const uint32_t* count) {
  if (ncl == 0) return 0;
  if (ncl > W1_MAXC) return -1;
  uint64_t tot = 0;
  for (int c = 0; c < ncl; c++) tot += count[c];
  return tot > 0 ? 1 : -1;
}

/*
 * Inputs are the per-cell cluster outputs, [R][S][K] and [R][S][K][W1_MAXC].
 * Outputs per (s, k): n_present, lo_ns, hi_ns, q1, q3, fence, n_flag; per
 * cell: score, flag. Returns the number of malformed cells.
 */
int orc_w1(int32_t R, int32_t S, int32_t K, const uint8_t* n_clusters, const uint32_t* count, const int64_t* p50,
           const int64_t* p99, int32_t G, int32_t min_ranks, int32_t alpha_pm, uint32_t* n_present, int64_t* lo_ns,
           int64_t* hi_ns, double* q1, double* q3, double* fence, uint32_t* n_flag, double* score, uint8_t* flag) {
  int32_t* ranks = malloc((size_t)R * sizeof(int32_t));
  uint32_t* q = malloc((size_t)R * (size_t)G * sizeof(uint32_t));
  double* sc = malloc((size_t)R * sizeof(double));
  double* sorted = malloc((size_t)R * sizeof(double));
  double* x = malloc((size_t)G * sizeof(double));
  int malformed = 0;
  for (int32_t s = 0; s < S; s++)
    for (int32_t k = 0; k < K; k++) {
      int64_t sk = (int64_t)s * K + k;
      int32_t n = 0;
      for (int32_t r = 0; r < R; r++) {
        int64_t c = ((int64_t)r * S + s) * K + k;
        score[c] = 0.0;
        flag[c] = 0;
        int st = cell_state(n_clusters[c], count + c * W1_MAXC);
        if (st > 0) ranks[n++] = r;
        if (st < 0) malformed++;
      }
      n_present[sk] = (uint32_t)n;
      lo_ns[sk] = hi_ns[sk] = 0;
      q1[sk] = q3[sk] = fence[sk] = 0.0;
      n_flag[sk] = 0;
      if (n < min_ranks || n < 2) continue;

      /* grid bounds over every cluster of the present ranks */
      uint64_t lo = UINT64_MAX, hi = 0;
      for (int32_t i = 0; i < n; i++) {
        int64_t c = ((int64_t)ranks[i] * S + s) * K + k;
        for (int cl = 0; cl < n_clusters[c]; cl++) {
          uint64_t a = p50[c * W1_MAXC + cl] > 1 ? (uint64_t)p50[c * W1_MAXC + cl] : 1;
          uint64_t b = p99[c * W1_MAXC + cl] > 1 ? (uint64_t)p99[c * W1_MAXC + cl] : 1;
          if (b < a) b = a;
          uint64_t l = lo_bound(a, b), h = hi_bound(a, b);
          if (l < lo) lo = l;
          if (h > hi) hi = h;
        }
      }
      if (lo < 1) lo = 1;
      lo_ns[sk] = (int64_t)lo;
      hi_ns[sk] = (int64_t)hi;

      /* log-uniform grid and the fixed-point CDF of every present rank */
      double lnlo = log((double)lo), lnhi = log((double)hi);
      double du = (lnhi - lnlo) / (double)(G - 1);
      for (int32_t g = 0; g < G; g++) x[g] = exp(lnlo + (double)g * du);
      for (int32_t i = 0; i < n; i++) {
        int64_t c = ((int64_t)ranks[i] * S + s) * K + k;
        for (int32_t g = 0; g < G; g++)
          q[(size_t)i * G + g] = mixture_q(n_clusters[c], count + c * W1_MAXC, p50 + c * W1_MAXC,
                                           p99 + c * W1_MAXC, lnlo + (double)g * du);
      }

      /* mean W1 to the other ranks, straight from the pairwise definition */
      for (int32_t i = 0; i < n; i++) {
        double acc = 0.0;
        for (int32_t g = 0; g < G; g++) {
          uint64_t sum = 0;
          for (int32_t j = 0; j < n; j++) {
            uint32_t u = q[(size_t)i * G + g], v = q[(size_t)j * G + g];
            sum += u > v ? u - v : v - u;
          }
          double w = (x[g + 1 < G ? g + 1 : G - 1] - x[g > 0 ? g - 1 : 0]) / 2.0;
          acc += w * (double)sum;
        }
        sc[i] = acc / (65536.0 * (double)(n - 1));
      }

      /* IQR upper fence over the scores */
      memcpy(sorted, sc, (size_t)n * sizeof(double));
      qsort(sorted, (size_t)n, sizeof(double), cmp_f64);
      double a1 = sorted[(n - 1) / 4], a3 = sorted[3 * (n - 1) / 4];
      double fz = a3 + (double)alpha_pm * (a3 - a1) / 1000.0;
      q1[sk] = a1;
      q3[sk] = a3;
      fence[sk] = fz;
      uint32_t nf = 0;
      for (int32_t i = 0; i < n; i++) {
        int64_t c = ((int64_t)ranks[i] * S + s) * K + k;
        score[c] = sc[i];
        if (sc[i] > fz) {
          flag[c] = 1;
          nf++;
        }
      }
      n_flag[sk] = nf;
    }
  free(x);
  free(sorted);
  free(sc);
  free(q);
  free(ranks);
  return malformed;
}

/* The fixed-point mixture CDF of one rank at duration x (tests). */
uint32_t orc_w1_cdf_q(int32_t ncl, const uint32_t* count, const int64_t* p50, const int64_t* p99, double x) {
  return mixture_q(ncl, count, p50, p99, log(x));
}

/* The same at log-duration u, as the score takes it at grid point g:
 * u = ln lo + g (ln hi - ln lo) / (G - 1) (tests). */
uint32_t orc_w1_cdf_q_at(int32_t ncl, const uint32_t* count, const int64_t* p50, const int64_t* p99, double u) {
  return mixture_q(ncl, count, p50, p99, u);
}
