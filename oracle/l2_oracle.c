/*
 * ARGUS oracle, part 4: parallelism-group-aware routing and the L2 coefficient
 * of variation / z-score comparison.
 *
 * TEST INFRASTRUCTURE ONLY, like the rest of liboracle: only the test suite,
 * the smoke check and the benchmark's CPU-baseline leg load it. It shares no
 * source with the HIP kernels.
 *
 * Section 6.1 (routing table, Table "routing") and Appendix B ("L2: CV and
 * z-score computation", Eq. 5): every event is compared only among the ranks
 * of the parallelism group the routing table assigns it to. For the average
 * durations {x_r} of one event on the ranks r of one group G in one window:
 *   mu = (1/|G|) sum x_r,  sigma = sqrt(sum (x_r - mu)^2 / (|G| - 1)),
 *   CV = sigma / mu: balanced below 0.02, mild imbalance below 0.05, severe
 *   imbalance otherwise; z_r = (x_r - mu) / sigma; a rank whose z exceeds the
 *   threshold is a straggler.
 *
 * Readings (the paper gives no z threshold, no minimum group size and no
 * representation of the groups):
 *   - events are the summaries' kernel ids; the window is one step; x_r is
 *     the exact integer mean floor(sum / count) of the rank's events (the
 *     sum read as unsigned), over ranks with count >= 1 and x_r < 2^40 ns
 *     (values at or above 2^40 are out of the domain: left out, status bit);
 *   - route[e] names the parallelism dimension of event e (0xFF: the event
 *     is not compared); each dimension's groups are given as lists of member
 *     ranks (offsets into a member array of R entries); a group whose range
 *     is not inside [0, R] with start <= end is malformed and skipped, a
 *     member id outside [0, R) is skipped (status bit 1); a rank listed more
 *     than once in one dimension counts only at its first listing (lowest
 *     group, then lowest position; status bit 2);
 *   - a group is evaluated when it has at least min_group present ranks
 *     (min_group >= 2: sigma needs two values);
 *   - every decision is exact: with n ranks, S = sum x and Q = sum x^2 as
 *     integers and D = n Q - S^2 (= n (n-1) sigma^2), CV < c_pm / 1000
 *     iff S > 0 and n D 10^6 < c_pm^2 (n - 1) S^2 (S = 0 is balanced), and
 *     z_r > z_pm / 1000 iff n x_r > S and (n x_r - S)^2 (n - 1) 10^6 >
 *     z_pm^2 n D (256-bit products);
 *   - reported values: mean = (double)S / n, std = sqrt((double)D / (n (n -
 *     1))), cv = std / mean (0 when mean = 0), z = (float)((x - mean) / std)
 *     (0 when std = 0), each a double operation in the order written.
 *
 * Parity pins (tests/test_oracle_l2.py): exact rational brute force
 * (fractions, statistics.variance) of every class and flag on random groups;
 * numpy mean / std(ddof=1) for the reported values; the closed form z =
 * (n - 1) / sqrt(n) of one outlier among equal values (flagged iff n >= 11 at
 * z > 3); class boundaries worked by hand; routing, membership and domain
 * rules; recovery of planted stragglers inside their data-parallel groups.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;

#define L2_DOMAIN (1ull << 40)
#define L2_NOT_EVALUATED 0xFF

/* 256-bit unsigned value as two 128-bit halves */
typedef struct {
  u128 hi, lo;
} u256;

static u256 mul128(u128 a, u128 b) {
  uint64_t a0 = (uint64_t)a, a1 = (uint64_t)(a >> 64), b0 = (uint64_t)b, b1 = (uint64_t)(b >> 64);
  u128 p00 = (u128)a0 * b0, p01 = (u128)a0 * b1, p10 = (u128)a1 * b0, p11 = (u128)a1 * b1;
  u128 mid = (p00 >> 64) + (uint64_t)p01 + (uint64_t)p10;
  u256 r;
  r.lo = (mid << 64) | (uint64_t)p00;
  r.hi = p11 + (p01 >> 64) + (p10 >> 64) + (mid >> 64);
  return r;
}

static int lt256(u256 a, u256 b) { return a.hi < b.hi || (a.hi == b.hi && a.lo < b.lo); }

int orc_l2(int32_t R, int32_t S, int32_t E, const uint32_t* count, const int64_t* sum_ns, const uint8_t* route,
           const int32_t* group_off, const int32_t* members, int32_t n_dims, int32_t max_groups, int32_t min_group,
           int32_t cv_mild_pm, int32_t cv_severe_pm, int32_t z_pm, uint32_t* n_out, double* mean_out,
           double* std_out, double* cv_out, uint8_t* cls_out, uint32_t* nstrag_out, float* z_out,
           uint8_t* flags_out) {
  int status = 0;
  int64_t* owner = malloc((size_t)(n_dims > 0 ? n_dims : 1) * (size_t)R * sizeof(int64_t));
  int64_t* xs = malloc((size_t)R * sizeof(int64_t));
  int32_t* rk = malloc((size_t)R * sizeof(int32_t));

  /* membership: a rank's first listing in a dimension (lowest group, then
   * lowest position) is the one that counts; key = g * R + position */
  for (int32_t d = 0; d < n_dims; d++) {
    int64_t* own = owner + (size_t)d * R;
    for (int32_t r = 0; r < R; r++) own[r] = INT64_MAX;
    const int32_t* off = group_off + (size_t)d * (max_groups + 1);
    for (int32_t g = 0; g < max_groups; g++) {
      int32_t a = off[g], b = off[g + 1];
      if (a < 0 || b < a || b > R) {
        status |= 1;
        continue;
      }
      for (int32_t i = a; i < b; i++) {
        int32_t m = members[(size_t)d * R + i];
        if (m < 0 || m >= R) {
          status |= 1;
          continue;
        }
        int64_t key = (int64_t)g * R + i;
        if (own[m] != INT64_MAX) status |= 2;
        if (key < own[m]) own[m] = key;
      }
    }
  }

  size_t cells = (size_t)R * S * E;
  for (size_t c = 0; c < cells; c++) {
    z_out[c] = 0.0f;
    flags_out[c] = 0;
  }
  for (int32_t s = 0; s < S; s++)
    for (int32_t e = 0; e < E; e++) {
      uint8_t d = route[e];
      for (int32_t g = 0; g < max_groups; g++) {
        size_t o = ((size_t)s * E + e) * max_groups + g;
        n_out[o] = 0;
        mean_out[o] = std_out[o] = cv_out[o] = 0.0;
        cls_out[o] = L2_NOT_EVALUATED;
        nstrag_out[o] = 0;
        if (d >= n_dims) continue;
        const int32_t* off = group_off + (size_t)d * (max_groups + 1);
        int32_t a = off[g], b = off[g + 1];
        if (a < 0 || b < a || b > R) continue;
        const int64_t* own = owner + (size_t)d * R;

        /* present members of this group, each at its first listing */
        int32_t n = 0;
        for (int32_t i = a; i < b; i++) {
          int32_t m = members[(size_t)d * R + i];
          if (m < 0 || m >= R || own[m] != (int64_t)g * R + i) continue;
          size_t c = ((size_t)m * S + s) * E + e;
          if (count[c] == 0) continue;
          uint64_t x = (uint64_t)sum_ns[c] / count[c];
          if (x >= L2_DOMAIN) {
            status |= 4;
            continue;
          }
          rk[n] = m;
          xs[n] = (int64_t)x;
          n++;
        }
        n_out[o] = (uint32_t)n;
        if (n < min_group || n < 2) continue;

        /* Eq. 5 with exact integer sums */
        u128 Ssum = 0, Q = 0;
        for (int32_t j = 0; j < n; j++) {
          Ssum += (u128)(uint64_t)xs[j];
          Q += (u128)(uint64_t)xs[j] * (uint64_t)xs[j];
        }
        u128 D = (u128)n * Q - Ssum * Ssum;
        double mean = (double)Ssum / (double)n;
        double var = (double)D / ((double)n * (double)(n - 1));
        double sd = sqrt(var);
        mean_out[o] = mean;
        std_out[o] = sd;
        cv_out[o] = mean > 0.0 ? sd / mean : 0.0;

        /* CV class: CV < c iff n D 10^6 < c^2 (n - 1) S^2 (S > 0) */
        uint8_t cls = 0;
        if (Ssum > 0) {
          u256 lhs = mul128((u128)n * 1000000u, D);
          u256 mild = mul128((u128)cv_mild_pm * (u128)cv_mild_pm * (u128)(n - 1), Ssum * Ssum);
          u256 sev = mul128((u128)cv_severe_pm * (u128)cv_severe_pm * (u128)(n - 1), Ssum * Ssum);
          if (!lt256(lhs, mild)) cls = lt256(lhs, sev) ? 1 : 2;
        }
        cls_out[o] = cls;

        /* z-scores and the straggler test z > z_pm / 1000 */
        uint32_t ns = 0;
        u256 rhs = mul128((u128)z_pm * (u128)z_pm * (u128)n, D);
        for (int32_t j = 0; j < n; j++) {
          size_t c = ((size_t)rk[j] * S + s) * E + e;
          float z = sd > 0.0 ? (float)(((double)xs[j] - mean) / sd) : 0.0f;
          uint8_t f = 1;
          u128 nx = (u128)n * (uint64_t)xs[j];
          if (nx > Ssum) {
            u128 dev = nx - Ssum;
            u256 lhs = mul128(dev * dev, (u128)(n - 1) * 1000000u);
            if (lt256(rhs, lhs)) {
              f |= 2;
              ns++;
            }
          }
          z_out[c] = z;
          flags_out[c] = f;
        }
        nstrag_out[o] = ns;
      }
    }
  free(rk);
  free(xs);
  free(owner);
  return status;
}
