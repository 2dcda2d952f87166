/*
 * ARGUS oracle: plain, slow, single-threaded CPU definition of the
 * trace-summarization and detection hot path.
 *
 * TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load or call this library. The product
 * path (libargus and its Python binding) never links, imports or falls back
 * to it. It shares no source with the HIP kernels.
 *
 * Paper: "ARGUS: Production-Scale Tracing and Performance Diagnosis for over
 * 10,000-GPU Clusters" (arXiv 2606.20374).
 *
 *   orc_summarize     - section 4.3 (record fields: kernel, launch time,
 *                       duration, stream) and section 5.2 (per (kernel,
 *                       stream, rank) grouping in each time window, log
 *                       transform evaluated on an equally spaced grid,
 *                       per-group count and order statistics). Plain
 *                       definition: an exact group-by.
 *   orc_summarize_keyed - the same group-by keyed by (kernel, stream).
 *   orc_compact       - the uploaded record stream of the summaries
 *                       (section 5.2, section 8.3 sizes). Plain definition:
 *                       fields written out in order.
 *   orc_cross_rank    - section 6.2 (the same kernel compared across ranks,
 *                       an anomalous rank shows as an elevated row, mean
 *                       distance to the other ranks as the deviation score,
 *                       IQR upper fence of Eq. 4) and Appendix B (z-score).
 *                       Order statistics by sorting.
 *   orc_iter_windows  - section 6.1 and Appendix B (sliding-window
 *                       ratio-gated jitter detection with effective width;
 *                       full-scan change-point detection; classification
 *                       into stable / jitter / regression / both). Algorithm
 *                       followed step by step.
 *
 * Readings where the paper leaves a value or rule open (bin grid, lower
 * median, MAD-based outlier rule, thresholds) are listed in the design
 * notes; each is restated at the point of use below.
 *
 * Parity pins (tests/test_oracle_*.py): brute-force recomputation with the
 * Python standard library on tiny inputs, closed forms on noise-free
 * traces, summary invariants on every segment, library order statistics
 * (statistics.median_low), hand-worked L1 series, and recovery of planted
 * stragglers, degraded pairs and stalled steps. The detection thresholds
 * themselves are proposals (the paper prints none): parity unpinned for
 * their values, pinned for their behaviour.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef unsigned __int128 u128;
typedef __int128 i128;

#define NB 32

/* ------------------------------------------------------------------ bins */

/* Octave bin of a duration: floor(log2 d) for d >= 2, 0 for d in {0, 1},
 * saturating at 31 (d >= 2^31 ns). The paper evaluates its density on an
 * equally spaced grid over log-duration (section 5.2); octave bins are that
 * grid with spacing ln 2. */
int orc_bin(uint64_t d) {
  int b = 0;
  while (d >= 2 && b < NB - 1) {
    d >>= 1;
    b++;
  }
  return b;
}

/* ------------------------------------------------------------- summarize */

/* The group-by of both keyings: key = kernel id (KC = K cells per segment),
 * or key = (kernel id, stream) as kid * NS + stream (KC = K * NS, section
 * 5.2 groups per (kernel, stream, rank)). Returns the number of malformed
 * segments (treated as empty). */
static int64_t summarize_impl(int keyed, int64_t n_seg, int32_t K, int32_t NS, int64_t n_events, const int32_t* kid,
                              const int32_t* stream, const int64_t* start, const int64_t* end, const int64_t* seg_off,
                              uint32_t* count, int64_t* sum_ns, int64_t* min_ns, int64_t* max_ns, uint32_t* hist,
                              uint32_t* n_valid, uint32_t* n_invalid, int64_t* t_first, int64_t* t_last,
                              int64_t* step_ns, int64_t* busy_ns, int64_t* stream_busy_ns, int64_t* wire_bytes) {
  const int64_t KC = keyed ? (int64_t)K * NS : K;
  int64_t bad = 0;
  for (int64_t g = 0; g < n_seg; g++) {
    /* identity values for every cell and segment */
    for (int64_t k = 0; k < KC; k++) {
      int64_t c = g * KC + k;
      count[c] = 0;
      sum_ns[c] = 0;
      min_ns[c] = INT64_MAX;
      max_ns[c] = INT64_MIN;
      for (int b = 0; b < NB; b++) hist[c * NB + b] = 0;
    }
    n_valid[g] = 0;
    n_invalid[g] = 0;
    t_first[g] = INT64_MAX;
    t_last[g] = INT64_MIN;
    busy_ns[g] = 0;
    for (int32_t s = 0; s < NS; s++) stream_busy_ns[g * NS + s] = 0;

    int64_t lo = seg_off[g], hi = seg_off[g + 1];
    int ok = lo >= 0 && lo <= hi && hi <= n_events && (hi - lo) <= (int64_t)UINT32_MAX;
    if (!ok) {
      bad++;
      lo = hi = 0;
    }
    for (int64_t i = lo; i < hi; i++) {
      /* a record is usable only with a known kernel id, a known stream, a
       * non-negative start and an end not before its start */
      int valid = kid[i] >= 0 && kid[i] < K && stream[i] >= 0 && stream[i] < NS && start[i] >= 0 &&
                  end[i] >= start[i];
      if (!valid) {
        n_invalid[g]++;
        continue;
      }
      uint64_t d = (uint64_t)end[i] - (uint64_t)start[i];
      int64_t c = g * KC + (keyed ? (int64_t)kid[i] * NS + stream[i] : kid[i]);
      count[c] += 1;
      sum_ns[c] = (int64_t)((uint64_t)sum_ns[c] + d); /* modulo 2^64 */
      if ((int64_t)d < min_ns[c]) min_ns[c] = (int64_t)d;
      if ((int64_t)d > max_ns[c]) max_ns[c] = (int64_t)d;
      hist[c * NB + orc_bin(d)] += 1;
      n_valid[g] += 1;
      busy_ns[g] = (int64_t)((uint64_t)busy_ns[g] + d);
      stream_busy_ns[g * NS + stream[i]] = (int64_t)((uint64_t)stream_busy_ns[g * NS + stream[i]] + d);
      if (start[i] < t_first[g]) t_first[g] = start[i];
      if (end[i] > t_last[g]) t_last[g] = end[i];
    }
    step_ns[g] = n_valid[g] ? t_last[g] - t_first[g] : 0;

    /* uploaded record size: key 4, count 4, sum 8, min 8, max 8, nnz 1,
     * then (bin u8, count u32) per nonzero bin */
    int64_t wb = 0;
    for (int64_t k = 0; k < KC; k++) {
      int64_t c = g * KC + k;
      if (count[c] == 0) continue;
      int nnz = 0;
      for (int b = 0; b < NB; b++) nnz += hist[c * NB + b] != 0;
      wb += 33 + 5 * nnz;
    }
    wire_bytes[g] = wb;
  }
  return bad;
}

/* Per-(rank, step, kernel id) cells [n_seg][K]. */
int64_t orc_summarize(int64_t n_seg, int32_t K, int32_t NS, int64_t n_events, const int32_t* kid,
                      const int32_t* stream, const int64_t* start, const int64_t* end, const int64_t* seg_off,
                      uint32_t* count, int64_t* sum_ns, int64_t* min_ns, int64_t* max_ns, uint32_t* hist,
                      uint32_t* n_valid, uint32_t* n_invalid, int64_t* t_first, int64_t* t_last, int64_t* step_ns,
                      int64_t* busy_ns, int64_t* stream_busy_ns, int64_t* wire_bytes) {
  return summarize_impl(0, n_seg, K, NS, n_events, kid, stream, start, end, seg_off, count, sum_ns, min_ns, max_ns,
                        hist, n_valid, n_invalid, t_first, t_last, step_ns, busy_ns, stream_busy_ns, wire_bytes);
}

/* Per-(rank, step, kernel id, stream) cells [n_seg][K][NS]. */
int64_t orc_summarize_keyed(int64_t n_seg, int32_t K, int32_t NS, int64_t n_events, const int32_t* kid,
                            const int32_t* stream, const int64_t* start, const int64_t* end, const int64_t* seg_off,
                            uint32_t* count, int64_t* sum_ns, int64_t* min_ns, int64_t* max_ns, uint32_t* hist,
                            uint32_t* n_valid, uint32_t* n_invalid, int64_t* t_first, int64_t* t_last,
                            int64_t* step_ns, int64_t* busy_ns, int64_t* stream_busy_ns, int64_t* wire_bytes) {
  return summarize_impl(1, n_seg, K, NS, n_events, kid, stream, start, end, seg_off, count, sum_ns, min_ns, max_ns,
                        hist, n_valid, n_invalid, t_first, t_last, step_ns, busy_ns, stream_busy_ns, wire_bytes);
}

/* -------------------------------------------------------------- compact */

static uint8_t* put_le(uint8_t* p, uint64_t v, int n) {
  for (int i = 0; i < n; i++) p[i] = (uint8_t)(v >> (8 * i));
  return p + n;
}

/* The uploaded summary (section 5.2: only compact statistics leave the
 * host; section 8.3 compares their size with the raw trace): for every
 * segment in order, every present cell (count >= 1) in key order becomes one
 * little-endian record: key u32 (the kernel id; with (kernel, stream) keys
 * kid | stream << 24), count u32, sum i64, min i64, max i64, nnz u8, then
 * (bin u8, count u32) for each nonzero octave bin in ascending order.
 * KC cells per segment; NS = 0 for kernel-id keys, else the stream count of
 * (kernel, stream) keys (KC = K NS). seg_byte_off[g] is the first byte of
 * segment g, seg_byte_off[n_seg] the total; bytes are written only while
 * they fit in cap. Returns the total. */
int64_t orc_compact(int64_t n_seg, int64_t KC, int32_t NS, const uint32_t* count, const int64_t* sum_ns,
                    const int64_t* min_ns, const int64_t* max_ns, const uint32_t* hist, uint8_t* out, int64_t cap,
                    int64_t* seg_byte_off) {
  int64_t pos = 0;
  uint8_t rec[33 + 5 * NB];
  for (int64_t g = 0; g < n_seg; g++) {
    seg_byte_off[g] = pos;
    for (int64_t k = 0; k < KC; k++) {
      int64_t c = g * KC + k;
      if (count[c] == 0) continue;
      uint32_t key = NS > 0 ? (uint32_t)(k / NS) | ((uint32_t)(k % NS) << 24) : (uint32_t)k;
      uint8_t* p = rec;
      p = put_le(p, key, 4);
      p = put_le(p, count[c], 4);
      p = put_le(p, (uint64_t)sum_ns[c], 8);
      p = put_le(p, (uint64_t)min_ns[c], 8);
      p = put_le(p, (uint64_t)max_ns[c], 8);
      uint8_t* nnz = p++;
      *nnz = 0;
      for (int b = 0; b < NB; b++) {
        if (hist[c * NB + b] == 0) continue;
        p = put_le(p, (uint64_t)b, 1);
        p = put_le(p, hist[c * NB + b], 4);
        (*nnz)++;
      }
      int64_t len = p - rec;
      if (pos + len <= cap) memcpy(out + pos, rec, (size_t)len);
      pos += len;
    }
  }
  seg_byte_off[n_seg] = pos;
  return pos;
}

/* ------------------------------------------------------------ cross-rank */

static int cmp_i64(const void* a, const void* b) {
  int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
  return (x > y) - (x < y);
}

/* Per-rank point statistic of one cell: the exact integer mean
 * floor(sum / count), the sum read as an unsigned 64-bit count of ns, the
 * result saturated at INT64_MAX. */
static int64_t cell_x(uint32_t count, int64_t sum) {
  uint64_t x = (uint64_t)sum / count;
  return x > (uint64_t)INT64_MAX ? INT64_MAX : (int64_t)x;
}

/* Ratio of a rank's statistic to the cross-rank median in permille,
 * floor(1000 x / med), saturated at INT32_MAX. */
static int32_t ratio_pm(int64_t x, int64_t med) {
  u128 q = ((u128)(uint64_t)x * 1000u) / (u128)(uint64_t)med;
  return q > (u128)INT32_MAX ? INT32_MAX : (int32_t)q;
}

int orc_cross_rank(int32_t R, int32_t S, int32_t K, const uint32_t* count, const int64_t* sum_ns,
                   /* parameters */
                   int32_t min_ranks, int32_t c_min_pair, int32_t min_kernels, int32_t k_mad_pm, int32_t ratio_pm_min,
                   int32_t alpha_pm, int32_t tau_rank_pm,
                   /* per (s,k) [S][K] */
                   uint32_t* n_present, int64_t* med_ns, int64_t* mad_ns, int64_t* q1_ns, int64_t* q3_ns,
                   float* xmean_ns, uint32_t* n_flag_k, uint32_t* n_degraded_k,
                   /* per cell [R][S][K] */
                   float* z, float* mean_ns, uint8_t* flags,
                   /* per (r,s) [R][S] */
                   int32_t* score_pm, uint32_t* n_eval, uint32_t* n_flag_r, uint8_t* straggler) {
  int64_t* v = (int64_t*)malloc(sizeof(int64_t) * (R > 0 ? R : 1));
  int64_t* dev = (int64_t*)malloc(sizeof(int64_t) * (R > 0 ? R : 1));
  int32_t* rat = (int32_t*)malloc(sizeof(int32_t) * (K > 0 ? K : 1));
  int64_t* rat64 = (int64_t*)malloc(sizeof(int64_t) * (K > 0 ? K : 1));
  if (!v || !dev || !rat || !rat64) return -1;

  for (int32_t s = 0; s < S; s++) {
    /* (1)-(3): per kernel, order statistics over the ranks where it ran */
    for (int32_t k = 0; k < K; k++) {
      int32_t n = 0;
      u128 xsum = 0;
      for (int32_t r = 0; r < R; r++) {
        int64_t c = ((int64_t)r * S + s) * K + k;
        if (count[c] >= 1) {
          v[n++] = cell_x(count[c], sum_ns[c]);
          xsum += (u128)(uint64_t)v[n - 1];
        }
      }
      int64_t sk = (int64_t)s * K + k;
      n_present[sk] = (uint32_t)n;
      n_flag_k[sk] = 0;
      n_degraded_k[sk] = 0;
      if (n < min_ranks || n == 0) {
        med_ns[sk] = mad_ns[sk] = q1_ns[sk] = q3_ns[sk] = -1;
        xmean_ns[sk] = 0.0f;
        continue;
      }
      qsort(v, (size_t)n, sizeof(int64_t), cmp_i64);
      /* lower median and lower nearest-rank quartiles */
      int64_t med = v[(n - 1) / 2];
      med_ns[sk] = med;
      q1_ns[sk] = v[(n - 1) / 4];
      q3_ns[sk] = v[(3 * (int64_t)(n - 1)) / 4];
      for (int32_t i = 0; i < n; i++) dev[i] = v[i] >= med ? v[i] - med : med - v[i];
      qsort(dev, (size_t)n, sizeof(int64_t), cmp_i64);
      mad_ns[sk] = dev[(n - 1) / 2];
      xmean_ns[sk] = (float)((double)xsum / (double)n);
    }

    /* (4)-(6): per rank, cell flags and the rank's typical slowdown */
    for (int32_t r = 0; r < R; r++) {
      int32_t ne = 0, nf = 0;
      for (int32_t k = 0; k < K; k++) {
        int64_t c = ((int64_t)r * S + s) * K + k;
        int64_t sk = (int64_t)s * K + k;
        z[c] = 0.0f;
        mean_ns[c] = 0.0f;
        flags[c] = 0;
        if (count[c] == 0) continue;
        mean_ns[c] = (float)((double)sum_ns[c] / (double)count[c]);
        uint32_t n = n_present[sk];
        if (n < (uint32_t)min_ranks || n == 0) continue;
        int64_t x = cell_x(count[c], sum_ns[c]);
        int64_t med = med_ns[sk], mad = mad_ns[sk], q1 = q1_ns[sk], q3 = q3_ns[sk];
        int64_t madf = mad > 1 ? mad : 1;
        int64_t iqr = q3 - q1 > 1 ? q3 - q1 : 1;
        /* robust z: MAD scaled to a normal sigma (1.4826 = 1 / Phi^-1(0.75)) */
        z[c] = (float)((double)(x - med) / (1.4826 * (double)madf));
        uint8_t f = 4; /* bit2: evaluated */
        /* bit0: slow-side outlier. Modified z above 3.5 (written as
         * 1000 (x - med) > k_mad_pm * mad), the rank at least ratio_pm_min
         * permille of the median, and enough samples in the cell */
        if (count[c] >= (uint32_t)c_min_pair && (i128)1000 * ((i128)x - med) > (i128)k_mad_pm * madf &&
            (i128)1000 * x >= (i128)ratio_pm_min * med)
          f |= 1;
        /* bit1: above the upper fence Q3 + alpha (Q3 - Q1) (Eq. 4) */
        if ((i128)1000 * ((i128)x - q3) > (i128)alpha_pm * iqr) f |= 2;
        flags[c] = f;
        if (med >= 1) {
          rat[ne++] = ratio_pm(x, med);
          if (f & 1) nf++;
        }
      }
      int64_t rs = (int64_t)r * S + s;
      n_eval[rs] = (uint32_t)ne;
      n_flag_r[rs] = (uint32_t)nf;
      if (ne == 0) {
        score_pm[rs] = -1;
      } else {
        for (int32_t i = 0; i < ne; i++) rat64[i] = rat[i];
        qsort(rat64, (size_t)ne, sizeof(int64_t), cmp_i64);
        score_pm[rs] = (int32_t)rat64[(ne - 1) / 2];
      }
      straggler[rs] = (ne >= min_kernels && (int64_t)score_pm[rs] >= 1000 + (int64_t)tau_rank_pm) ? 1 : 0;
      /* bit3: degraded (rank, kernel) pair = outlier cell on a rank that is
       * not a straggler as a whole */
      for (int32_t k = 0; k < K; k++) {
        int64_t c = ((int64_t)r * S + s) * K + k;
        int64_t sk = (int64_t)s * K + k;
        if (flags[c] & 1) {
          n_flag_k[sk]++;
          if (!straggler[rs]) {
            flags[c] |= 8;
            n_degraded_k[sk]++;
          }
        }
      }
    }
  }
  free(v);
  free(dev);
  free(rat);
  free(rat64);
  return 0;
}

/* ----------------------------------------------------------- iter windows */

#define Y_LIMIT ((int64_t)1 << 40) /* step times must lie in [0, 2^40) ns */

/* lower median of y[idx[0..m)] by sorting a copy */
static int64_t lower_median(const int64_t* vals, int32_t m, int64_t* scratch) {
  memcpy(scratch, vals, sizeof(int64_t) * (size_t)m);
  qsort(scratch, (size_t)m, sizeof(int64_t), cmp_i64);
  return scratch[(m - 1) / 2];
}

/* exact a*b vs c*d for unsigned 128-bit operands: -1, 0, +1 */
static void mul_wide(u128 a, u128 b, u128* hi, u128* lo) {
  uint64_t a0 = (uint64_t)a, a1 = (uint64_t)(a >> 64), b0 = (uint64_t)b, b1 = (uint64_t)(b >> 64);
  u128 p00 = (u128)a0 * b0, p01 = (u128)a0 * b1, p10 = (u128)a1 * b0, p11 = (u128)a1 * b1;
  u128 mid = (p00 >> 64) + (uint64_t)p01 + (uint64_t)p10;
  *lo = (u128)(uint64_t)p00 | (mid << 64);
  *hi = p11 + (p01 >> 64) + (p10 >> 64) + (mid >> 64);
}

static int cmp_products(u128 a, u128 b, u128 c, u128 d) {
  u128 h1, l1, h2, l2;
  mul_wide(a, b, &h1, &l1);
  mul_wide(c, d, &h2, &l2);
  if (h1 != h2) return h1 < h2 ? -1 : 1;
  if (l1 != l2) return l1 < l2 ? -1 : 1;
  return 0;
}

/* sample relative std (ddof 1) of a segment at most cmax_pm / 1000:
 * 10^6 n (n Q - S^2) <= cmax^2 S^2 (n - 1) */
static int rel_std_ok(int64_t n, u128 sum, u128 sumsq, int32_t cmax_pm) {
  u128 v = (u128)n * sumsq - sum * sum;
  return cmp_products((u128)1000000u * (u128)n, v, (u128)cmax_pm * (u128)cmax_pm * (u128)(n - 1), sum * sum) <= 0;
}

int orc_iter_windows(int32_t R, int32_t S, const int64_t* step_ns, int32_t W, int32_t theta_pm, int32_t beta_pm,
                     int32_t rho_pm, int32_t cmax_pm, int32_t min_seg, uint8_t* flags /* [R][S] */,
                     uint8_t* cls /* [R] */, int32_t* eff_width, int32_t* cp, float* cp_ratio) {
  if (R < 0 || S < 0 || S > 4096 || W < 1 || min_seg < 1 || theta_pm < 0 || beta_pm < 0 || rho_pm < 0 ||
      cmax_pm < 0)
    return -2;
  int64_t* outside = (int64_t*)malloc(sizeof(int64_t) * (S > 0 ? S : 1));
  int64_t* scratch = (int64_t*)malloc(sizeof(int64_t) * (S > 0 ? S : 1));
  uint8_t* cand = (uint8_t*)malloc((size_t)(S > 0 ? S : 1));
  if (!outside || !scratch || !cand) return -1;
  for (int32_t r = 0; r < R; r++) {
    const int64_t* y = step_ns + (int64_t)r * S;
    uint8_t* f = flags + (int64_t)r * S;
    for (int32_t i = 0; i < S; i++) f[i] = 0;
    eff_width[r] = 0;
    cp[r] = -1;
    cp_ratio[r] = 0.0f;
    cls[r] = 0;
    int in_domain = 1;
    for (int32_t i = 0; i < S; i++)
      if (y[i] < 0 || y[i] >= Y_LIMIT) in_domain = 0;
    if (!in_domain) {
      cls[r] = 0x80; /* input out of range: nothing evaluated */
      continue;
    }
    if (S == 0) continue;

    /* phase 1, sensitivity gating: windows of width W whose max/min ratio
     * exceeds theta are candidates */
    int32_t w = W < S ? W : S;
    for (int32_t i = 0; i < S; i++) cand[i] = 0;
    for (int32_t t = 0; t + w <= S; t++) {
      int64_t mx = y[t], mn = y[t];
      for (int32_t i = t; i < t + w; i++) {
        if (y[i] > mx) mx = y[i];
        if (y[i] < mn) mn = y[i];
      }
      if ((u128)1000 * (u128)mx > (u128)theta_pm * (u128)mn)
        for (int32_t i = t; i < t + w; i++) cand[i] = 1;
    }
    /* merge overlapping or touching candidate windows: a maximal run of
     * candidate points is one interval (windows cover contiguous points) */
    int32_t best_width = 0;
    for (int32_t a = 0; a < S;) {
      if (!cand[a]) {
        a++;
        continue;
      }
      int32_t b = a;
      while (b + 1 < S && cand[b + 1]) b++;
      /* phase 2: baseline = lower median of the points outside [a, b] (all
       * points when nothing lies outside) */
      int32_t m = 0;
      for (int32_t i = 0; i < S; i++)
        if (i < a || i > b) outside[m++] = y[i];
      int64_t base = m > 0 ? lower_median(outside, m, scratch) : lower_median(y, S, scratch);
      /* points significantly above the baseline; the longest contiguous run
       * of them is the interval's effective jitter width */
      int32_t run = 0;
      for (int32_t i = a; i <= b; i++) {
        f[i] |= 1;
        if ((u128)1000 * (u128)y[i] > (u128)beta_pm * (u128)base) {
          f[i] |= 2;
          run++;
          if (run > best_width) best_width = run;
        } else {
          run = 0;
        }
      }
      a = b + 1;
    }
    eff_width[r] = best_width;

    /* full-scan change point: split t with left y[0..t) and right y[t..S),
     * both at least min_seg long; valid when the regression ratio
     * mean_R / mean_L reaches rho and both sides have relative std at most
     * cmax; the valid split with the largest ratio wins (earliest on ties) */
    u128 tot = 0, totsq = 0;
    for (int32_t i = 0; i < S; i++) {
      tot += (u128)y[i];
      totsq += (u128)y[i] * (u128)y[i];
    }
    u128 sl = 0, ql = 0;
    int32_t best_t = -1;
    u128 best_num = 0, best_den = 1;
    for (int32_t t = 1; t < S; t++) {
      sl += (u128)y[t - 1];
      ql += (u128)y[t - 1] * (u128)y[t - 1];
      int64_t nl = t, nr = S - t;
      if (nl < min_seg || nr < min_seg) continue;
      u128 sr = tot - sl, qr = totsq - ql;
      if (sl == 0) continue; /* ratio undefined without a positive left mean */
      u128 num = sr * (u128)nl, den = sl * (u128)nr; /* ratio = num / den */
      if ((u128)1000 * num < (u128)rho_pm * den) continue;
      if (!rel_std_ok(nl, sl, ql, cmax_pm) || !rel_std_ok(nr, sr, qr, cmax_pm)) continue;
      if (best_t < 0 || cmp_products(num, best_den, best_num, den) > 0) {
        best_t = t;
        best_num = num;
        best_den = den;
      }
    }
    if (best_t >= 0) {
      cp[r] = best_t;
      cp_ratio[r] = (float)((double)best_num / (double)best_den);
      for (int32_t i = best_t; i < S; i++) f[i] |= 4;
    }
    cls[r] = (uint8_t)((best_width > 0 ? 1 : 0) | (best_t >= 0 ? 2 : 0));
  }
  free(outside);
  free(scratch);
  free(cand);
  return 0;
}
