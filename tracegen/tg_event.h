/*
 * Seeded synthetic kernel-event trace generator: the per-event rule.
 *
 * This header is the single definition of how event i of segment g is
 * generated. It is compiled twice from the same text: into the host fill
 * (plain C++ loops) and into the device fill kernel, so both produce the
 * same bytes. It holds no part of the trace-summarization method: it only
 * draws kernel ids, streams and timestamps from tables that the Python side
 * builds once per configuration.
 *
 * Event record shape follows the kernel-activity records of the paper's
 * kernel tracing (section 4.3): kernel name (as an integer id), stream,
 * start and end timestamps in ns. Shapes of the workloads (repeated
 * per-stream templates, section 5.2; straggler ranks, degraded kernels and
 * host stalls, section 9 and Appendix D) are encoded in the tables.
 *
 * Randomness is counter based: u = fmix64(key + (i + 1) * GOLDEN), where
 * fmix64 is the output function of SplitMix64 (Steele, Lea and Flood,
 * "Fast splittable pseudorandom number generators", OOPSLA 2014) and key is
 * derived from (seed, tag, rank, step). No floating point is used here.
 */
#ifndef TG_EVENT_H
#define TG_EVENT_H

#include <stdint.h>

#if defined(__HIPCC__)
#define TG_HD __host__ __device__ inline
#else
#define TG_HD static inline
#endif

#define TG_GOLDEN 0x9E3779B97F4A7C15ull
#define TG_TAG_EVENT 0x45564e54ull   /* per-event duration / jitter draws */
#define TG_TAG_SWAP 0x53574150ull    /* per-rank template pair swaps */
#define TG_TAG_CORRUPT 0x42414421ull /* per-event corruption draws */

typedef struct tg_params {
  uint64_t seed;
  int32_t n_ranks, n_steps, n_kernels, n_streams;
  int32_t tmpl_len;    /* T: template positions */
  int32_t n_hot;       /* ids [0, n_hot) draw Pareto durations; others lognormal */
  int32_t swap_pm;     /* per-rank probability (permille) of swapping template pair (2q, 2q+1) */
  int32_t invalid_ppm; /* per-event probability (ppm) of a corrupted record */
  int64_t epoch_ns;       /* timestamp of step 0 */
  int64_t step_period_ns; /* distance between step starts */
  int64_t t_span_ns;      /* span of one template repetition */
} tg_params_t;

typedef struct tg_tables {
  const int32_t* tmpl_kid;     /* [T] kernel id of template position p */
  const int64_t* tmpl_off;     /* [T] nominal start offset of position p within a repetition */
  const int64_t* tmpl_base_ns; /* [T] nominal duration at position p (kernel base x position mode) */
  const uint32_t* ln_q24;      /* [65536] lognormal multipliers in 8.24 fixed point */
  const uint32_t* pareto_ns;   /* [65536] Pareto quantiles in ns */
  const int32_t* mult_hot_pm;  /* [R] per-rank multiplier (permille) for ids < n_hot */
  const int32_t* mult_cold_pm; /* [R] per-rank multiplier (permille) for ids >= n_hot */
  const int32_t* pair_off;     /* [R+1] CSR offsets into the pair list */
  const int32_t* pair_kid;     /* [P] degraded (rank, kid) pairs: kid */
  const int32_t* pair_pm;      /* [P] multiplier (permille) */
  const int32_t* stall_rep;    /* [R*S] first repetition that is stalled (INT32_MAX: none) */
  const int64_t* stall_ns;     /* [R*S] stall added to every stalled event */
} tg_tables_t;

TG_HD uint64_t tg_fmix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

TG_HD uint64_t tg_key(uint64_t seed, uint64_t tag, int32_t r, int32_t s) {
  uint64_t k = tg_fmix64(seed + tag * TG_GOLDEN);
  return tg_fmix64(k ^ (((uint64_t)(uint32_t)r << 32) | (uint32_t)s));
}

TG_HD uint64_t tg_at(uint64_t key, int64_t i) {
  return tg_fmix64(key + (uint64_t)(i + 1) * TG_GOLDEN);
}

/* Generate event i (local index within segment g = r * n_steps + s). */
TG_HD void tg_event(const tg_params_t* P, const tg_tables_t* Tb, int32_t r, int32_t s, int64_t i,
                    int32_t* kid_out, int32_t* stream_out, int64_t* start_out, int64_t* end_out) {
  const int64_t T = P->tmpl_len;
  int64_t j = i / T;
  int32_t p = (int32_t)(i - j * T);
  if (P->swap_pm > 0) {
    int32_t q = p >> 1;
    if ((p ^ 1) < T) {
      uint64_t h = tg_at(tg_key(P->seed, TG_TAG_SWAP, r, 0), q);
      if ((int32_t)(h % 1000u) < P->swap_pm) p ^= 1;
    }
  }
  const int32_t g = r * P->n_steps + s;
  int32_t kid = Tb->tmpl_kid[p];
  int32_t stream = kid % P->n_streams;
  uint64_t u = tg_at(tg_key(P->seed, TG_TAG_EVENT, r, s), i);
  int64_t d;
  int32_t m;
  if (kid < P->n_hot) {
    d = (int64_t)Tb->pareto_ns[u & 0xFFFFu];
    m = Tb->mult_hot_pm[r];
  } else {
    d = (int64_t)(((uint64_t)Tb->tmpl_base_ns[p] * (uint64_t)Tb->ln_q24[u & 0xFFFFu]) >> 24);
    m = Tb->mult_cold_pm[r];
  }
  d = d * m / 1000;
  for (int32_t e = Tb->pair_off[r]; e < Tb->pair_off[r + 1]; ++e)
    if (Tb->pair_kid[e] == kid) d = d * Tb->pair_pm[e] / 1000;
  int64_t start = P->epoch_ns + (int64_t)s * P->step_period_ns + j * P->t_span_ns + Tb->tmpl_off[p] +
                  (int64_t)((u >> 32) % 1000u);
  if (j >= Tb->stall_rep[g]) start += Tb->stall_ns[g];
  int64_t end = start + d;
  if (P->invalid_ppm > 0) {
    uint64_t w = tg_at(tg_key(P->seed, TG_TAG_CORRUPT, r, s), i);
    if ((int32_t)(w % 1000000u) < P->invalid_ppm) {
      int32_t small = (int32_t)((w >> 40) % 16u);
      switch ((w >> 32) % 5u) {
        case 0: kid = P->n_kernels + small; break;             /* id past the table */
        case 1: kid = -1 - small; break;                       /* negative id */
        case 2: stream = P->n_streams + small; break;          /* unknown stream */
        case 3: end = start - 1 - (int64_t)small; break;       /* end before start */
        default: start = -1 - (int64_t)small; end = start + d; /* negative timestamp */
      }
    }
  }
  *kid_out = kid;
  *stream_out = stream;
  *start_out = start;
  *end_out = end;
}

#endif /* TG_EVENT_H */
