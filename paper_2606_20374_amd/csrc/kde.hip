// Duration clustering per (rank, step, kernel id): valleys of a Gaussian KDE
// over log-duration, each cluster reported as (count, p50, p99) (section 5.2,
// Eq. 1; the step-by-step definition is in include/argus.h).
//
// Three kernels:
//   kde_scatter_kernel  one workgroup per segment (persistent queue): the
//                       segment's valid durations are bucketed by kernel id
//                       into the workspace (a counting sort whose counts come
//                       from argus_summarize), so every cell's durations are
//                       contiguous. HBM bound: 24 B read + 8 B written per event.
//   kde_cell_kernel<fast>  one wavefront per cell, cells claimed 64 at a time:
//                       grid histogram in LDS, exact bandwidth, integer-weight
//                       density, valleys, filters, and exact order statistics
//                       by radix selection inside the target grid bin. Cells
//                       whose grid, kernel or valley list exceed its 19 KB of
//                       LDS are appended to a deferred list.
//   kde_cell_kernel<slow>  the deferred cells, 56 KB of LDS per wavefront.
#include <atomic>
#include <cmath>
#include <mutex>
#include <vector>

#include "argus_internal.h"

namespace argus {
namespace {

constexpr int kScatterThreads = 512;
constexpr int kWave = 64;
constexpr int kFastWords = 4096;  // grid histogram + kernel weights, fast path
constexpr int kFastCand = 256;
constexpr int kSlowWords = 8192;  // 4096-point grid + 4096 weights
constexpr int kSlowCand = 2047;   // a 4096-point grid has at most 2047 valleys
constexpr int kMaxC = ARGUS_KDE_MAXC;
constexpr int kMaxT = 2 * kMaxC;  // selection targets: p50 and p99 per cluster
constexpr int kPowTab = 65536;    // n^-0.2 for n below this, from the host libm
constexpr int kRegVals = 4;       // cells of up to 256 durations stay in registers

// n^-0.2 for small n, filled once per device from the host's pow().
__device__ double g_kde_pow[kPowTab];

struct KdeArgs {
  const int32_t* kernel_id;
  const int32_t* stream;
  const int64_t* start_ns;
  const int64_t* end_ns;
  const int64_t* seg_off;
  int64_t n_events;
  int32_t n_seg, K, NS;
  int32_t sub_bits, frac_pm, min_count, gap;
  const uint32_t* count;
  const int64_t* min_ns;
  const int64_t* max_ns;
  uint8_t* n_clusters;
  uint32_t* cl_count;
  int64_t* p50;
  int64_t* p99;
  int32_t* bw_q8;
  int32_t* dev_status;
  uint32_t* counters;  // [0] scatter queue, [1] cell queue, [2] deferred count, [3] deferred queue
  uint64_t* bucket;    // [n_events], segment g's durations at seg_off[g] + local position
  uint32_t* cell_end;  // [cells]: local end offset of each cell's durations
  uint32_t* deferred;  // [cells]
  uint32_t theta[64];  // ceil(2^(23 + t/64))
};

// ----------------------------------------------------------------- helpers

// floor(64 log2 d') with d' the 24 leading significant bits of d: a hardware
// log2 estimate, corrected against the exact mantissa thresholds.
__device__ __forceinline__ int grid64(uint64_t d, const uint32_t* th) {
  if (d < 2) return 0;
  const int e = 63 - __builtin_clzll(d);
  const uint32_t m = e >= 23 ? (uint32_t)(d >> (e - 23)) : (uint32_t)(d << (23 - e));
  int t = (int)((__log2f((float)m) - 23.0f) * 64.0f);
  t = t < 0 ? 0 : (t > 63 ? 63 : t);
  while (t > 0 && m < th[t]) --t;
  while (t < 63 && m >= th[t + 1]) ++t;
  return e * 64 + t;
}

// Smallest duration whose 64-per-octave grid value is >= b.
__device__ __forceinline__ uint64_t grid64_lb(int b, const uint32_t* th) {
  if (b <= 0) return 0;
  const int e = b >> 6, t = b & 63;
  if (e >= 64) return ~0ull;
  const uint64_t m = th[t];
  return e >= 23 ? (m << (e - 23)) : ((m + (1ull << (23 - e)) - 1) >> (23 - e));
}

// Correctly rounded conversion of an unsigned 128-bit integer to double.
__device__ __forceinline__ double u128_to_f64(unsigned __int128 v) {
  const uint64_t hi = (uint64_t)(v >> 64);
  if (hi == 0) return (double)(uint64_t)v;
  const int sh = 64 - __builtin_clzll(hi);
  uint64_t top = (uint64_t)(v >> sh);
  const unsigned __int128 low_mask = (((unsigned __int128)1) << sh) - 1;
  top |= (v & low_mask) != 0 ? 1ull : 0ull;
  return ldexp((double)top, sh);
}

__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, l);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t w = __shfl_xor(v, o, kWave);
    v = w < v ? w : v;
  }
  return v;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t w = __shfl_xor(v, o, kWave);
    v = w > v ? w : v;
  }
  return v;
}

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  const int l = lane_id();
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t t = __shfl_up(v, o, kWave);
    if (l >= o) v += t;
  }
  return v;
}

__device__ __forceinline__ void flag(const KdeArgs& a, int bit) {
  if (a.dev_status) atomicOr(a.dev_status, bit);
}

// ----------------------------------------------------------------- scatter

__global__ __launch_bounds__(kScatterThreads) void kde_scatter_kernel(KdeArgs a) {
  __shared__ uint32_t cur[ARGUS_MAX_KDE_KERNELS];
  __shared__ uint32_t wave_tot[kScatterThreads / kWave];
  __shared__ uint32_t claim;
  const int tid = threadIdx.x, K = a.K;
  const int per = (K + kScatterThreads - 1) / kScatterThreads;
  while (true) {
    if (tid == 0) claim = atomicAdd(&a.counters[0], 1u);
    __syncthreads();
    const uint32_t g = claim;
    if (g >= (uint32_t)a.n_seg) break;
    // cursors = exclusive prefix of the segment's per-kernel counts
    const uint32_t* cnt = a.count + (int64_t)g * K;
    const int k0 = tid * per, k1 = min(K, k0 + per);
    uint32_t own = 0;
    for (int k = k0; k < k1; ++k) own += cnt[k];
    const uint32_t incl = wave_incl_scan(own);
    if (lane_id() == kWave - 1) wave_tot[tid / kWave] = incl;
    __syncthreads();
    uint32_t base = incl - own;
    for (int w = 0; w < tid / kWave; ++w) base += wave_tot[w];
    for (int k = k0; k < k1; ++k) {
      cur[k] = base;
      base += cnt[k];
    }
    __syncthreads();
    const int64_t lo = a.seg_off[g], hi = a.seg_off[g + 1];
    const bool bad = !(lo >= 0 && lo <= hi && hi <= a.n_events && hi - lo <= (int64_t)UINT32_MAX);
    if (!bad) {
      const uint32_t len = (uint32_t)(hi - lo);
      uint64_t* out = a.bucket + lo;
      for (int64_t i = lo + tid; i < hi; i += kScatterThreads) {
        const int32_t kid = a.kernel_id[i], st = a.stream[i];
        const int64_t t0 = a.start_ns[i], t1 = a.end_ns[i];
        if (kid >= 0 && kid < K && st >= 0 && st < a.NS && t0 >= 0 && t1 >= t0) {
          const uint32_t p = atomicAdd(&cur[kid], 1u);
          if (p < len) out[p] = (uint64_t)t1 - (uint64_t)t0;
        }
      }
    }
    __syncthreads();
    uint32_t* ends = a.cell_end + (int64_t)g * K;
    for (int k = tid; k < K; k += kScatterThreads) ends[k] = cur[k];
    __syncthreads();
  }
}

// -------------------------------------------------------------------- cells

template <int WORDS, int CAND>
struct CellLds {
  uint64_t cval[CAND];  // valley depth f
  uint64_t tlb[kMaxT];  // target bin: smallest duration
  uint64_t tub[kMaxT];  // target bin: one past the largest duration
  uint64_t tpre[kMaxT]; // digits selected so far
  uint64_t trank[kMaxT];
  uint32_t buf[WORDS];  // grid histogram (then its prefix) | weights; later selection histograms
  int32_t cpos[CAND];   // valley grid index
  uint32_t th[64];
};

template <int WORDS, int CAND>
__device__ void remove_valley(CellLds<WORDS, CAND>& L, int idx, int m) {
  const int l = lane_id();
  for (int qb = idx; qb < m - 1; qb += kWave) {
    const int q = qb + l;
    int32_t p = 0;
    uint64_t v = 0;
    if (q < m - 1) {
      p = L.cpos[q + 1];
      v = L.cval[q + 1];
    }
    __syncthreads();
    if (q < m - 1) {
      L.cpos[q] = p;
      L.cval[q] = v;
    }
    __syncthreads();
  }
}

__device__ void write_empty(const KdeArgs& a, int64_t c) {
  const int l = lane_id();
  if (l < kMaxC) {
    a.cl_count[c * kMaxC + l] = 0;
    a.p50[c * kMaxC + l] = 0;
    a.p99[c * kMaxC + l] = 0;
  }
  if (l == 0) {
    a.n_clusters[c] = 0;
    if (a.bw_q8) a.bw_q8[c] = 0;
  }
}

// One cell on one wavefront. vals: the cell's n durations (global memory);
// when n <= 64 * kRegVals they are also held in registers (rv). Returns false
// when the cell does not fit this kernel's LDS (only if may_defer).
template <int WORDS, int CAND>
__device__ bool kde_one_cell(const KdeArgs& a, CellLds<WORDS, CAND>& L, int64_t c, uint32_t n, uint64_t mn,
                             uint64_t mx, const uint64_t* vals, bool may_defer) {
  const int l = lane_id();
  const int sh = 6 - a.sub_bits;
  const int lo = grid64(mn, L.th) >> sh;
  const int G = (grid64(mx, L.th) >> sh) - lo + 1;
  uint32_t* cgrid = L.buf;
  const bool in_regs = n <= (uint32_t)(kWave * kRegVals);
  uint64_t rv[kRegVals];
#pragma unroll
  for (int r = 0; r < kRegVals; ++r) rv[r] = 0;
  if (in_regs) {
#pragma unroll
    for (int r = 0; r < kRegVals; ++r) {
      const uint32_t i = (uint32_t)(l + r * kWave);
      if (i < n) rv[r] = __builtin_nontemporal_load(vals + i);
    }
  }

  // 1. grid histogram
  for (int j = l; j < G; j += kWave) cgrid[j] = 0;
  __syncthreads();
  bool out_of_range = false;
  if (in_regs) {
#pragma unroll
    for (int r = 0; r < kRegVals; ++r) {
      const uint32_t i = (uint32_t)(l + r * kWave);
      if (i < n) {
        const int x = (grid64(rv[r], L.th) >> sh) - lo;
        if (x >= 0 && x < G) atomicAdd(&cgrid[x], 1u);
        else out_of_range = true;
      }
    }
  } else {
    for (uint32_t i = l; i < n; i += kWave) {
      const int x = (grid64(vals[i], L.th) >> sh) - lo;
      if (x >= 0 && x < G) atomicAdd(&cgrid[x], 1u);
      else out_of_range = true;
    }
  }
  __syncthreads();
  if (__any(out_of_range)) {  // durations outside the summarized [min, max]
    if (l == 0) flag(a, ARGUS_DEV_KDE_SUMMARY);
    write_empty(a, c);
    return true;
  }

  // 2. bandwidth
  uint64_t s1 = 0, s2 = 0;
  for (int j = l; j < G; j += kWave) {
    const uint64_t k = cgrid[j];
    s1 += k * (uint64_t)j;
    s2 += k * (uint64_t)j * (uint64_t)j;
  }
  s1 = wave_sum_u64(s1);
  s2 = wave_sum_u64(s2);
  int64_t H = 0;
  if (n >= 2) {
    const unsigned __int128 V = (unsigned __int128)n * s2 - (unsigned __int128)s1 * s1;
    const double var = u128_to_f64(V) / ((double)n * (double)(n - 1));
    const double pw = n < (uint32_t)kPowTab ? g_kde_pow[n] : pow((double)n, -0.2);
    const double h = 1.06 * sqrt(var) * pw;
    H = (int64_t)floor(h * 256.0 + 0.5);
  }

  // 3-4. weights, density and valleys
  int m = 0;
  if (H > 0 && G >= 3) {
    uint32_t* w = L.buf + G;
    const double H2 = (double)(H * H);
    int T = -1;
    for (int tb = 0; tb < G; tb += kWave) {
      const int t = tb + l;
      uint32_t wt = 0;
      if (t < G) wt = (uint32_t)floor(65536.0 * exp(-(double)(32768ll * t * t) / H2) + 0.5);
      const uint64_t nz = __ballot(wt != 0);
      const int cnt = __popcll(nz);  // weights are non-increasing in t
      if (G + tb + cnt > WORDS) {
        if (may_defer) return false;
      }
      if (wt != 0 && G + t < WORDS) w[t] = wt;
      T = tb + cnt - 1;
      if (cnt < kWave) break;
    }
    __syncthreads();
    int carry_start = -1, carry_drop = 0;
    uint64_t prev_last = 0;
    bool overflow = false;
    for (int jb = 0; jb < G; jb += kWave) {
      const int j = jb + l;
      const bool valid = j < G;
      uint64_t fj = 0;
      if (valid) {
        const int b0 = j - T > 0 ? j - T : 0, b1 = j + T < G - 1 ? j + T : G - 1;
        for (int b = b0; b <= b1; ++b) fj += (uint64_t)cgrid[b] * w[j > b ? j - b : b - j];
      }
      uint64_t fl = __shfl_up(fj, 1, kWave);
      if (l == 0) fl = prev_last;
      const bool start = valid && (j == 0 || fj != fl);
      const bool drop = start && j > 0 && fl > fj;
      const bool rise = start && j > 0 && fl < fj;
      const uint64_t S = __ballot(start), D = __ballot(drop);
      int a_idx = carry_start, a_drop = carry_drop;
      const uint64_t below = S & ((1ull << l) - 1ull);
      if (below) {
        const int al = 63 - __builtin_clzll(below);
        a_idx = jb + al;
        a_drop = (int)((D >> al) & 1ull);
      }
      const bool is_valley = rise && a_drop;
      const uint64_t Vb = __ballot(is_valley);
      if (is_valley) {
        const int idx = m + __popcll(Vb & ((1ull << l) - 1ull));
        if (idx < CAND) {
          L.cpos[idx] = (a_idx + j - 1) / 2;
          L.cval[idx] = fl;
        }
      }
      m += __popcll(Vb);
      if (m > CAND) overflow = true;
      if (S) {
        const int ls = 63 - __builtin_clzll(S);
        carry_start = jb + ls;
        carry_drop = (int)((D >> ls) & 1ull);
      }
      const int last = G - 1 - jb < kWave - 1 ? G - 1 - jb : kWave - 1;
      prev_last = readlane64(fj, last);
    }
    __syncthreads();
    if (overflow) {
      if (may_defer) return false;
      m = CAND;  // unreachable for the large-LDS instantiation
    }
  }

  // grid histogram -> inclusive prefix counts (in place)
  {
    uint32_t carry = 0;
    for (int jb = 0; jb < G; jb += kWave) {
      const int j = jb + l;
      const uint32_t v = j < G ? cgrid[j] : 0u;
      const uint32_t incl = wave_incl_scan(v) + carry;
      if (j < G) cgrid[j] = incl;
      carry = __builtin_amdgcn_readlane(incl, kWave - 1);
    }
    __syncthreads();
  }
  const uint32_t* P = cgrid;
  auto bound = [&](int q, int mm) -> int { return q < mm ? L.cpos[q] : G - 1; };

  // 5. cluster-level filter
  uint64_t need = ((uint64_t)a.frac_pm * n + 999u) / 1000u;
  if (need < (uint64_t)a.min_count) need = (uint64_t)a.min_count;
  while (m > 0) {
    uint64_t best = ~0ull;  // size * 4096 + q: smallest size, then lowest q
    for (int qb = 0; qb <= m; qb += kWave) {
      const int q = qb + l;
      if (q <= m) {
        const uint64_t hiP = P[bound(q, m)];
        const uint64_t loP = q > 0 ? P[L.cpos[q - 1]] : 0;
        const uint64_t key = ((hiP - loP) << 12) | (uint64_t)q;
        best = key < best ? key : best;
      }
    }
    best = wave_min_u64(best);
    if ((best >> 12) >= need) break;
    const int q = (int)(best & 4095u);
    int idx;
    if (q == 0) idx = 0;
    else if (q == m) idx = m - 1;
    else idx = L.cval[q - 1] > L.cval[q] ? q - 1 : q;
    remove_valley(L, idx, m);
    --m;
  }

  // 6. spacing filter over [0, valleys..., G - 1]
  while (m > 0) {
    int hit = -1;
    for (int qb = 0; qb <= m && hit < 0; qb += kWave) {
      const int q = qb + l;
      bool close = false;
      if (q <= m) {
        const int lo_b = q > 0 ? L.cpos[q - 1] : 0;
        close = bound(q, m) - lo_b < a.gap;
      }
      const uint64_t bm = __ballot(close);
      if (bm) hit = qb + __builtin_ctzll(bm);
    }
    if (hit < 0) break;
    int idx;
    if (hit == 0) idx = 0;
    else if (hit == m) idx = m - 1;
    else idx = L.cval[hit - 1] > L.cval[hit] ? hit - 1 : hit;
    remove_valley(L, idx, m);
    --m;
  }

  // 7. cluster cap: drop the largest-f valley (the upper one on ties)
  while (m > kMaxC - 1) {
    uint64_t best_v = 0;
    int best_q = -1;
    for (int qb = 0; qb < m; qb += kWave) {
      const int q = qb + l;
      uint64_t v = 0;
      bool on = q < m;
      if (on) v = L.cval[q];
      const uint64_t mv = wave_max_u64(on ? v : 0ull);
      const uint64_t bm = __ballot(on && v == mv);
      if (bm && (best_q < 0 || mv >= best_v)) {
        best_v = mv;
        best_q = qb + 63 - __builtin_clzll(bm);
      }
    }
    remove_valley(L, best_q, m);
    --m;
  }

  // 8. counts and selection targets (global ranks in the cell's sorted order)
  const int ncl = m + 1;
  uint32_t ccount[kMaxC];
#pragma unroll
  for (int q = 0; q < kMaxC; ++q) ccount[q] = 0;
  int NT = 0;
  {
    uint64_t before = 0;
    for (int q = 0; q < ncl; ++q) {
      const uint64_t hiP = P[bound(q, m)];
      const uint64_t size = hiP - before;
#pragma unroll
      for (int qq = 0; qq < kMaxC; ++qq)
        if (qq == q) ccount[qq] = (uint32_t)size;
      const uint64_t r50 = before + (size - 1) / 2;
      const uint64_t r99 = before + (99 * size + 99) / 100 - 1;
      for (int t2 = 0; t2 < 2; ++t2) {
        const uint64_t r = t2 == 0 ? r50 : r99;
        // smallest grid index j with P[j] > r
        int lo_j = 0, hi_j = G - 1;
        while (lo_j < hi_j) {
          const int mid = (lo_j + hi_j) >> 1;
          if ((uint64_t)P[mid] > r) hi_j = mid;
          else lo_j = mid + 1;
        }
        const uint64_t below = lo_j > 0 ? P[lo_j - 1] : 0;
        if (l == 0) {
          L.tlb[NT] = grid64_lb((lo + lo_j) << sh, L.th);
          L.tub[NT] = grid64_lb((lo + lo_j + 1) << sh, L.th);
          L.tpre[NT] = 0;
          L.trank[NT] = r - below;
        }
        ++NT;
      }
      before = hiP;
    }
  }
  __syncthreads();

  // 9. exact selection inside each target bin, 8 bits per pass
  int nbits = 0;
  for (int t = 0; t < NT; ++t) {
    const uint64_t width = L.tub[t] - L.tlb[t];
    const int b = width > 1 ? 64 - __builtin_clzll(width - 1) : 0;
    nbits = b > nbits ? b : nbits;
  }
  const int npass = (nbits + 7) / 8;
  uint32_t* hist = L.buf;  // NT x 256 counters; the prefix counts are no longer needed
  for (int p = 0; p < npass; ++p) {
    const int shift = 8 * (npass - 1 - p);
    for (int i = l; i < NT * 256; i += kWave) hist[i] = 0;
    __syncthreads();
    auto consider = [&](uint64_t v) {
      for (int t = 0; t < NT; ++t) {
        const uint64_t lb = L.tlb[t];
        if (v >= lb && v < L.tub[t]) {
          const uint64_t u = v - lb;
          const uint64_t hi_part = shift + 8 >= 64 ? 0 : u >> (shift + 8);
          if (hi_part == L.tpre[t]) atomicAdd(&hist[t * 256 + (int)((u >> shift) & 255u)], 1u);
        }
      }
    };
    if (in_regs) {
#pragma unroll
      for (int r = 0; r < kRegVals; ++r)
        if ((uint32_t)(l + r * kWave) < n) consider(rv[r]);
    } else {
      for (uint32_t i = l; i < n; i += kWave) consider(vals[i]);
    }
    __syncthreads();
    for (int t = 0; t < NT; ++t) {
      // digit holding the target rank: 4 counters per lane, then a wave scan
      const uint32_t* h = hist + t * 256;
      const uint32_t c0 = h[4 * l], c1 = h[4 * l + 1], c2 = h[4 * l + 2], c3 = h[4 * l + 3];
      const uint32_t tot = c0 + c1 + c2 + c3;
      const uint32_t incl = wave_incl_scan(tot);
      const uint64_t r = L.trank[t];
      const bool mine = (uint64_t)(incl - tot) <= r && r < (uint64_t)incl;
      const uint64_t bm = __ballot(mine);
      const int owner = bm ? __builtin_ctzll(bm) : 0;
      if (l == owner) {
        uint64_t rr = r - (incl - tot);
        int d = 4 * l;
        if (rr >= c0) {
          rr -= c0;
          ++d;
          if (rr >= c1) {
            rr -= c1;
            ++d;
            if (rr >= c2) {
              rr -= c2;
              ++d;
            }
          }
        }
        L.trank[t] = rr;
        L.tpre[t] = (L.tpre[t] << 8) | (uint64_t)d;
      }
      __syncthreads();
    }
  }

  // outputs
  if (l < kMaxC) {
    const int64_t o = c * kMaxC + l;
    uint32_t cnt = 0;
#pragma unroll
    for (int q = 0; q < kMaxC; ++q)
      if (q == l) cnt = ccount[q];
    a.cl_count[o] = l < ncl ? cnt : 0u;
    a.p50[o] = l < ncl ? (int64_t)(L.tlb[2 * l] + L.tpre[2 * l]) : 0;
    a.p99[o] = l < ncl ? (int64_t)(L.tlb[2 * l + 1] + L.tpre[2 * l + 1]) : 0;
  }
  if (l == 0) {
    a.n_clusters[c] = (uint8_t)ncl;
    if (a.bw_q8) a.bw_q8[c] = (int32_t)H;
  }
  __syncthreads();
  return true;
}

// Checks of one cell's summary against the bucketed durations; on success
// returns the cell's durations in *vals.
__device__ bool cell_source(const KdeArgs& a, int64_t c, uint32_t n, int64_t mn, int64_t mx, uint32_t end,
                            uint32_t prev_end, const uint64_t** vals) {
  const int64_t g = c / a.K;
  const int64_t lo = a.seg_off[g], hi = a.seg_off[g + 1];
  const bool seg_ok = lo >= 0 && lo <= hi && hi <= a.n_events && hi - lo <= (int64_t)UINT32_MAX;
  const bool ok = seg_ok && end >= n && end - n == prev_end && (int64_t)end <= hi - lo && mn >= 0 && mn <= mx;
  if (ok) *vals = a.bucket + lo + (end - n);
  return ok;
}

template <int WORDS, int CAND, bool SLOW>
__global__ __launch_bounds__(kWave) void kde_cell_kernel(KdeArgs a) {
  __shared__ CellLds<WORDS, CAND> L;
  const int l = lane_id();
  L.th[l] = a.theta[l];
  __syncthreads();
  const int64_t C = (int64_t)a.n_seg * a.K;
  while (true) {
    uint32_t claim = 0;
    if (l == 0) claim = atomicAdd(&a.counters[SLOW ? 3 : 1], 1u);
    claim = __builtin_amdgcn_readfirstlane(claim);
    int64_t c0;
    int ncells;
    if (SLOW) {
      const uint32_t nd = __builtin_amdgcn_readfirstlane(__hip_atomic_load(&a.counters[2], __ATOMIC_RELAXED,
                                                                            __HIP_MEMORY_SCOPE_AGENT));
      if (claim >= nd) break;
      c0 = a.deferred[claim];
      ncells = 1;
    } else {
      c0 = (int64_t)claim * kWave;
      if (c0 >= C) break;
      ncells = C - c0 < kWave ? (int)(C - c0) : kWave;
    }
    // per-lane prefetch of the cells' summaries
    uint32_t n = 0, end = 0, prev = 0;
    int64_t mn = 0, mx = 0;
    const int64_t cl = SLOW ? c0 : c0 + l;
    if ((SLOW && l == 0) || (!SLOW && l < ncells)) {
      n = a.count[cl];
      if (n) {
        mn = a.min_ns[cl];
        mx = a.max_ns[cl];
        end = a.cell_end[cl];
        prev = cl % a.K ? a.cell_end[cl - 1] : 0u;
      }
    }
    for (int i = 0; i < ncells; ++i) {
      const int64_t c = c0 + i;
      const uint32_t cn = __builtin_amdgcn_readlane(n, i);
      if (cn == 0) {
        write_empty(a, c);
        continue;
      }
      const uint32_t ce = __builtin_amdgcn_readlane(end, i), cp = __builtin_amdgcn_readlane(prev, i);
      const int64_t cmn = (int64_t)readlane64((uint64_t)mn, i), cmx = (int64_t)readlane64((uint64_t)mx, i);
      const uint64_t* vals = nullptr;
      if (!cell_source(a, c, cn, cmn, cmx, ce, cp, &vals)) {
        if (l == 0) flag(a, ARGUS_DEV_KDE_SUMMARY);
        write_empty(a, c);
        continue;
      }
      if (!kde_one_cell<WORDS, CAND>(a, L, c, cn, (uint64_t)cmn, (uint64_t)cmx, vals, !SLOW)) {
        if (l == 0) a.deferred[atomicAdd(&a.counters[2], 1u)] = (uint32_t)c;
        __syncthreads();
      }
    }
  }
}

// ---------------------------------------------------------------- host side

// Exact thresholds ceil(2^(23 + t/64)): the smallest m with
// floor(log2(m^64)) >= 1472 + t, found by bisection with big-integer powers.
int bitlen_pow64(uint32_t m) {
  std::vector<uint32_t> x{m};
  for (int s = 0; s < 6; ++s) {
    std::vector<uint32_t> r(2 * x.size(), 0u);
    for (size_t i = 0; i < x.size(); ++i) {
      uint64_t carry = 0;
      for (size_t j = 0; j < x.size(); ++j) {
        const uint64_t t = (uint64_t)x[i] * x[j] + r[i + j] + carry;
        r[i + j] = (uint32_t)t;
        carry = t >> 32;
      }
      r[i + x.size()] = (uint32_t)carry;
    }
    while (r.size() > 1 && r.back() == 0) r.pop_back();
    x.swap(r);
  }
  return (int)(x.size() - 1) * 32 + (32 - __builtin_clz(x.back()));
}

const uint32_t* thresholds() {
  static uint32_t th[64];
  static std::once_flag once;
  std::call_once(once, [] {
    th[0] = 1u << 23;
    for (int t = 1; t < 64; ++t) {
      uint32_t lo = 1u << 23, hi = (1u << 24) - 1;
      while (lo < hi) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (bitlen_pow64(mid) - 1 >= 1472 + t) hi = mid;
        else lo = mid + 1;
      }
      th[t] = lo;
    }
  });
  return th;
}

// Fill g_kde_pow on the current device once.
hipError_t ensure_pow_table() {
  static std::mutex mu;
  static bool done[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (done[dev]) return hipSuccess;
  std::vector<double> tab(kPowTab);
  tab[0] = 0.0;
  for (int n = 1; n < kPowTab; ++n) tab[n] = std::pow((double)n, -0.2);
  e = hipMemcpyToSymbol(HIP_SYMBOL(g_kde_pow), tab.data(), sizeof(double) * kPowTab);
  if (e == hipSuccess) done[dev] = true;
  return e;
}

template <typename Kern>
int resident(Kern kern, int threads) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, threads, 0) != hipSuccess) return 0;
  return cus * (per_cu > 0 ? per_cu : 1);
}

__global__ void kde_clear_kernel(uint32_t* counters, int32_t* dev_status) {
  if (threadIdx.x < 4) counters[threadIdx.x] = 0;
  if (threadIdx.x == 0 && dev_status) *dev_status = 0;
}

}  // namespace

size_t kde_workspace_bytes(int64_t n_events, int64_t cells) {
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  return 256 + al((size_t)n_events * 8) + al((size_t)cells * 4) + al((size_t)cells * 4);
}

hipError_t launch_kde(const KdeLaunch& l, hipStream_t st) {
  hipError_t e = ensure_pow_table();
  if (e != hipSuccess) return e;
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const int64_t cells = (int64_t)l.n_seg * l.n_kernels;
  char* ws = static_cast<char*>(l.workspace);
  KdeArgs a{};
  a.kernel_id = l.kernel_id;
  a.stream = l.stream;
  a.start_ns = l.start_ns;
  a.end_ns = l.end_ns;
  a.seg_off = l.seg_off;
  a.n_events = l.n_events;
  a.n_seg = l.n_seg;
  a.K = l.n_kernels;
  a.NS = l.n_streams;
  a.sub_bits = l.p.sub_bits;
  a.frac_pm = l.p.frac_pm;
  a.min_count = l.p.min_count;
  a.gap = l.p.gap;
  a.count = l.count;
  a.min_ns = l.min_ns;
  a.max_ns = l.max_ns;
  a.n_clusters = l.o.n_clusters;
  a.cl_count = l.o.count;
  a.p50 = l.o.p50_ns;
  a.p99 = l.o.p99_ns;
  a.bw_q8 = l.o.bw_q8;
  a.dev_status = l.o.dev_status;
  a.counters = reinterpret_cast<uint32_t*>(ws);
  a.bucket = reinterpret_cast<uint64_t*>(ws + 256);
  a.cell_end = reinterpret_cast<uint32_t*>(ws + 256 + al((size_t)l.n_events * 8));
  a.deferred = reinterpret_cast<uint32_t*>(ws + 256 + al((size_t)l.n_events * 8) + al((size_t)cells * 4));
  const uint32_t* th = thresholds();
  for (int t = 0; t < 64; ++t) a.theta[t] = th[t];

  hipLaunchKernelGGL(kde_clear_kernel, dim3(1), dim3(64), 0, st, a.counters, a.dev_status);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (cells == 0) return hipSuccess;

  // resident workgroups per kernel, cached per device
  static std::atomic<int> grids[64][3];
  int dev = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  int gs = grids[dev][0].load(), gf = grids[dev][1].load(), gl = grids[dev][2].load();
  if (gs == 0) grids[dev][0].store(gs = resident(kde_scatter_kernel, kScatterThreads));
  if (gf == 0) grids[dev][1].store(gf = resident(kde_cell_kernel<kFastWords, kFastCand, false>, kWave));
  if (gl == 0) grids[dev][2].store(gl = resident(kde_cell_kernel<kSlowWords, kSlowCand, true>, kWave));
  if (gs <= 0 || gf <= 0 || gl <= 0) return hipErrorInvalidDevice;
  const int g1 = l.n_seg < gs ? l.n_seg : gs;
  hipLaunchKernelGGL(kde_scatter_kernel, dim3(g1), dim3(kScatterThreads), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int64_t chunks = (cells + kWave - 1) / kWave;
  const int g2 = chunks < gf ? (int)chunks : gf;
  hipLaunchKernelGGL((kde_cell_kernel<kFastWords, kFastCand, false>), dim3(g2), dim3(kWave), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL((kde_cell_kernel<kSlowWords, kSlowCand, true>), dim3(gl), dim3(kWave), 0, st, a);
  return hipGetLastError();
}

}  // namespace argus
