// L1 iteration-level detection over per-rank step times (paper section 6.1
// and Appendix B): sliding-window ratio-gated jitter detection with
// effective-width measurement, and full-scan change-point detection; the two
// together classify a rank's series as stable, jitter, regression or both.
//
// One 64-lane wavefront per rank. The series lives in LDS; per-point marks
// (covered by a candidate window, above the baseline) are 64-bit ballot
// words, so merged intervals and longest runs come from bit operations; the
// baseline median is a wavefront radix select; prefix sums for the change
// point are a chunked wavefront scan. All decisions are exact integer
// comparisons (128-bit products, 256-bit where the relative-std test needs
// them).
#include "argus_internal.h"

namespace argus {
namespace {

typedef unsigned __int128 u128;
constexpr int64_t kYLimit = (int64_t)1 << 40;

// a * b as a 256-bit (hi, lo) pair
__device__ __forceinline__ void mul_128x128(u128 a, u128 b, u128& hi, u128& lo) {
  const uint64_t a0 = (uint64_t)a, a1 = (uint64_t)(a >> 64), b0 = (uint64_t)b, b1 = (uint64_t)(b >> 64);
  const u128 p00 = (u128)a0 * b0, p01 = (u128)a0 * b1, p10 = (u128)a1 * b0, p11 = (u128)a1 * b1;
  const u128 mid = (p00 >> 64) + (uint64_t)p01 + (uint64_t)p10;
  lo = (u128)(uint64_t)p00 | (mid << 64);
  hi = p11 + (p01 >> 64) + (p10 >> 64) + (mid >> 64);
}

// sign of a*b - c*d
__device__ __forceinline__ int cmp_prod(u128 a, u128 b, u128 c, u128 d) {
  u128 h1, l1, h2, l2;
  mul_128x128(a, b, h1, l1);
  mul_128x128(c, d, h2, l2);
  if (h1 != h2) return h1 < h2 ? -1 : 1;
  if (l1 != l2) return l1 < l2 ? -1 : 1;
  return 0;
}

// sample (n-1) relative std <= cmax_pm / 1000, exactly
__device__ __forceinline__ bool rel_std_ok(int64_t n, u128 s, u128 q, int32_t cmax_pm) {
  const u128 v = (u128)n * q - s * s;
  return cmp_prod((u128)1000000u * (u128)n, v, (u128)cmax_pm * (u128)cmax_pm * (u128)(n - 1), s * s) <= 0;
}

// inclusive prefix over the wavefront of a 128-bit value
__device__ __forceinline__ u128 wave_incl_scan128(u128 v) {
  const int lane = threadIdx.x & 63;
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t lo = __shfl_up((uint64_t)v, o, 64), hi = __shfl_up((uint64_t)(v >> 64), o, 64);
    if (lane >= o) v += ((u128)hi << 64) | lo;
  }
  return v;
}

struct Args {
  const int64_t* step_ns;
  int32_t R, S;
  argus_l1_params_t p;
  uint8_t* flags;
  uint8_t* cls;
  int32_t* eff_width;
  int32_t* cp;
  float* cp_ratio;
  int32_t* dev_status;
};

template <int SCAP>
struct L1Smem {
  int64_t y[SCAP];
  uint64_t pre_s[SCAP + 1];
  u128 pre_q[SCAP + 1];
  uint8_t candw[SCAP];      // window t is a candidate
  uint8_t fl[SCAP];         // output flag bits 0-1 per point
  uint64_t cov[SCAP / 64];  // bit i: point i covered by a candidate window
  uint32_t hist[256];
  int32_t iv[SCAP / 2 + 1][2];  // merged intervals [a, b] (separated by uncovered points)
  u128 best_num[64], best_den[64];
  int32_t best_t[64];
  int32_t n_iv, width, cpt;
  uint32_t digit, before;
};

// Lower median (rank (m-1)/2) of y over the m points outside [ea, eb] (no
// exclusion when ea > eb), by MSD radix select over 8-bit digits of y
// (every y < 2^40). Wavefront-wide.
template <int SCAP>
__device__ int64_t wave_lower_median(L1Smem<SCAP>& sm, int S, int ea, int eb) {
  const int lane = threadIdx.x & 63;
  uint32_t m = 0;
  for (int i = lane; i < S; i += 64) m += !(i >= ea && i <= eb);
  for (int o = 32; o > 0; o >>= 1) m += __shfl_xor(m, o, 64);
  uint32_t k = (m - 1) / 2;
  uint64_t prefix = 0;
  for (int shift = 32; shift >= 0; shift -= 8) {
    for (int b = lane; b < 256; b += 64) sm.hist[b] = 0;
    __syncthreads();
    for (int i = lane; i < S; i += 64) {
      if (i >= ea && i <= eb) continue;
      const uint64_t v = (uint64_t)sm.y[i];
      if (shift == 32 || (v >> (shift + 8)) == prefix) atomicAdd(&sm.hist[(v >> shift) & 255u], 1u);
    }
    __syncthreads();
    // lane owns bins 4 lane .. 4 lane + 3
    uint32_t h[4], tot = 0;
    for (int j = 0; j < 4; ++j) {
      h[j] = sm.hist[4 * lane + j];
      tot += h[j];
    }
    uint32_t incl = tot;
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t n = __shfl_up(incl, o, 64);
      if (lane >= o) incl += n;
    }
    uint32_t run = incl - tot;
    for (int j = 0; j < 4; ++j) {
      if (run <= k && k < run + h[j]) {
        sm.digit = 4 * lane + j;
        sm.before = run;
      }
      run += h[j];
    }
    __syncthreads();
    prefix = (prefix << 8) | sm.digit;
    k -= sm.before;
    __syncthreads();
  }
  return (int64_t)prefix;
}

template <int SCAP>
__global__ __launch_bounds__(64) void l1_kernel(Args a) {
  __shared__ L1Smem<SCAP> sm;
  const int lane = threadIdx.x;
  const int64_t r = blockIdx.x;
  const int S = a.S;
  if (S == 0) {
    if (lane == 0) {
      a.cls[r] = 0;
      a.eff_width[r] = 0;
      a.cp[r] = -1;
      if (a.cp_ratio) a.cp_ratio[r] = 0.0f;
    }
    return;
  }
  const int64_t* yr = a.step_ns + r * S;
  bool ok = true;
  for (int i = lane; i < S; i += 64) {
    const int64_t v = yr[i];
    sm.y[i] = v;
    sm.fl[i] = 0;
    ok &= v >= 0 && v < kYLimit;
  }
  ok = __all(ok);
  __syncthreads();
  if (!ok) {
    for (int i = lane; i < S; i += 64) a.flags[r * S + i] = 0;
    if (lane == 0) {
      a.cls[r] = 0x80;
      a.eff_width[r] = 0;
      a.cp[r] = -1;
      if (a.cp_ratio) a.cp_ratio[r] = 0.0f;
      if (a.dev_status) atomicOr(a.dev_status, (int32_t)ARGUS_DEV_L1_DOMAIN);
    }
    return;
  }

  // sensitivity gating: window t = [t, t+w-1] is a candidate when its
  // max/min ratio exceeds theta
  const int w = a.p.W < S ? a.p.W : S;
  const int nwin = S - w + 1;
  for (int t = lane; t < nwin; t += 64) {
    int64_t mx = sm.y[t], mn = sm.y[t];
    for (int i = t + 1; i < t + w; ++i) {
      mx = sm.y[i] > mx ? sm.y[i] : mx;
      mn = sm.y[i] < mn ? sm.y[i] : mn;
    }
    sm.candw[t] = (u128)1000u * (u128)mx > (u128)a.p.theta_pm * (u128)mn;
  }
  __syncthreads();
  // point i is covered when a candidate window contains it
  for (int i0 = 0; i0 < S; i0 += 64) {
    const int i = i0 + lane;
    bool c = false;
    if (i < S) {
      const int t_lo = i - w + 1 > 0 ? i - w + 1 : 0, t_hi = i < nwin - 1 ? i : nwin - 1;
      for (int t = t_lo; t <= t_hi && !c; ++t) c = sm.candw[t] != 0;
    }
    const unsigned long long word = __ballot(c);
    if (lane == 0) sm.cov[i0 >> 6] = word;
  }
  __syncthreads();
  // merged intervals: maximal runs of covered points (overlapping or
  // touching candidate windows merge)
  if (lane == 0) {
    int n = 0, i = 0;
    while (i < S) {
      const uint64_t rest = sm.cov[i >> 6] >> (i & 63);
      if (rest == 0) {
        i = ((i >> 6) + 1) << 6;
        continue;
      }
      i += __builtin_ctzll(rest);
      if (i >= S) break;
      int j = i;  // first uncovered point at or after i
      while (j < S) {
        const uint64_t ones = sm.cov[j >> 6] >> (j & 63);
        const int avail = 64 - (j & 63);
        int len = ~ones == 0 ? 64 : __builtin_ctzll(~ones);
        if (len > avail) len = avail;
        j += len;
        if (len < avail) break;
      }
      if (j > S) j = S;
      sm.iv[n][0] = i;
      sm.iv[n][1] = j - 1;
      ++n;
      i = j;
    }
    sm.n_iv = n;
    sm.width = 0;
  }
  __syncthreads();
  const int n_iv = sm.n_iv;
  for (int q = 0; q < n_iv; ++q) {
    const int ia = sm.iv[q][0], ib = sm.iv[q][1];
    // baseline: lower median of the points outside [ia, ib], of all points
    // when none lie outside
    const bool all_inside = ia == 0 && ib == S - 1;
    const int64_t base = all_inside ? wave_lower_median(sm, S, 1, 0) : wave_lower_median(sm, S, ia, ib);
    // points significantly above the baseline; the longest contiguous run
    // of them is the interval's effective width (wave-uniform bit scan)
    int best = 0, run = 0;
    for (int i0 = ia; i0 <= ib; i0 += 64) {
      const int i = i0 + lane;
      bool ex = false;
      if (i <= ib) {
        ex = (u128)1000u * (u128)sm.y[i] > (u128)a.p.beta_pm * (u128)base;
        sm.fl[i] = ex ? 3 : 1;
      }
      const uint64_t word = __ballot(ex);
      const int nbits = ib - i0 + 1 < 64 ? ib - i0 + 1 : 64;
      int b = 0;
      while (b < nbits) {
        const uint64_t rest = word >> b;
        if (rest & 1u) {
          int len = ~rest == 0 ? 64 - b : __builtin_ctzll(~rest);
          if (b + len > nbits) len = nbits - b;
          run += len;
          best = run > best ? run : best;
          b += len;
        } else {
          run = 0;
          b = rest == 0 ? nbits : b + __builtin_ctzll(rest);
        }
      }
    }
    if (lane == 0 && best > sm.width) sm.width = best;
    __syncthreads();
  }

  // change point: chunked prefix sums (each lane sums a contiguous chunk,
  // one wavefront scan of the chunk totals, then each lane fills its chunk)
  const int chunk = (S + 63) / 64;
  const int c0 = lane * chunk, c1 = c0 + chunk < S ? c0 + chunk : S;
  uint64_t ls = 0;
  u128 lq = 0;
  for (int i = c0; i < c1; ++i) {
    ls += (uint64_t)sm.y[i];
    lq += (u128)(uint64_t)sm.y[i] * (u128)(uint64_t)sm.y[i];
  }
  uint64_t es = ls;
  for (int o = 1; o < 64; o <<= 1) {
    const uint64_t n = __shfl_up(es, o, 64);
    if (lane >= o) es += n;
  }
  es -= ls;
  u128 eq = wave_incl_scan128(lq) - lq;
  if (lane == 0) {
    sm.pre_s[0] = 0;
    sm.pre_q[0] = 0;
  }
  for (int i = c0; i < c1; ++i) {
    es += (uint64_t)sm.y[i];
    eq += (u128)(uint64_t)sm.y[i] * (u128)(uint64_t)sm.y[i];
    sm.pre_s[i + 1] = es;
    sm.pre_q[i + 1] = eq;
  }
  __syncthreads();
  int32_t bt = -1;
  u128 bn = 0, bd = 1;
  const int ms = a.p.min_seg;
  for (int t = (ms > 1 ? ms : 1) + lane; t <= S - ms; t += 64) {
    const u128 sl = sm.pre_s[t], ql = sm.pre_q[t];
    const u128 sr = (u128)sm.pre_s[S] - sl, qr = sm.pre_q[S] - ql;
    const int64_t nl = t, nr = S - t;
    if (sl == 0) continue;  // the ratio needs a positive left mean
    const u128 num = sr * (u128)nl, den = sl * (u128)nr;
    if ((u128)1000u * num < (u128)a.p.rho_pm * den) continue;
    if (!rel_std_ok(nl, sl, ql, a.p.cmax_pm) || !rel_std_ok(nr, sr, qr, a.p.cmax_pm)) continue;
    if (bt < 0 || cmp_prod(num, bd, bn, den) > 0) {
      bt = t;
      bn = num;
      bd = den;
    }
  }
  sm.best_t[lane] = bt;
  sm.best_num[lane] = bn;
  sm.best_den[lane] = bd;
  __syncthreads();
  if (lane == 0) {
    int32_t t0 = -1;
    u128 n0 = 0, d0 = 1;
    for (int l = 0; l < 64; ++l) {
      const int32_t t = sm.best_t[l];
      if (t < 0) continue;
      const int c = t0 < 0 ? 1 : cmp_prod(sm.best_num[l], d0, n0, sm.best_den[l]);
      if (c > 0 || (c == 0 && t < t0)) {
        t0 = t;
        n0 = sm.best_num[l];
        d0 = sm.best_den[l];
      }
    }
    sm.cpt = t0;
    a.cp[r] = t0;
    if (a.cp_ratio) a.cp_ratio[r] = t0 >= 0 ? (float)((double)n0 / (double)d0) : 0.0f;
    a.eff_width[r] = sm.width;
    a.cls[r] = (uint8_t)((sm.width > 0 ? 1 : 0) | (t0 >= 0 ? 2 : 0));
  }
  __syncthreads();
  const int cpt = sm.cpt;
  for (int i = lane; i < S; i += 64) a.flags[r * S + i] = sm.fl[i] | ((cpt >= 0 && i >= cpt) ? 4 : 0);
}

template <int SCAP>
hipError_t launch_t(const Args& args, hipStream_t st) {
  hipLaunchKernelGGL(l1_kernel<SCAP>, dim3(args.R), dim3(64), 0, st, args);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_iter_windows(const IterWindowsLaunch& l, hipStream_t st) {
  Args a{l.step_ns, l.R, l.S, l.p, l.flags, l.cls, l.eff_width, l.cp, l.cp_ratio, l.dev_status};
  if (l.R == 0) return hipSuccess;
  if (l.S <= 64) return launch_t<64>(a, st);
  if (l.S <= 512) return launch_t<512>(a, st);
  if (l.S <= 1024) return launch_t<1024>(a, st);
  return launch_t<ARGUS_MAX_L1_STEPS>(a, st);
}

}  // namespace argus
