// L1 iteration-level detection over per-rank step times (paper section 6.1
// and Appendix B): sliding-window ratio-gated jitter detection with
// effective-width measurement, and full-scan change-point detection; the two
// together classify a rank's series as stable, jitter, regression or both.
//
// One 64-lane wavefront per rank; the series, candidate marks and prefix
// sums live in LDS. All decisions are exact integer comparisons (128-bit
// products, 256-bit where the relative-std test needs them).
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
__global__ __launch_bounds__(64) void l1_kernel(Args a) {
  __shared__ int64_t y[SCAP];
  __shared__ uint8_t cand[SCAP];
  __shared__ uint8_t fl[SCAP];
  __shared__ uint64_t pre_s[SCAP + 1];
  __shared__ u128 pre_q[SCAP + 1];
  __shared__ u128 best_num[64], best_den[64];
  __shared__ int32_t best_t[64];
  __shared__ int32_t iv_a, iv_b, width_sh;
  __shared__ int64_t base_sh;

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
    y[i] = v;
    cand[i] = 0;
    fl[i] = 0;
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

  // sensitivity gating: windows whose max/min ratio exceeds theta
  const int w = a.p.W < S ? a.p.W : S;
  for (int t = lane; t + w <= S; t += 64) {
    int64_t mx = y[t], mn = y[t];
    for (int i = t + 1; i < t + w; ++i) {
      mx = y[i] > mx ? y[i] : mx;
      mn = y[i] < mn ? y[i] : mn;
    }
    if ((u128)1000u * (u128)mx > (u128)a.p.theta_pm * (u128)mn)
      for (int i = t; i < t + w; ++i) cand[i] = 1;
  }
  __syncthreads();

  // effective width per merged interval (maximal run of candidate points)
  if (lane == 0) {
    width_sh = 0;
    iv_b = -1;
  }
  __syncthreads();
  while (true) {
    if (lane == 0) {
      int s0 = iv_b + 1;
      while (s0 < S && !cand[s0]) ++s0;
      int e0 = s0;
      while (e0 + 1 < S && cand[e0 + 1]) ++e0;
      iv_a = s0 < S ? s0 : -1;
      iv_b = e0;
    }
    __syncthreads();
    const int ia = iv_a, ib = iv_b;
    if (ia < 0) break;
    // baseline: lower median of the points outside [ia, ib] (all if none),
    // found by counting: v is the target-th smallest iff
    // #{< v} <= target < #{<= v}
    const int m_out = S - (ib - ia + 1);
    const bool use_all = m_out == 0;
    const int target = ((use_all ? S : m_out) - 1) / 2;
    for (int j = lane; j < S; j += 64) {
      if (!use_all && j >= ia && j <= ib) continue;
      const int64_t v = y[j];
      int lt = 0, le = 0;
      for (int i = 0; i < S; ++i) {
        if (!use_all && i >= ia && i <= ib) continue;
        lt += y[i] < v;
        le += y[i] <= v;
      }
      if (lt <= target && target < le) base_sh = v;
    }
    __syncthreads();
    if (lane == 0) {
      const int64_t base = base_sh;
      int run = 0, best = width_sh;
      for (int i = ia; i <= ib; ++i) {
        uint8_t f = 1;
        if ((u128)1000u * (u128)y[i] > (u128)a.p.beta_pm * (u128)base) {
          f |= 2;
          ++run;
          best = run > best ? run : best;
        } else {
          run = 0;
        }
        fl[i] = f;
      }
      width_sh = best;
    }
    __syncthreads();
  }

  // change point: prefix sums, then each lane scans its share of splits
  if (lane == 0) {
    uint64_t s = 0;
    u128 q = 0;
    pre_s[0] = 0;
    pre_q[0] = 0;
    for (int i = 0; i < S; ++i) {
      s += (uint64_t)y[i];
      q += (u128)(uint64_t)y[i] * (u128)(uint64_t)y[i];
      pre_s[i + 1] = s;
      pre_q[i + 1] = q;
    }
  }
  __syncthreads();
  int32_t bt = -1;
  u128 bn = 0, bd = 1;
  const int ms = a.p.min_seg;
  for (int t = (ms > 1 ? ms : 1) + lane; t <= S - ms; t += 64) {
    const u128 sl = pre_s[t], ql = pre_q[t];
    const u128 sr = (u128)pre_s[S] - sl, qr = pre_q[S] - ql;
    const int64_t nl = t, nr = S - t;
    if (sl == 0) continue;
    const u128 num = sr * (u128)nl, den = sl * (u128)nr;
    if ((u128)1000u * num < (u128)a.p.rho_pm * den) continue;
    if (!rel_std_ok(nl, sl, ql, a.p.cmax_pm) || !rel_std_ok(nr, sr, qr, a.p.cmax_pm)) continue;
    if (bt < 0 || cmp_prod(num, bd, bn, den) > 0) {
      bt = t;
      bn = num;
      bd = den;
    }
  }
  best_t[lane] = bt;
  best_num[lane] = bn;
  best_den[lane] = bd;
  __syncthreads();
  if (lane == 0) {
    int32_t t0 = -1;
    u128 n0 = 0, d0 = 1;
    for (int l = 0; l < 64; ++l) {
      const int32_t t = best_t[l];
      if (t < 0) continue;
      const int c = t0 < 0 ? 1 : cmp_prod(best_num[l], d0, n0, best_den[l]);
      if (c > 0 || (c == 0 && t < t0)) {
        t0 = t;
        n0 = best_num[l];
        d0 = best_den[l];
      }
    }
    iv_a = t0;
    a.cp[r] = t0;
    if (a.cp_ratio) a.cp_ratio[r] = t0 >= 0 ? (float)((double)n0 / (double)d0) : 0.0f;
    a.eff_width[r] = width_sh;
    a.cls[r] = (uint8_t)((width_sh > 0 ? 1 : 0) | (t0 >= 0 ? 2 : 0));
  }
  __syncthreads();
  const int cpt = iv_a;
  for (int i = lane; i < S; i += 64) a.flags[r * S + i] = fl[i] | ((cpt >= 0 && i >= cpt) ? 4 : 0);
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
