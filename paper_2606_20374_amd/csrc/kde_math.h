// The log grid and the floating-point steps of the KDE clustering definition
// (section 5.2, Eq. 1: log-duration grid, Gaussian kernel, bandwidth 1.06
// sigma n^(-1/5)), one copy for every cell tier. The integer outputs follow
// from these results exactly. The grid index and n^(-1/5) are decided
// exactly (no math library involved); sqrt is correctly rounded; exp enters
// the weights, and a GPU test evaluates these same functions over their
// whole reachable domain against the oracle and the host C library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>
#include <vector>

namespace argus {

// ------------------------------------------------------------ the log grid
// Bit length of m^64, exactly (big-integer squaring, six times).
inline int kde_bitlen_pow64(uint32_t m) {
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
  return 32 * (int)(x.size() - 1) + (32 - __builtin_clz(x.back()));
}

// The 64 mantissa thresholds ceil(2^(23 + t/64)) of the grid (host, computed
// once): the smallest m with floor(log2(m^64)) >= 1472 + t, by bisection.
inline const uint32_t* kde_thresholds() {
  static uint32_t th[64];
  static std::once_flag once;
  std::call_once(once, [] {
    th[0] = 1u << 23;
    for (int t = 1; t < 64; ++t) {
      uint32_t lo = 1u << 23, hi = (1u << 24) - 1;
      while (lo < hi) {
        const uint32_t mid = lo + (hi - lo) / 2;
        if (kde_bitlen_pow64(mid) - 1 >= 1472 + t) hi = mid;
        else lo = mid + 1;
      }
      th[t] = lo;
    }
  });
  return th;
}

// Grid index floor(64 log2 d') of a duration d >= 2, with d' its 24 leading
// significant bits (exact below 2^24 ns); 0 for d < 2. A hardware log2
// estimate is checked against the exact thresholds th (kde_thresholds): the
// estimate's bracket [th[t], th[t + 1]) is read at once, a result equal to
// the estimate is proved by those two comparisons, and only an estimate off
// by a step (a mantissa next to a threshold) walks the table to the exact
// index. kde_grid_of_mantissa takes d's exponent e = floor(log2 d) and m = d'
// (in [2^23, 2^24)).
__device__ __forceinline__ int kde_grid_of_mantissa(int e, uint32_t m, const uint32_t* th) {
  int t0 = (int)((__log2f((float)m) - 23.0f) * 64.0f);
  t0 = t0 < 0 ? 0 : (t0 > 63 ? 63 : t0);
  const uint32_t a0 = th[t0], a1 = th[t0 < 63 ? t0 + 1 : 63];
  int t = t0 - 1 + (m >= a0 ? 1 : 0) + (t0 < 63 && m >= a1 ? 1 : 0);
  if (t != t0) {
    t = t < 0 ? 0 : t;
    while (t > 0 && m < th[t]) --t;
    while (t < 63 && m >= th[t + 1]) ++t;
  }
  return e * 64 + t;
}

__device__ __forceinline__ int kde_grid64(uint64_t d, const uint32_t* th) {
  if (d < 2) return 0;
  const int e = 63 - __builtin_clzll(d);
  return kde_grid_of_mantissa(e, e >= 23 ? (uint32_t)(d >> (e - 23)) : (uint32_t)(d << (23 - e)), th);
}

// The same index for a duration held in 32 bits (4-byte records): the same
// exponent and mantissa from 32-bit operations.
__device__ __forceinline__ int kde_grid32(uint32_t d, const uint32_t* th) {
  if (d < 2) return 0;
  const int e = 31 - __builtin_clz(d);
  return kde_grid_of_mantissa(e, e >= 23 ? d >> (e - 23) : d << (23 - e), th);
}

// Sign of c^5 n - 2^e, exactly (c < 2^55, n < 2^33, so the product has at
// most 308 bits: six 64-bit limbs).
__device__ inline int kde_fifth_cmp(uint64_t c, uint64_t n, int e) {
  uint64_t a[6] = {1, 0, 0, 0, 0, 0};
#pragma unroll 1
  for (int r = 0; r < 6; ++r) {
    const uint64_t m = r < 5 ? c : n;
    unsigned __int128 carry = 0;
#pragma unroll
    for (int i = 0; i < 6; ++i) {
      const unsigned __int128 v = (unsigned __int128)a[i] * m + carry;
      a[i] = (uint64_t)v;
      carry = v >> 64;
    }
  }
  int top = 5;
  while (top > 0 && a[top] == 0) --top;
  const int bits = 64 * top + (a[top] ? 64 - __builtin_clzll(a[top]) : 0);
  if (bits != e + 1) return bits > e + 1 ? 1 : -1;
  for (int i = 0; i < 6; ++i)
    if (a[i] != (i == e / 64 ? (1ull << (e % 64)) : 0ull)) return 1;
  return 0;
}

// n^(-1/5) for the bandwidth: the double nearest to the real value, for
// 1 <= n < 2^33. Starting from the device pow (a few units in the last place
// off), the candidate y = M 2^q (M in [2^52, 2^53)) moves one unit at a time
// until z = n^(-1/5) lies between the midpoints to its neighbours; z < c 2^k
// iff c^5 n > 2^(-5k). Below a power of two the lower neighbour is half a
// unit away, so that midpoint is (4M - 1) 2^(q-2). Out of line: the cell
// kernels call it only for cells of 65,536 or more durations (the others
// read a table this function filled).
__device__ __attribute__((noinline)) inline double kde_pw(uint64_t n) {
  double y = pow((double)n, -0.2);
  for (int it = 0; it < 64; ++it) {
    const uint64_t bits = (uint64_t)__double_as_longlong(y);
    const uint64_t M = (bits & ((1ull << 52) - 1)) | (1ull << 52);
    const int q = (int)(bits >> 52) - 1075;
    if (kde_fifth_cmp(2 * M + 1, n, 5 * (1 - q)) <= 0) {  // z above the upper midpoint
      y = __longlong_as_double((long long)(bits + 1));
      continue;
    }
    const int below = M == (1ull << 52) ? kde_fifth_cmp(4 * M - 1, n, 5 * (2 - q))
                                        : kde_fifth_cmp(2 * M - 1, n, 5 * (1 - q));
    if (below >= 0) {  // z below the lower midpoint
      y = __longlong_as_double((long long)(bits - 1));
      continue;
    }
    break;
  }
  return y;
}

// Quantised bandwidth H = floor(256 h + 0.5), h = 1.06 sqrt(var) n^(-1/5),
// in 1/256 grid steps; pw = kde_pw(n).
__device__ __forceinline__ int64_t kde_bw_q8(double var, double pw) {
  const double h = 1.06 * sqrt(var) * pw;
  return (int64_t)floor(h * 256.0 + 0.5);
}

// Integer Gaussian weight of grid distance t for bandwidth H (H2 = H * H as
// a double): floor(65536 exp(-t^2 / (2 (H / 256)^2)) + 0.5).
__device__ __forceinline__ uint32_t kde_weight(int t, double H2) {
  return (uint32_t)floor(65536.0 * exp(-(double)(32768ll * t * t) / H2) + 0.5);
}

}  // namespace argus
