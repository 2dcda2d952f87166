// Cross-rank Wasserstein-1 deviation scores over the duration clusters of
// every (step, kernel) (section 6.2, Eq. 2 - 4; the step-by-step definition
// is in include/argus.h).
//
// Launches, in order:
//   w1_init     per (step, kernel): n_present = 0 and the identities of the
//               grid-bound minimum / maximum.
//   w1_bounds   one lane per kernel id (64 ids x 64 ranks per workgroup, so
//               the cluster records of neighbouring ids are read together):
//               present ranks, grid bounds lo / hi by 64-bit atomics,
//               malformed records.
//   w1_cdf      one lane per rank (64 ranks of one kernel id per wavefront,
//               eight kernel ids per wavefront): the count-weighted lognormal
//               mixture of Eq. 2 at every grid point, quantised to 16 bits,
//               into a [S][K][G][R'] workspace (R' = R rounded up to even;
//               ranks contiguous, so the writes and the next kernel's reads
//               are coalesced). Phi comes from a cubic Hermite table (error
//               below 2e-10); a grid point
//               whose quantised value is not settled by that bound (within
//               1e-4 of a step of 2^-16) is recomputed with erfc in double,
//               the defining formula, so every output equals the erfc form.
//   w1_score    one workgroup per (step, kernel): for each grid point the
//               exact sums S_a = sum_b |q_a - q_b| over all present ranks
//               from a counting sort of the 16-bit values in LDS (a
//               256-bucket histogram, then the 256 bins of each occupied
//               bucket, 16-bit counters two to a word) and a prefix sum over
//               the sorted values: with c the number of values below q_a and
//               P their sum, S_a = q_a (2 c - n) + T - 2 P. The trapezoid
//               weights are applied in grid order, then the lower
//               nearest-rank quartiles of the scores come from a radix
//               selection on their bit patterns (non-negative doubles order
//               like their bits), then the upper fence of Eq. 4 and the
//               flags, written to the workspace contiguously.
//               Workgroups are numbered so that neighbouring kernel ids run
//               on one XCD.
//   w1_out      the scores and flags from the workspace to the
//               [rank][step][kernel] outputs through 64 x 64 LDS tiles.
// The pairwise matrix of the paper is never formed: S_a is the row sum of
// |F_a - F_b| at one grid point, which is all the mean-W1 score needs.
#include <cmath>
#include <mutex>
#include <vector>

#include "argus_internal.h"
#include "argus_select.h"

namespace argus {
namespace {

typedef unsigned __int128 u128;

constexpr int kMaxC = ARGUS_KDE_MAXC;
constexpr double kZ99 = 2.326;                     // standard normal 99th percentile, as printed (Eq. 2)
constexpr double kSqrt2 = 1.41421356237309504880;  // Phi(z) = erfc(-z / sqrt 2) / 2
constexpr int kFineWords = 32768;                  // 65536 16-bit bin counters, two per word

// Phi(z) by cubic Hermite interpolation on [-kPhiZ, kPhiZ] in steps of
// 1/kPhiSteps; outside, 0 or 1 (Phi(-8) < 6.3e-16). The interpolation error
// is at most h^4 / 384 max|Phi''''| <= 1.6e-10 (h = 1/64, |Phi''''| =
// |z^3 - 3z| phi(z) <= 1.2), about 1e-5 of a 2^-16 step of the mixture; with
// rounding the quantised value is certain once v +- kBand fall in one step.
constexpr double kPhiZ = 8.0;
constexpr int kPhiSteps = 64;
constexpr int kPhiN = 2 * 8 * kPhiSteps;  // intervals
constexpr double kBand = 1e-4;            // in units of 2^-16
constexpr int kCdfKPerWave = 8;

// per interval i (z from -kPhiZ + i / kPhiSteps), the cubic in t in [0, 1]:
// c0 + t (c1 + t (c2 + t c3)); filled once per device from the host's erfc / exp
__device__ double g_phi_tab[kPhiN * 4];

struct W1Args {
  const uint8_t* ncl;
  const uint32_t* cnt;
  const int64_t* p50;
  const int64_t* p99;
  int32_t R, S, K, G, min_ranks, alpha_pm;
  argus_w1_out_t o;
  uint16_t* q;  // workspace [S][K][G][R rounded up to even]
};

// Workspace layout: the CDF values, one block per (step, kernel) of G rows
// of R' 16-bit values, R' (the row stride) the rank count rounded up to
// even, so that the values of ranks 2p and 2p + 1 share one aligned 32-bit
// word; then, 256-byte aligned, the scores ([step, kernel][R'] doubles) and
// the flags ([step, kernel][R'] bytes) on their way to the
// [rank][step][kernel] outputs.
__host__ __device__ __forceinline__ int64_t ws_row_stride(int32_t R) { return (int64_t)R + (R & 1); }
__host__ __device__ __forceinline__ int64_t ws_q_bytes(int32_t R, int32_t S, int32_t K, int32_t G) {
  return ((int64_t)S * K * G * ws_row_stride(R) * 2 + 255) & ~(int64_t)255;
}
__device__ __forceinline__ int64_t row_stride(const W1Args& a) { return ws_row_stride(a.R); }
__device__ __forceinline__ uint16_t* ws_block(const W1Args& a, int64_t sk) {
  return a.q + sk * a.G * ws_row_stride(a.R);
}
__device__ __forceinline__ double* ws_scores(const W1Args& a, int64_t sk) {
  return reinterpret_cast<double*>(reinterpret_cast<char*>(a.q) + ws_q_bytes(a.R, a.S, a.K, a.G)) +
         sk * ws_row_stride(a.R);
}
__device__ __forceinline__ uint8_t* ws_flags(const W1Args& a, int64_t sk) {
  const int64_t SK = (int64_t)a.S * a.K, rs = ws_row_stride(a.R);
  return reinterpret_cast<uint8_t*>(reinterpret_cast<char*>(a.q) + ws_q_bytes(a.R, a.S, a.K, a.G) + SK * rs * 8) +
         sk * rs;
}

__device__ __forceinline__ int64_t cell_of(const W1Args& a, int r, int s, int k) {
  return ((int64_t)r * a.S + s) * a.K + k;
}

// 1: usable cluster record, 0: absent, -1: malformed (more clusters than the
// record holds, or clusters of total count 0). tot: total count.
__device__ __forceinline__ int cell_state(const W1Args& a, int64_t c, uint32_t& nc, uint64_t& tot) {
  nc = a.ncl[c];
  tot = 0;
  if (nc == 0) return 0;
  if (nc > kMaxC) return -1;
  for (uint32_t cl = 0; cl < nc; ++cl) tot += a.cnt[c * kMaxC + cl];
  return tot > 0 ? 1 : -1;
}

// Cluster median and 99th percentile, at least 1 ns, p99 not below p50.
__device__ __forceinline__ void cluster_ab(const W1Args& a, int64_t c, uint32_t cl, uint64_t& x, uint64_t& y) {
  const int64_t p = a.p50[c * kMaxC + cl], t = a.p99[c * kMaxC + cl];
  x = p > 1 ? (uint64_t)p : 1;
  y = t > 1 ? (uint64_t)t : 1;
  if (y < x) y = x;
}

// floor(a / b) for a < 2^53, 1 <= b < 2^53: both are exact doubles, and the
// correctly rounded quotient truncates to the exact floor or one above it
// (never below: the floor is representable), which one exact product detects.
__device__ __forceinline__ uint64_t floor_div53(uint64_t a, uint64_t b) {
  uint64_t q = (uint64_t)((double)a / (double)b);
  if (q * b > a) --q;
  return q;
}

// floor(x^2 / y) and min(ceil(y^2 / x), INT64_MAX), for 1 <= x <= y: the
// lognormal's mirror of its 99th percentile below the median, and its
// 99.99th percentile.
__device__ __forceinline__ uint64_t lo_of(uint64_t x, uint64_t y) {
  if (x < (1ull << 26) && y < (1ull << 53)) return floor_div53(x * x, y);
  if (x < (1ull << 32)) return (x * x) / y;
  return (uint64_t)(((u128)x * x) / y);
}
__device__ __forceinline__ uint64_t hi_of(uint64_t x, uint64_t y) {
  if (y < (1ull << 26)) return floor_div53(y * y + (x - 1), x);  // x <= y
  u128 q;
  if (y < (1ull << 32))
    q = (y * y + (x - 1)) / x;
  else
    q = ((u128)y * y + (x - 1)) / x;
  return q > (u128)INT64_MAX ? (uint64_t)INT64_MAX : (uint64_t)q;
}

// ------------------------------------------------------------------- init
__global__ __launch_bounds__(256) void w1_init(W1Args a) {
  const int64_t sk = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (sk >= (int64_t)a.S * a.K) return;
  a.o.n_present[sk] = 0;
  a.o.lo_ns[sk] = -1;  // all ones: identity of the unsigned minimum
  a.o.hi_ns[sk] = 0;
}

// ----------------------------------------------------------------- bounds
__global__ __launch_bounds__(256) void w1_bounds(W1Args a) {
  __shared__ uint32_t n_sh[4][64];
  __shared__ unsigned long long lo_sh[4][64], hi_sh[4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int k = blockIdx.x * 64 + lane, s = blockIdx.z, r0 = blockIdx.y * 64;
  uint32_t n = 0;
  uint64_t lo = ~0ull, hi = 0;
  bool bad = false;
  if (k < a.K) {
    for (int i = w; i < 64; i += 4) {
      const int r = r0 + i;
      if (r >= a.R) break;
      const int64_t c = cell_of(a, r, s, k);
      uint32_t nc;
      uint64_t tot;
      const int st = cell_state(a, c, nc, tot);
      if (st < 0) bad = true;
      if (st <= 0) continue;
      ++n;
      for (uint32_t cl = 0; cl < nc; ++cl) {
        uint64_t x, y;
        cluster_ab(a, c, cl, x, y);
        const uint64_t l = lo_of(x, y), h = hi_of(x, y);
        lo = l < lo ? l : lo;
        hi = h > hi ? h : hi;
      }
    }
  }
  if (__ballot(bad) != 0 && lane == 0 && a.o.dev_status) atomicOr(a.o.dev_status, (int32_t)ARGUS_DEV_W1_INPUT);
  n_sh[w][lane] = n;
  lo_sh[w][lane] = lo;
  hi_sh[w][lane] = hi;
  __syncthreads();
  if (w != 0 || k >= a.K) return;
#pragma unroll
  for (int i = 1; i < 4; ++i) {
    n += n_sh[i][lane];
    lo = lo_sh[i][lane] < lo ? lo_sh[i][lane] : lo;
    hi = hi_sh[i][lane] > hi ? hi_sh[i][lane] : hi;
  }
  if (n == 0) return;
  const int64_t sk = (int64_t)s * a.K + k;
  atomicAdd(&a.o.n_present[sk], n);
  atomicMin(reinterpret_cast<unsigned long long*>(&a.o.lo_ns[sk]), (unsigned long long)lo);
  atomicMax(reinterpret_cast<unsigned long long*>(&a.o.hi_ns[sk]), (unsigned long long)hi);
}

__device__ __forceinline__ bool evaluated(const W1Args& a, uint32_t n) {
  return n >= (uint32_t)a.min_ranks && n >= 2;
}

// Grid coordinates of one (step, kernel): u_g = lnlo + g du.
__device__ __forceinline__ void grid_of(const W1Args& a, int64_t sk, double& lnlo, double& du) {
  const uint64_t lo = (uint64_t)a.o.lo_ns[sk], hi = (uint64_t)a.o.hi_ns[sk];
  lnlo = log((double)(lo < 1 ? 1 : lo));
  const double lnhi = log((double)hi);
  du = (lnhi - lnlo) / (double)(a.G - 1);
}

// -------------------------------------------------------------------- CDF
__device__ __forceinline__ uint32_t quant16(double v) {
  if (!(v > 0.0)) return 0u;
  const double f = floor(v);
  return f >= 65535.0 ? 65535u : (uint32_t)f;
}

__global__ __launch_bounds__(256) void w1_cdf(W1Args a) {
  __shared__ double tab[kPhiN * 4];
  for (int i = threadIdx.x; i < kPhiN * 4; i += 256) tab[i] = g_phi_tab[i];
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int r = blockIdx.y * 64 + lane, s = blockIdx.z;
  if (r >= a.R) return;
  for (int j = 0; j < kCdfKPerWave; ++j) {
    const int k = (blockIdx.x * 4 + w) * kCdfKPerWave + j;
    if (k >= a.K) break;
    const int64_t sk = (int64_t)s * a.K + k;
    if (!evaluated(a, a.o.n_present[sk])) continue;
    const int64_t c = cell_of(a, r, s, k);
    uint32_t nc;
    uint64_t tot;
    if (cell_state(a, c, nc, tot) <= 0) continue;
    double lnlo, du;
    grid_of(a, sk, lnlo, du);
    // per cluster: the table coordinate sx = kPhiSteps (z + kPhiZ) of grid
    // point g is sx0 + g dsx (its rounding differs from the direct form's by
    // far less than the band below allows for)
    double mu[kMaxC], den[kMaxC], wt[kMaxC], sx0[kMaxC], dsx[kMaxC];
    bool spread[kMaxC];
#pragma unroll
    for (int cl = 0; cl < kMaxC; ++cl) {
      mu[cl] = den[cl] = wt[cl] = sx0[cl] = dsx[cl] = 0.0;
      spread[cl] = false;
      if ((uint32_t)cl >= nc) continue;
      const int64_t p = a.p50[c * kMaxC + cl], t = a.p99[c * kMaxC + cl];
      const double x = p > 1 ? (double)p : 1.0;
      double y = t > 1 ? (double)t : 1.0;
      if (y < x) y = x;
      mu[cl] = log(x);
      const double sigma = (log(y) - mu[cl]) / kZ99;
      spread[cl] = sigma > 0.0;
      den[cl] = sigma * kSqrt2;
      const double isg = spread[cl] ? 1.0 / sigma : 0.0;
      sx0[cl] = fma((lnlo - mu[cl]) * isg, (double)kPhiSteps, kPhiZ * (double)kPhiSteps);
      dsx[cl] = du * isg * (double)kPhiSteps;
      wt[cl] = (double)a.cnt[c * kMaxC + cl] / (double)tot;
    }
    const int64_t rs = row_stride(a);
    uint16_t* out = ws_block(a, sk) + r;
    for (int gb = 0; gb < a.G; gb += 64) {
      const int gn = a.G - gb < 64 ? a.G - gb : 64;
      uint64_t unsure = 0;
      // the mixture at grid point g: two points per step, so that the two
      // dependent chains of table evaluations overlap
      auto mix = [&](double gd) -> double {
        const double u = lnlo + gd * du;
        double F = 0.0;
#pragma unroll
        for (int cl = 0; cl < kMaxC; ++cl) {
          if ((uint32_t)cl >= nc) break;
          double ph;
          if (!spread[cl]) {
            ph = u >= mu[cl] ? 1.0 : 0.0;
          } else {
            const double sx = fma(gd, dsx[cl], sx0[cl]);
            if (sx <= 0.0) {
              ph = 0.0;
            } else if (sx >= (double)kPhiN) {
              ph = 1.0;
            } else {
              // fused multiply-adds: their rounding differs from separate
              // operations by far less than the band below allows for
              int i = (int)sx;
              i = i < kPhiN - 1 ? i : kPhiN - 1;
              const double t = sx - (double)i;
              const double* cf = tab + 4 * i;
              ph = fma(t, fma(t, fma(t, cf[3], cf[2]), cf[1]), cf[0]);
            }
          }
          F = fma(wt[cl], ph, F);
        }
        return F;
      };
      // quant16(v - kBand) == quant16(v + kBand), decided from one floor:
      // both ends below 1 (q = 0), both at or above 65535, or one integer part
      auto emit = [&](int gi, double F) {
        const double v = F * 65536.0, vlo = v - kBand, vhi = v + kBand;
        const double fh = floor(vhi);
        if (vhi < 1.0 || vlo >= fh || vlo >= 65535.0)
          out[(int64_t)(gb + gi) * rs] = (uint16_t)(vhi < 1.0 ? 0u : (fh >= 65535.0 ? 65535u : (uint32_t)fh));
        else
          unsure |= 1ull << gi;
      };
      int gi = 0;
      for (; gi + 1 < gn; gi += 2) {
        const double F0 = mix((double)(gb + gi)), F1 = mix((double)(gb + gi + 1));
        emit(gi, F0);
        emit(gi + 1, F1);
      }
      if (gi < gn) emit(gi, mix((double)(gb + gi)));
      // grid points near a quantisation step: the defining erfc form
      while (unsure) {
        const int gi = __builtin_ctzll(unsure);
        unsure &= unsure - 1;
        const double u = lnlo + (double)(gb + gi) * du;
        double F = 0.0;
#pragma unroll
        for (int cl = 0; cl < kMaxC; ++cl) {
          if ((uint32_t)cl >= nc) break;
          const double phi = spread[cl] ? 0.5 * erfc((mu[cl] - u) / den[cl]) : (u >= mu[cl] ? 1.0 : 0.0);
          F += wt[cl] * phi;
        }
        out[(int64_t)(gb + gi) * rs] = (uint16_t)quant16(F * 65536.0);
      }
    }
  }
}

// ------------------------------------------------------------------ score
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t t = __shfl_up(v, o, 64);
    if (lane >= o) v += t;
  }
  return v;
}

// Claims for slots j0 .. j0 + B - 1 of every lane (qt[j] holds the value;
// bit j of pm: slot j active): the 16-bit counter of bin v (two counters per
// word) counts one per active lane, and each lane gets the counter's value
// before its own claim, so lanes with equal v get distinct consecutive
// values. Per slot one atomic instruction, in which the first active lane
// adds for every lane sharing its value (at the ends of the grid most ranks
// share the value 0 or 65535) and the lanes with other values add one each;
// every slot's atomic is issued before any result is waited for. On return
// qt[j] = value | claim << 16. Must be reached by every lane of the
// wavefront.
template <int VS, int B>
__device__ __forceinline__ void claim_bins(uint32_t* fine, uint32_t (&qt)[VS], uint32_t pm, int j0) {
  const int lane = threadIdx.x & 63;
  const unsigned long long below = (1ull << lane) - 1ull;
  uint32_t old[B];
  int leader[B];
#pragma unroll
  for (int i = 0; i < B; ++i) {
    const int j = j0 + i;
    const uint32_t v = qt[j] & 0xFFFFu;
    const bool active = ((pm >> j) & 1u) != 0;
    const unsigned long long act = __ballot(active);
    leader[i] = act ? __ffsll((long long)act) - 1 : 0;
    const uint32_t lv = __builtin_amdgcn_readlane(v, leader[i]);
    const bool mine = active && v == lv;
    const unsigned long long same = __ballot(mine);
    const bool lead = mine && lane == leader[i];
    const uint32_t add = (lead ? (uint32_t)__popcll(same) : 1u) << ((v & 1u) * 16u);
    old[i] = 0;
    if (active && (lead || !mine)) old[i] = atomicAdd(&fine[v >> 1], add);
    // lanes sharing the leader's value: their place among those lanes
    qt[j] = v | ((mine ? 0x8000u | (uint32_t)__popcll(same & below) : 0u) << 16);
  }
#pragma unroll
  for (int i = 0; i < B; ++i) {
    const int j = j0 + i;
    const uint32_t v = qt[j] & 0xFFFFu, sh = (v & 1u) * 16u;
    const uint32_t lo = __builtin_amdgcn_readlane(old[i], leader[i]);
    const uint32_t c = (qt[j] >> 31) ? ((lo >> sh) & 0xFFFFu) + ((qt[j] >> 16) & 0x7FFFu) : (old[i] >> sh) & 0xFFFFu;
    qt[j] = v | (c << 16);
  }
}

// Rank of slot j of thread tid: slots come in pairs of neighbouring ranks,
// 2 (tid + m NT) and 2 (tid + m NT) + 1 for pair m, whose two 16-bit values
// are one aligned 32-bit word of a workspace row.
template <int NT>
__device__ __forceinline__ int slot_rank(int tid, int j) {
  return 2 * (tid + (j >> 1) * NT) + (j & 1);
}

template <int NT, int V>
__global__ __launch_bounds__(NT) void w1_score(W1Args a) {
  constexpr int NW = NT / 64;
  constexpr int V2 = (V + 1) / 2;  // slot pairs per thread
  constexpr int VS = 2 * V2;       // slots per thread
  __shared__ uint32_t fine[kFineWords];  // bin counters, then the sorted values and their prefix sums
  __shared__ double wts[ARGUS_MAX_W1_GRID];  // trapezoid weights
  __shared__ uint32_t bcnt[256], bexcl[256];
  __shared__ uint32_t wtot[NW];
  __shared__ SelShared<2> sel;
  __shared__ unsigned long long mn_sh, mx_sh;
  __shared__ uint32_t nf_sh;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t sk = xcd_item(blockIdx.x, gridDim.x);
  const int s = (int)(sk / a.K), k = (int)(sk % a.K);
  const uint32_t n = a.o.n_present[sk];
  // scores and flags go to the workspace, contiguous per (step, kernel);
  // w1_out moves them to the cell layout
  const int64_t rs = row_stride(a);
  double* ws_score = ws_scores(a, sk);
  uint8_t* ws_flag = ws_flags(a, sk);

  if (!evaluated(a, n)) {
#pragma unroll
    for (int j = 0; j < VS; ++j) {
      const int r = slot_rank<NT>(tid, j);
      if (r >= a.R) break;
      ws_score[r] = 0.0;
      ws_flag[r] = 0;
    }
    if (tid == 0) {
      a.o.lo_ns[sk] = 0;
      a.o.hi_ns[sk] = 0;
      a.o.q1[sk] = a.o.q3[sk] = a.o.fence[sk] = 0.0;
      a.o.n_flag[sk] = 0;
    }
    return;
  }

  uint32_t pm = 0;  // bit j: slot j is present
#pragma unroll
  for (int j = 0; j < VS; ++j) {
    const int r = slot_rank<NT>(tid, j);
    if (r >= a.R) break;
    uint32_t nc;
    uint64_t tot;
    if (cell_state(a, cell_of(a, r, s, k), nc, tot) > 0) pm |= 1u << j;
  }
  double lnlo, du;
  grid_of(a, sk, lnlo, du);
  const int G = a.G;
  // this kernel's rows as a buffer: the word of pair m in row g is at byte
  // 2 rs g + 4 (tid + m NT); words of pairs past the ranks are never used,
  // and those past the last row read 0 (buffer range check)
  const __amdgpu_buffer_rsrc_t qbuf =
      __builtin_amdgcn_make_buffer_rsrc(ws_block(a, sk), (short)0, (int)(2 * rs * G), 0x00020000);
  auto pair_word = [&](int g, int m) -> uint32_t {
    return __builtin_amdgcn_raw_buffer_load_b32(qbuf, (int)(2u * (uint32_t)rs * (uint32_t)g + 4u * (uint32_t)(tid + m * NT)), 0, 0);
  };
  // w_g = (x_{min(g+1,G-1)} - x_{max(g-1,0)}) / 2, x_i = exp(lnlo + i du)
  for (int g = tid; g < G; g += NT)
    wts[g] = (exp(lnlo + (double)(g + 1 < G ? g + 1 : G - 1) * du) - exp(lnlo + (double)(g > 0 ? g - 1 : 0) * du)) /
             2.0;

  // per slot: acc = weighted sum; qt = q | (rank among equal values) << 16;
  // cl2 / qn2: values below q / the next grid point's q, 16 bits each, two
  // slots to a word (keeps the 16-slot variant in registers). A slot that is
  // not present may hold any value; every use is masked by present().
  double acc[VS];
  uint32_t qt[VS], cl2[V2], qn2[V2];
  auto present = [&](int j) { return ((pm >> j) & 1u) != 0; };
#pragma unroll
  for (int m = 0; m < V2; ++m) {
    const uint32_t w = pair_word(0, m);
    qt[2 * m] = w & 0xFFFFu;
    qt[2 * m + 1] = w >> 16;
    acc[2 * m] = acc[2 * m + 1] = 0.0;
    cl2[m] = qn2[m] = 0;
  }
  if (tid < 256) bcnt[tid] = 0;
  if (tid == 0) {
    mn_sh = ~0ull;
    mx_sh = 0;
    nf_sh = 0;
  }
  __syncthreads();

  const int E = ((int)n + NT - 1) / NT;  // sorted values per thread in the prefix sum
  for (int g = 0; g < G; ++g) {
    // 1. bucket (high byte) counts
#pragma unroll
    for (int j = 0; j < VS; ++j) hist_add<1>(bcnt, (qt[j] & 0xFFFFu) >> 8, present(j));
    lds_barrier();
    // 2. bucket scan, first half; clear the bins of the occupied buckets
    uint32_t bc = 0, binc = 0;
    if (tid < 256) {
      bc = bcnt[tid];
      binc = wave_incl_scan(bc);
      if (lane == 63) wtot[wv] = binc;
    }
    // (16-bin chunks tid + i NT, 32 to a bucket: their buckets' counts are
    // read together, then the chunks of occupied buckets cleared one by one;
    // unrolled, the stores' addresses would stay live across the loop over
    // grid points and push other values out of registers)
    constexpr int kChunks = kFineWords / 4 / NT;
    static_assert(kChunks <= 32, "chunk mask");
    uint32_t occ = 0;
#pragma unroll
    for (int i = 0; i < kChunks; ++i) occ |= (bcnt[(tid + i * NT) >> 5] != 0 ? 1u : 0u) << i;
#pragma unroll 1
    for (int i = 0; i < kChunks; ++i)
      if ((occ >> i) & 1u) *reinterpret_cast<uint4*>(&fine[(tid + i * NT) * 4]) = make_uint4(0, 0, 0, 0);
    lds_barrier();
    // 3. bucket exclusive prefix; per-value claims (rank among equal values)
    if (tid < 256) {
      uint32_t base = 0;
      for (int w = 0; w < wv; ++w) base += wtot[w];
      bexcl[tid] = base + binc - bc;
    }
    claim_bins<VS, VS>(fine, qt, pm, 0);
    lds_barrier();
    // the next point's words, one load per pair with no arithmetic on the
    // result: the loads stay in flight until step 8 (the barriers of the
    // steps in between order LDS only). Issued here, after the last reload
    // of spilled registers before step 8 (loads complete in order, so a
    // reload waits for every load issued before it).
    if (g + 1 < G) {
#pragma unroll
      for (int m = 0; m < V2; ++m) qn2[m] = pair_word(g + 1, m);
      // keeps the compiler from sinking the loads to their use
      __asm__ volatile("" ::: "memory");
    }
    // 4. exclusive prefix over the 256 bins of each occupied bucket
    // (buckets wv + NW i of this wavefront: one count per lane, then the
    // occupied ones only)
    constexpr int kWaveBuckets = 256 / NW;
    static_assert(kWaveBuckets <= 64, "one bucket per lane");
    const uint64_t occb = __ballot(lane < kWaveBuckets && bcnt[lane < kWaveBuckets ? wv + NW * lane : 0] != 0);
    for (uint64_t mb = occb; mb; mb &= mb - 1) {
      const int h = wv + NW * (int)__builtin_ctzll(mb);
      uint2* p = reinterpret_cast<uint2*>(&fine[h * 128 + 2 * lane]);
      const uint2 wd = *p;
      const uint32_t b0 = wd.x & 0xFFFFu, b1 = wd.x >> 16, b2 = wd.y & 0xFFFFu, b3 = wd.y >> 16;
      const uint32_t t = b0 + b1 + b2 + b3;
      const uint32_t e0 = wave_incl_scan(t) - t, e1 = e0 + b0, e2 = e1 + b1, e3 = e2 + b2;
      *p = make_uint2(e0 | (e1 << 16), e2 | (e3 << 16));
    }
    lds_barrier();
    // 5. values below q: bucket prefix + bin prefix
#pragma unroll
    for (int j = 0; j < VS; ++j) {
      const uint32_t v = qt[j] & 0xFFFFu;
      const uint32_t clt = present(j) ? bexcl[v >> 8] + ((fine[v >> 1] >> ((v & 1u) * 16u)) & 0xFFFFu) : 0u;
      cl2[j >> 1] = (j & 1) ? (cl2[j >> 1] & 0xFFFFu) | (clt << 16) : (cl2[j >> 1] & 0xFFFF0000u) | clt;
    }
    lds_barrier();
    // 6. counting-sort scatter to position (values below) + (rank among
    //    equal values); clear the bucket counts for the next point
#pragma unroll
    for (int j = 0; j < VS; ++j)
      if (present(j)) fine[((cl2[j >> 1] >> ((j & 1) * 16)) & 0xFFFFu) + (qt[j] >> 16)] = qt[j] & 0xFFFFu;
    if (tid < 256) bcnt[tid] = 0;
    lds_barrier();
    // 7. exclusive prefix sums of the sorted values, in place
    const int i0 = tid * E, i1 = i0 + E < (int)n ? i0 + E : (int)n;
    uint32_t loc = 0;
    for (int i = i0; i < i1; ++i) loc += fine[i];
    const uint32_t linc = wave_incl_scan(loc);
    if (lane == 63) wtot[wv] = linc;
    lds_barrier();
    uint32_t run = linc - loc, T = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const uint32_t x = wtot[w];
      if (w < wv) run += x;
      T += x;
    }
    for (int i = i0; i < i1; ++i) {
      const uint32_t x = fine[i];
      fine[i] = run;
      run += x;
    }
    lds_barrier();
    // 8. S_a = q (2 c - n) + T - 2 P, weighted by the trapezoid rule
    const double wg = wts[g];
#pragma unroll
    for (int j = 0; j < VS; ++j) {
      if (present(j)) {
        // S <= (n - 1) 65535 < 2^32: the sum is exact modulo 2^32
        const uint32_t clt = (cl2[j >> 1] >> ((j & 1) * 16)) & 0xFFFFu;
        const uint32_t S = (qt[j] & 0xFFFFu) * (2u * clt - n) + T - 2u * fine[clt];
        acc[j] += wg * (double)S;
      }
      qt[j] = (qn2[j >> 1] >> ((j & 1) * 16)) & 0xFFFFu;
    }
  }

  // deviation scores; quartiles by radix selection on their bit patterns
  // (the scores are kept only as their bits, offset by the minimum)
  const double norm = 65536.0 * (double)(n - 1);
  uint64_t key[VS];
  unsigned long long mn = ~0ull, mx = 0;
#pragma unroll
  for (int j = 0; j < VS; ++j) {
    key[j] = (uint64_t)__double_as_longlong(acc[j] / norm);
    if (present(j)) {
      mn = key[j] < mn ? key[j] : mn;
      mx = key[j] > mx ? key[j] : mx;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long x = __shfl_xor(mn, o, 64), y = __shfl_xor(mx, o, 64);
    mn = x < mn ? x : mn;
    mx = y > mx ? y : mx;
  }
  if (lane == 0) {
    atomicMin(&mn_sh, mn);
    atomicMax(&mx_sh, mx);
  }
  __syncthreads();
  const uint64_t kmin = mn_sh, kmax = mx_sh;
#pragma unroll
  for (int j = 0; j < VS; ++j) key[j] = present(j) ? key[j] - kmin : 0;
  const uint32_t nm1 = n - 1;
  const uint32_t ranks[2] = {nm1 / 4, (uint32_t)((3ull * nm1) / 4)};
  uint64_t qs[2];
  select_ranks<NT, VS, 2>(key, (uint64_t)pm, kmax - kmin, ranks, qs, sel);
  const double a1 = __longlong_as_double((long long)(kmin + qs[0]));
  const double a3 = __longlong_as_double((long long)(kmin + qs[1]));
  const double fence = a3 + (double)a.alpha_pm * (a3 - a1) / 1000.0;

  uint32_t nf = 0;
#pragma unroll
  for (int j = 0; j < VS; ++j) {
    const int r = slot_rank<NT>(tid, j);
    if (r >= a.R) break;
    const bool p = present(j);
    const double sc = __longlong_as_double((long long)(kmin + key[j]));
    const bool f = p && sc > fence;
    nf += f ? 1u : 0u;
    ws_score[r] = p ? sc : 0.0;
    ws_flag[r] = f ? 1 : 0;
  }
  for (int o = 32; o > 0; o >>= 1) nf += __shfl_xor(nf, o, 64);
  if (lane == 0 && nf) atomicAdd(&nf_sh, nf);
  // orders the LDS count only: the score and flag stores are not waited for,
  // so the workgroup ends (and the next one starts) while they drain
  lds_barrier();
  if (tid == 0) {
    a.o.lo_ns[sk] = a.o.lo_ns[sk] < 1 ? 1 : a.o.lo_ns[sk];
    a.o.q1[sk] = a1;
    a.o.q3[sk] = a3;
    a.o.fence[sk] = fence;
    a.o.n_flag[sk] = nf_sh;
  }
}

// ------------------------------------------------------------------ out
// The scores and flags of the workspace blocks ([step, kernel][rank]) into
// the [rank][step][kernel] outputs, through 64 x 64 LDS tiles so that both
// the reads and the writes are contiguous.
__global__ __launch_bounds__(256) void w1_out(W1Args a) {
  __shared__ double ts[64][65];
  __shared__ uint8_t tf[64][68];
  const int64_t SK = (int64_t)a.S * a.K, sk0 = (int64_t)blockIdx.x * 64;
  const int r0 = blockIdx.y * 64, t = threadIdx.x;
  for (int i = t; i < 64 * 64; i += 256) {
    const int row = i >> 6, col = i & 63;  // row: (step, kernel), col: rank
    const int64_t sk = sk0 + row;
    const int r = r0 + col;
    double v = 0.0;
    uint8_t f = 0;
    if (sk < SK && r < a.R) {
      v = ws_scores(a, sk)[r];
      f = ws_flags(a, sk)[r];
    }
    ts[row][col] = v;
    tf[row][col] = f;
  }
  __syncthreads();
  for (int i = t; i < 64 * 64; i += 256) {
    const int row = i >> 6, col = i & 63;  // row: rank, col: (step, kernel)
    const int r = r0 + row;
    const int64_t sk = sk0 + col;
    if (sk < SK && r < a.R) {
      const int64_t c = (int64_t)r * SK + sk;  // cell (r, s, k)
      a.o.score[c] = ts[col][row];
      a.o.flag[c] = tf[col][row];
    }
  }
}

template <int NT, int V>
void launch_score(const W1Args& wa, hipStream_t st) {
  hipLaunchKernelGGL((w1_score<NT, V>), dim3((unsigned)((int64_t)wa.S * wa.K)), dim3(NT), 0, st, wa);
}

// Fill g_phi_tab on the current device once.
hipError_t ensure_phi_table() {
  static std::mutex mu;
  static bool done[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (done[dev]) return hipSuccess;
  std::vector<double> tab(kPhiN * 4);
  const double h = 1.0 / kPhiSteps, inv_sqrt_2pi = 0.39894228040143267794;
  auto Phi = [](double z) { return 0.5 * std::erfc(-z / kSqrt2); };
  auto dphi = [&](double z) { return h * inv_sqrt_2pi * std::exp(-0.5 * z * z); };  // d Phi / d t
  for (int i = 0; i < kPhiN; ++i) {
    const double z0 = -kPhiZ + (double)i * h, z1 = -kPhiZ + (double)(i + 1) * h;
    const double y0 = Phi(z0), y1 = Phi(z1), m0 = dphi(z0), m1 = dphi(z1);
    tab[4 * i] = y0;
    tab[4 * i + 1] = m0;
    tab[4 * i + 2] = 3.0 * (y1 - y0) - 2.0 * m0 - m1;
    tab[4 * i + 3] = 2.0 * (y0 - y1) + m0 + m1;
  }
  e = hipMemcpyToSymbol(HIP_SYMBOL(g_phi_tab), tab.data(), sizeof(double) * tab.size());
  if (e == hipSuccess) done[dev] = true;
  return e;
}

}  // namespace

size_t w1_workspace_bytes(int32_t R, int32_t S, int32_t K, int32_t G) {
  if (R < 0 || S < 0 || K < 0 || G < 0) return 0;
  return (size_t)ws_q_bytes(R, S, K, G) + (size_t)S * (size_t)K * (size_t)ws_row_stride(R) * 9;
}

hipError_t launch_w1(const W1Launch& l, hipStream_t st) {
  W1Args wa{l.n_clusters, l.count, l.p50, l.p99, l.R, l.S, l.K, l.p.grid, l.p.min_ranks, l.p.alpha_pm, l.o,
            static_cast<uint16_t*>(l.workspace)};
  const int64_t SK = (int64_t)l.S * l.K;
  hipError_t e = ensure_phi_table();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(w1_init, dim3((unsigned)((SK + 255) / 256)), dim3(256), 0, st, wa);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(w1_bounds, dim3((l.K + 63) / 64, (l.R + 63) / 64, l.S), dim3(256), 0, st, wa);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(w1_cdf, dim3((l.K + 4 * kCdfKPerWave - 1) / (4 * kCdfKPerWave), (l.R + 63) / 64, l.S), dim3(256),
                     0, st, wa);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  // register-resident slots per thread: R <= 1024 with 256 threads, else 1024 threads
  const int R = l.R;
  if (R <= 256) launch_score<256, 1>(wa, st);
  else if (R <= 512) launch_score<256, 2>(wa, st);
  else if (R <= 1024) launch_score<256, 4>(wa, st);
  else if (R <= 2048) launch_score<1024, 2>(wa, st);
  else if (R <= 4096) launch_score<1024, 4>(wa, st);
  else if (R <= 8192) launch_score<1024, 8>(wa, st);
  else if (R <= 10240) launch_score<1024, 10>(wa, st);
  else if (R <= 12288) launch_score<1024, 12>(wa, st);
  else launch_score<1024, 16>(wa, st);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(w1_out, dim3((unsigned)((SK + 63) / 64), (unsigned)((l.R + 63) / 64)), dim3(256), 0, st, wa);
  return hipGetLastError();
}

}  // namespace argus
