// Kernel-level cross-rank analysis (paper section 6.2; Eq. 4; the z-score
// of Appendix B).
//
// Each rank's summary of a kernel is reduced to its exact integer mean x;
// the same kernel is then compared across ranks with robust order
// statistics (lower median, lower nearest-rank quartiles, MAD). With point
// summaries the paper's mean Wasserstein-1 distance of a rank to its peers
// is the mean |x_r - x_b|, and its outlier-robust, median-centred form
// |x_r - med| is what the MAD scales. The IQR upper fence of Eq. 4 is kept
// as a second flag bit.
//
// Three launches per call:
//   1. transpose: [R][S][K] (count, sum) -> x in a [S][K][R] workspace,
//      64x64 tiles through LDS so both the read and the write are coalesced;
//   2. per (step, kernel): one workgroup of 256-1024 threads holds the
//      kernel's x of every rank in registers (up to 24 per thread) and runs
//      an MSD radix select over x - min, 11-bit digits, for q1, median and
//      q3 together, then once more on |x - median| for the MAD; exact
//      128-bit sum for the mean;
//   3. per (rank, step): per-cell z, mean and flags, a radix select of the
//      rank's typical per-kernel ratio to the median, the straggler decision
//      and the degraded-pair bit.
// Digit histograms live in LDS; lanes of a wavefront that hit the same bin
// are counted by one atomic (values of one kernel cluster tightly around
// the median, so most lanes share a bin in the leading digits).

#include "argus_internal.h"
#include "argus_select.h"

namespace argus {
namespace {

typedef unsigned __int128 u128;
typedef __int128 i128;

// Radix-select digit widths: a kernel's means span about 2^22 ns, which 11-bit
// digits resolve in two passes (8-bit digits: three); a rank's permille
// ratios span a few thousand (two 8-bit passes; a 4,096-bin single pass
// costs more to clear and scan than it saves).
constexpr int kStatsDigit = 11;
constexpr int kRankDigit = 8;
// One aggregation round per histogram add: it takes the dominant bin of the
// leading digit; a second round costs more than the conflicts it saves.
constexpr int kAggRounds = 1;

// floor(sum / count) with sum read as uint64, saturated at INT64_MAX. Below
// 2^53 both operands are exact doubles and the correctly rounded quotient
// truncates to the exact floor or one above it (never below: the floor is
// representable), which one exact product detects; larger sums take the
// integer division.
__device__ __forceinline__ int64_t cell_x(uint32_t count, int64_t sum) {
  const uint64_t s = (uint64_t)sum;
  uint64_t x;
  if (s < (1ull << 53)) {
    x = (uint64_t)((double)s / (double)count);
    if (x * count > s) --x;
  } else {
    x = s / count;
  }
  return x > (uint64_t)INT64_MAX ? INT64_MAX : (int64_t)x;
}

// ---------------------------------------------------------------- transpose
__global__ __launch_bounds__(256) void xr_transpose(const uint32_t* __restrict__ count,
                                                    const int64_t* __restrict__ sum, int32_t R, int32_t S,
                                                    int32_t K, int64_t* __restrict__ xT) {
  __shared__ int64_t tile[64][65];
  const int k0 = blockIdx.x * 64, r0 = blockIdx.y * 64, s = blockIdx.z;
  const int t = threadIdx.x, c64 = t & 63;
  // all 32 loads of a thread are issued before the first is used (the sum
  // is read whether or not the count is zero)
  uint32_t n[16];
  int64_t sm[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int r = r0 + (t >> 6) + 4 * i, k = k0 + c64;
    n[i] = 0;
    sm[i] = 0;
    if (r < R && k < K) {
      const int64_t c = ((int64_t)r * S + s) * K + k;
      n[i] = count[c];
      sm[i] = sum[c];
    }
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) tile[(t >> 6) + 4 * i][c64] = n[i] ? cell_x(n[i], sm[i]) : -1;
  __syncthreads();
  for (int kk = t >> 6; kk < 64; kk += 4) {
    const int k = k0 + kk, r = r0 + c64;
    if (r < R && k < K) xT[((int64_t)s * K + k) * R + r] = tile[c64][kk];
  }
}

// ------------------------------------------------------ per (step, kernel)
struct StatsArgs {
  const int64_t* xT;
  int32_t R, S, K, min_ranks;
  uint32_t* n_present;
  int64_t *med, *mad, *q1, *q3;
  float* xmean;
  uint32_t *n_flag, *n_degraded;
};

template <int NT, int V>
__global__ __launch_bounds__(NT) void xr_kernel_stats(StatsArgs a) {
  __shared__ SelShared<3, kStatsDigit> sh3;
  __shared__ SelShared<1, kStatsDigit> sh1;
  __shared__ uint32_t n_sh;
  __shared__ unsigned long long red_min, red_max, red_lo, red_hi;
  const int tid = threadIdx.x;
  const int64_t sk = blockIdx.x;
  const int64_t* row = a.xT + sk * a.R;
  if (tid == 0) {
    n_sh = 0;
    red_min = ~0ull;
    red_max = 0;
    red_lo = 0;
    red_hi = 0;
  }
  uint64_t key[V];
  uint64_t vm = 0;
  uint32_t cnt = 0;
  unsigned long long mn = ~0ull, mx = 0;
  u128 acc = 0;
#pragma unroll
  for (int j = 0; j < V; ++j) {
    const int r = tid + j * NT;
    const int64_t x = r < a.R ? row[r] : -1;
    key[j] = x >= 0 ? (uint64_t)x : 0;
    if (x >= 0) {
      vm |= 1ull << j;
      ++cnt;
      mn = (uint64_t)x < mn ? (uint64_t)x : mn;
      mx = (uint64_t)x > mx ? (uint64_t)x : mx;
      acc += (uint64_t)x;
    }
  }
  __syncthreads();
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long mo = __shfl_xor(mn, o, 64), xo = __shfl_xor(mx, o, 64);
    mn = mo < mn ? mo : mn;
    mx = xo > mx ? xo : mx;
    cnt += __shfl_xor(cnt, o, 64);
  }
  if ((tid & 63) == 0) {
    atomicMin(&red_min, mn);
    atomicMax(&red_max, mx);
    atomicAdd(&n_sh, cnt);
  }
  // exact 128-bit sum of x: low words added with explicit carry detection
  if (acc != 0) {
    const unsigned long long lo = (unsigned long long)acc, hi = (unsigned long long)(acc >> 64);
    const unsigned long long old = atomicAdd(&red_lo, lo);
    atomicAdd(&red_hi, hi + (old + lo < old ? 1ull : 0ull));
  }
  __syncthreads();
  const int n = (int)n_sh;
  if (tid == 0) {
    a.n_present[sk] = (uint32_t)n;
    a.n_flag[sk] = 0;
    a.n_degraded[sk] = 0;
  }
  if (n < a.min_ranks || n == 0) {
    if (tid == 0) {
      a.med[sk] = a.mad[sk] = a.q1[sk] = a.q3[sk] = -1;
      a.xmean[sk] = 0.0f;
    }
    return;
  }
  const uint64_t vmin = red_min, vmax = red_max;
#pragma unroll
  for (int j = 0; j < V; ++j) key[j] -= (vm >> j) & 1u ? vmin : 0;
  const uint32_t nm1 = (uint32_t)(n - 1);
  const uint32_t ranks[3] = {nm1 / 4, nm1 / 2, (uint32_t)((3ull * nm1) / 4)};
  uint64_t qs[3];
  select_ranks<NT, V, 3, kStatsDigit, kAggRounds>(key, vm, vmax - vmin, ranks, qs, sh3);
  const uint64_t dmed = qs[1];  // median - vmin
#pragma unroll
  for (int j = 0; j < V; ++j) key[j] = key[j] >= dmed ? key[j] - dmed : dmed - key[j];
  const uint64_t top = vmax - vmin - dmed;
  const uint32_t r1[1] = {nm1 / 2};
  uint64_t md[1];
  select_ranks<NT, V, 1, kStatsDigit, kAggRounds>(key, vm, top > dmed ? top : dmed, r1, md, sh1);
  if (tid == 0) {
    a.q1[sk] = (int64_t)(vmin + qs[0]);
    a.med[sk] = (int64_t)(vmin + qs[1]);
    a.q3[sk] = (int64_t)(vmin + qs[2]);
    a.mad[sk] = (int64_t)md[0];
    const u128 total = ((u128)red_hi << 64) | (u128)red_lo;
    a.xmean[sk] = (float)((double)total / (double)n);
  }
}

// --------------------------------------------------------- per (rank, step)
struct RankArgs {
  const uint32_t* count;
  const int64_t* sum;
  int32_t R, S, K;
  argus_xr_params_t p;
  argus_xr_out_t o;
};

// floor(1000 x / med), saturated at INT32_MAX (x >= 0, med >= 1). Below
// 2^53 the quotient comes from a correctly rounded double division and one
// product check, as in cell_x.
__device__ __forceinline__ uint32_t ratio_pm(int64_t x, int64_t med) {
  uint64_t q;
  if ((uint64_t)x < (1ull << 53) / 1000u && (uint64_t)med < (1ull << 53)) {
    const uint64_t num = (uint64_t)x * 1000u;
    q = (uint64_t)((double)num / (double)med);
    if (q * (uint64_t)med > num) --q;
  } else if ((uint64_t)x <= ~0ull / 1000u) {
    q = ((uint64_t)x * 1000u) / (uint64_t)med;
  } else {
    const u128 w = ((u128)(uint64_t)x * 1000u) / (u128)(uint64_t)med;
    q = w > (u128)INT32_MAX ? (uint64_t)INT32_MAX : (uint64_t)w;
  }
  return q > (uint64_t)INT32_MAX ? (uint32_t)INT32_MAX : (uint32_t)q;
}

template <int NT, int V>
__global__ __launch_bounds__(NT) void xr_rank(RankArgs a) {
  __shared__ SelShared<1, kRankDigit> sh;
  __shared__ uint32_t ne_sh, nf_sh, rmin_sh, rmax_sh;
  const int tid = threadIdx.x;
  const int32_t K = a.K;
  const int64_t rs = blockIdx.x;  // r * S + s
  const int32_t s = (int32_t)(rs % a.S);
  if (tid == 0) {
    ne_sh = 0;
    nf_sh = 0;
    rmin_sh = 0xFFFFFFFFu;
    rmax_sh = 0;
  }
  uint32_t rat[V];
  uint32_t fl[(V + 3) / 4];
#pragma unroll
  for (int j = 0; j < (V + 3) / 4; ++j) fl[j] = 0;
  uint64_t em = 0;
  uint32_t ne = 0, nf = 0, rmin = 0xFFFFFFFFu, rmax = 0;
  // cells in groups of four: every load of a group (the cells and their
  // kernels' statistics) is issued before the first is used
  constexpr int VB = V < 4 ? V : 4;
  static_assert(V % VB == 0, "cell groups");
#pragma unroll
  for (int jb = 0; jb < V; jb += VB) {
    uint32_t cnt_[VB], np_[VB];
    int64_t sm_[VB], med_[VB], mad_[VB], q1_[VB], q3_[VB];
#pragma unroll
    for (int u = 0; u < VB; ++u) {
      const int j = jb + u;
      const int k = tid + j * NT < K ? tid + j * NT : K - 1;
      const int64_t c = rs * K + k;
      const int64_t sk = (int64_t)s * K + k;
      cnt_[u] = a.count[c];
      sm_[u] = a.sum[c];
      np_[u] = a.o.n_present[sk];
      med_[u] = a.o.med_ns[sk];
      mad_[u] = a.o.mad_ns[sk];
      q1_[u] = a.o.q1_ns[sk];
      q3_[u] = a.o.q3_ns[sk];
    }
#pragma unroll
    for (int u = 0; u < VB; ++u) {
      const int j = jb + u;
      const int k = tid + j * NT;
      rat[j] = 0;
      if (k >= K) continue;
      const int64_t c = rs * K + k;
      const uint32_t cnt = cnt_[u];
      float z = 0.0f, mean = 0.0f;
      uint32_t f = 0;
      if (cnt) {
        const int64_t sm = sm_[u];
        mean = (float)((double)sm / (double)cnt);
        const uint32_t n = np_[u];
        if (n >= (uint32_t)a.p.min_ranks && n) {
          const int64_t x = cell_x(cnt, sm);
          const int64_t med = med_[u], mad = mad_[u];
          const int64_t q1 = q1_[u], q3 = q3_[u];
          const int64_t madf = mad > 1 ? mad : 1;
          const int64_t iqr = q3 - q1 > 1 ? q3 - q1 : 1;
          z = (float)((double)(x - med) / (1.4826 * (double)madf));
          f = 4;
          if (cnt >= (uint32_t)a.p.c_min_pair && (i128)1000 * ((i128)x - med) > (i128)a.p.k_mad_pm * madf &&
              (i128)1000 * x >= (i128)a.p.ratio_pm * med)
            f |= 1;
          if ((i128)1000 * ((i128)x - q3) > (i128)a.p.alpha_pm * iqr) f |= 2;
          if (med >= 1) {
            const uint32_t r = ratio_pm(x, med);
            rat[j] = r;
            em |= 1ull << j;
            ++ne;
            rmin = r < rmin ? r : rmin;
            rmax = r > rmax ? r : rmax;
            if (f & 1) ++nf;
          }
        }
      }
      a.o.z[c] = z;
      if (a.o.mean_ns) a.o.mean_ns[c] = mean;
      fl[j >> 2] |= f << (8 * (j & 3));
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    ne += __shfl_xor(ne, o, 64);
    nf += __shfl_xor(nf, o, 64);
    const uint32_t a1 = __shfl_xor(rmin, o, 64), a2 = __shfl_xor(rmax, o, 64);
    rmin = a1 < rmin ? a1 : rmin;
    rmax = a2 > rmax ? a2 : rmax;
  }
  __syncthreads();
  if ((tid & 63) == 0) {
    atomicAdd(&ne_sh, ne);
    atomicAdd(&nf_sh, nf);
    atomicMin(&rmin_sh, rmin);
    atomicMax(&rmax_sh, rmax);
  }
  __syncthreads();
  const int n_eval = (int)ne_sh;
  int32_t score = -1;
  if (n_eval > 0) {
    const uint32_t lo = rmin_sh;
#pragma unroll
    for (int j = 0; j < V; ++j) rat[j] -= (em >> j) & 1u ? lo : 0u;
    const uint32_t rk[1] = {(uint32_t)(n_eval - 1) / 2};
    uint64_t sel[1];
    select_ranks<NT, V, 1, kRankDigit, kAggRounds>(rat, em, rmax_sh - lo, rk, sel, sh);
    score = (int32_t)(lo + (uint32_t)sel[0]);
  }
  const bool strag = n_eval >= a.p.min_kernels && (int64_t)score >= 1000 + (int64_t)a.p.tau_rank_pm;
#pragma unroll
  for (int j = 0; j < V; ++j) {
    const int k = tid + j * NT;
    if (k >= K) continue;
    uint32_t f = (fl[j >> 2] >> (8 * (j & 3))) & 0xFFu;
    if (f & 1) {
      const int64_t sk = (int64_t)s * K + k;
      atomicAdd(&a.o.n_flag[sk], 1u);
      if (!strag) {
        f |= 8;
        atomicAdd(&a.o.n_degraded[sk], 1u);
      }
    }
    a.o.flags[rs * K + k] = (uint8_t)f;
  }
  if (tid == 0) {
    a.o.score_pm[rs] = score;
    a.o.n_eval[rs] = (uint32_t)n_eval;
    a.o.n_flag_rank[rs] = nf_sh;
    a.o.straggler[rs] = strag ? 1 : 0;
  }
}

template <int NT, int V>
void launch_stats(const StatsArgs& sa, dim3 g, hipStream_t st) {
  hipLaunchKernelGGL((xr_kernel_stats<NT, V>), g, dim3(NT), 0, st, sa);
}

template <int NT, int V>
void launch_rank(const RankArgs& ra, dim3 g, hipStream_t st) {
  hipLaunchKernelGGL((xr_rank<NT, V>), g, dim3(NT), 0, st, ra);
}

}  // namespace

hipError_t launch_cross_rank(const CrossRankLaunch& l, hipStream_t st) {
  const int32_t R = l.R, S = l.S, K = l.K;
  hipLaunchKernelGGL(xr_transpose, dim3((K + 63) / 64, (R + 63) / 64, S), dim3(256), 0, st, l.count, l.sum_ns, R,
                     S, K, l.xT);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  StatsArgs sa{l.xT, R, S, K, l.p.min_ranks, l.o.n_present, l.o.med_ns, l.o.mad_ns, l.o.q1_ns, l.o.q3_ns,
               l.o.xmean_ns, l.o.n_flag, l.o.n_degraded};
  const dim3 g2((unsigned)((int64_t)S * K));
  dispatch_block(R, [&](auto nt, auto v) { launch_stats<decltype(nt)::value, decltype(v)::value>(sa, g2, st); });
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  RankArgs ra{l.count, l.sum_ns, R, S, K, l.p, l.o};
  const dim3 g3((unsigned)((int64_t)R * S));
  dispatch_block(K, [&](auto nt, auto v) { launch_rank<decltype(nt)::value, decltype(v)::value>(ra, g3, st); });
  return hipGetLastError();
}

}  // namespace argus
