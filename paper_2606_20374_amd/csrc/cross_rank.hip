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
//   2. per (step, kernel): load the kernel's row of x into LDS, then an
//      MSD radix select (8-bit digits over x - min) for q1, median, q3 and,
//      on |x - median|, the MAD; exact 128-bit sum for the mean;
//   3. per (rank, step): per-cell z, mean and flags, then a radix select of
//      the rank's typical per-kernel ratio to the median, the straggler
//      decision, and the degraded-pair bit on the rank's outlier cells.
#include "argus_internal.h"

namespace argus {
namespace {

typedef unsigned __int128 u128;
typedef __int128 i128;

constexpr int kSelThreads = 256;

// Inclusive scan of one value per thread over a 256-thread block.
__device__ __forceinline__ uint32_t block_scan_256(uint32_t v, uint32_t* wave_tot) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t n = __shfl_up(v, o, 64);
    if (lane >= o) v += n;
  }
  if (lane == 63) wave_tot[wave] = v;
  __syncthreads();
  uint32_t add = 0;
  for (int w = 0; w < wave; ++w) add += wave_tot[w];
  __syncthreads();
  return v + add;
}

struct SelShared {
  uint32_t hist[256];
  uint32_t wave_tot[4];
  uint32_t digit, before;
};

// k-th smallest (0-based) of keys[0..n), all keys <= range. Block-wide; all
// threads of the 256-thread block must call it.
template <typename KeyT>
__device__ uint64_t block_select(const KeyT* keys, int n, uint32_t k, uint64_t range, SelShared& sh) {
  if (range == 0) return 0;
  const int nbits = 64 - __builtin_clzll(range);
  const int passes = (nbits + 7) >> 3;
  uint64_t prefix = 0;
  for (int p = passes - 1; p >= 0; --p) {
    const int shift = p * 8;
    sh.hist[threadIdx.x] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += kSelThreads) {
      const uint64_t key = keys[i];
      if (p == passes - 1 || (key >> (shift + 8)) == prefix) atomicAdd(&sh.hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    const uint32_t h = sh.hist[threadIdx.x];
    const uint32_t incl = block_scan_256(h, sh.wave_tot);
    const uint32_t excl = incl - h;
    if (excl <= k && k < incl) {
      sh.digit = threadIdx.x;
      sh.before = excl;
    }
    __syncthreads();
    prefix = (prefix << 8) | sh.digit;
    k -= sh.before;
    __syncthreads();
  }
  return prefix;
}

__device__ __forceinline__ int64_t cell_x(uint32_t count, int64_t sum) {
  const uint64_t x = (uint64_t)sum / count;
  return x > (uint64_t)INT64_MAX ? INT64_MAX : (int64_t)x;
}

// ---------------------------------------------------------------- transpose
__global__ __launch_bounds__(256) void xr_transpose(const uint32_t* __restrict__ count,
                                                    const int64_t* __restrict__ sum, int32_t R, int32_t S,
                                                    int32_t K, int64_t* __restrict__ xT) {
  __shared__ int64_t tile[64][65];
  const int k0 = blockIdx.x * 64, r0 = blockIdx.y * 64, s = blockIdx.z;
  const int t = threadIdx.x, c64 = t & 63;
  for (int rr = t >> 6; rr < 64; rr += 4) {
    const int r = r0 + rr, k = k0 + c64;
    int64_t x = -1;
    if (r < R && k < K) {
      const int64_t c = ((int64_t)r * S + s) * K + k;
      const uint32_t n = count[c];
      if (n) x = cell_x(n, sum[c]);
    }
    tile[rr][c64] = x;
  }
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

template <int RCAP>
__global__ __launch_bounds__(kSelThreads) void xr_kernel_stats(StatsArgs a) {
  __shared__ uint64_t vals[RCAP];
  __shared__ SelShared sh;
  __shared__ uint32_t n_sh;
  __shared__ unsigned long long red_min, red_max, red_lo, red_hi;
  const int64_t sk = blockIdx.x;
  const int64_t* row = a.xT + sk * a.R;
  if (threadIdx.x == 0) {
    n_sh = 0;
    red_min = ~0ull;
    red_max = 0;
    red_lo = 0;
    red_hi = 0;
  }
  __syncthreads();
  unsigned long long mn = ~0ull, mx = 0;
  u128 acc = 0;
  for (int r = threadIdx.x; r < a.R; r += kSelThreads) {
    const int64_t x = row[r];
    if (x >= 0) {
      const uint32_t i = atomicAdd(&n_sh, 1u);
      vals[i] = (uint64_t)x;
      mn = (uint64_t)x < mn ? (uint64_t)x : mn;
      mx = (uint64_t)x > mx ? (uint64_t)x : mx;
      acc += (uint64_t)x;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const unsigned long long mo = __shfl_xor(mn, o, 64), xo = __shfl_xor(mx, o, 64);
    mn = mo < mn ? mo : mn;
    mx = xo > mx ? xo : mx;
  }
  if ((threadIdx.x & 63) == 0) {
    atomicMin(&red_min, mn);
    atomicMax(&red_max, mx);
  }
  // exact 128-bit sum of x: low words added with explicit carry detection
  if (acc != 0) {
    const unsigned long long lo = (unsigned long long)acc, hi = (unsigned long long)(acc >> 64);
    const unsigned long long old = atomicAdd(&red_lo, lo);
    atomicAdd(&red_hi, hi + (old + lo < old ? 1ull : 0ull));
  }
  __syncthreads();
  const int n = (int)n_sh;
  if (threadIdx.x == 0) {
    a.n_present[sk] = (uint32_t)n;
    a.n_flag[sk] = 0;
    a.n_degraded[sk] = 0;
  }
  if (n < a.min_ranks || n == 0) {
    if (threadIdx.x == 0) {
      a.med[sk] = a.mad[sk] = a.q1[sk] = a.q3[sk] = -1;
      a.xmean[sk] = 0.0f;
    }
    return;
  }
  const uint64_t vmin = red_min, vmax = red_max;
  for (int i = threadIdx.x; i < n; i += kSelThreads) vals[i] -= vmin;
  __syncthreads();
  const uint64_t range = vmax - vmin;
  const uint32_t nm1 = (uint32_t)(n - 1);
  const int64_t q1 = (int64_t)(vmin + block_select(vals, n, nm1 / 4, range, sh));
  const int64_t med = (int64_t)(vmin + block_select(vals, n, nm1 / 2, range, sh));
  const int64_t q3 = (int64_t)(vmin + block_select(vals, n, (uint32_t)((3ull * nm1) / 4), range, sh));
  // absolute deviations from the median, in place
  const uint64_t dmed = (uint64_t)med - vmin;
  for (int i = threadIdx.x; i < n; i += kSelThreads) {
    const uint64_t v = vals[i];
    vals[i] = v >= dmed ? v - dmed : dmed - v;
  }
  __syncthreads();
  const uint64_t drange = (vmax - (uint64_t)med) > dmed ? (vmax - (uint64_t)med) : dmed;
  const int64_t mad = (int64_t)block_select(vals, n, nm1 / 2, drange, sh);
  if (threadIdx.x == 0) {
    a.med[sk] = med;
    a.mad[sk] = mad;
    a.q1[sk] = q1;
    a.q3[sk] = q3;
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

template <int KCAP>
__global__ __launch_bounds__(kSelThreads) void xr_rank(RankArgs a) {
  __shared__ uint32_t rat[KCAP];
  __shared__ uint8_t fl[KCAP];
  __shared__ SelShared sh;
  __shared__ uint32_t ne_sh, nf_sh, rmin_sh, rmax_sh;
  const int32_t K = a.K;
  const int64_t rs = blockIdx.x;  // r * S + s
  const int32_t s = (int32_t)(rs % a.S);
  if (threadIdx.x == 0) {
    ne_sh = 0;
    nf_sh = 0;
    rmin_sh = 0xFFFFFFFFu;
    rmax_sh = 0;
  }
  __syncthreads();
  uint32_t nf = 0;
  for (int k = threadIdx.x; k < K; k += kSelThreads) {
    const int64_t c = rs * K + k;
    const int64_t sk = (int64_t)s * K + k;
    const uint32_t cnt = a.count[c];
    float z = 0.0f, mean = 0.0f;
    uint8_t f = 0;
    if (cnt) {
      const int64_t sm = a.sum[c];
      mean = (float)((double)sm / (double)cnt);
      const uint32_t n = a.o.n_present[sk];
      if (n >= (uint32_t)a.p.min_ranks && n) {
        const int64_t x = cell_x(cnt, sm);
        const int64_t med = a.o.med_ns[sk], mad = a.o.mad_ns[sk];
        const int64_t q1 = a.o.q1_ns[sk], q3 = a.o.q3_ns[sk];
        const int64_t madf = mad > 1 ? mad : 1;
        const int64_t iqr = q3 - q1 > 1 ? q3 - q1 : 1;
        z = (float)((double)(x - med) / (1.4826 * (double)madf));
        f = 4;
        if (cnt >= (uint32_t)a.p.c_min_pair && (i128)1000 * ((i128)x - med) > (i128)a.p.k_mad_pm * madf &&
            (i128)1000 * x >= (i128)a.p.ratio_pm * med)
          f |= 1;
        if ((i128)1000 * ((i128)x - q3) > (i128)a.p.alpha_pm * iqr) f |= 2;
        if (med >= 1) {
          uint64_t q;
          if ((uint64_t)x <= ~0ull / 1000u)
            q = ((uint64_t)x * 1000u) / (uint64_t)med;
          else
            q = (uint64_t)(((u128)(uint64_t)x * 1000u) / (u128)(uint64_t)med > (u128)INT32_MAX
                               ? (u128)INT32_MAX
                               : ((u128)(uint64_t)x * 1000u) / (u128)(uint64_t)med);
          const uint32_t ratio = q > (uint64_t)INT32_MAX ? (uint32_t)INT32_MAX : (uint32_t)q;
          const uint32_t i = atomicAdd(&ne_sh, 1u);
          rat[i] = ratio;
          atomicMin(&rmin_sh, ratio);
          atomicMax(&rmax_sh, ratio);
          if (f & 1) nf++;
        }
      }
    }
    a.o.z[c] = z;
    if (a.o.mean_ns) a.o.mean_ns[c] = mean;
    fl[k] = f;
  }
  atomicAdd(&nf_sh, nf);
  __syncthreads();
  const int ne = (int)ne_sh;
  int32_t score = -1;
  if (ne > 0) {
    const uint32_t rmin = rmin_sh;
    for (int i = threadIdx.x; i < ne; i += kSelThreads) rat[i] -= rmin;
    __syncthreads();
    score = (int32_t)(rmin + block_select(rat, ne, (uint32_t)(ne - 1) / 2, rmax_sh - rmin, sh));
  }
  const bool strag = ne >= a.p.min_kernels && (int64_t)score >= 1000 + (int64_t)a.p.tau_rank_pm;
  for (int k = threadIdx.x; k < K; k += kSelThreads) {
    uint8_t f = fl[k];
    if (f & 1) {
      const int64_t sk = (int64_t)s * K + k;
      atomicAdd(&a.o.n_flag[sk], 1u);
      if (!strag) {
        f |= 8;
        atomicAdd(&a.o.n_degraded[sk], 1u);
      }
    }
    a.o.flags[rs * K + k] = f;
  }
  if (threadIdx.x == 0) {
    a.o.score_pm[rs] = score;
    a.o.n_eval[rs] = (uint32_t)ne;
    a.o.n_flag_rank[rs] = nf_sh;
    a.o.straggler[rs] = strag ? 1 : 0;
  }
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
  if (R <= 2048)
    hipLaunchKernelGGL(xr_kernel_stats<2048>, g2, dim3(kSelThreads), 0, st, sa);
  else
    hipLaunchKernelGGL(xr_kernel_stats<ARGUS_MAX_XR_RANKS>, g2, dim3(kSelThreads), 0, st, sa);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  RankArgs ra{l.count, l.sum_ns, R, S, K, l.p, l.o};
  const dim3 g3((unsigned)((int64_t)R * S));
  if (K <= 2048)
    hipLaunchKernelGGL(xr_rank<2048>, g3, dim3(kSelThreads), 0, st, ra);
  else
    hipLaunchKernelGGL(xr_rank<ARGUS_MAX_XR_KERNELS>, g3, dim3(kSelThreads), 0, st, ra);
  return hipGetLastError();
}

}  // namespace argus
