// Parallelism-group-aware L2 comparison (section 6.1 routing table; Appendix
// B, Eq. 5; the step-by-step definition is in include/argus.h).
//
// Launches, in order:
//   l2_init     default outputs: every cell z = 0, flags = 0; every (step,
//               event, group) not evaluated; ownership keys cleared.
//   l2_owner    one workgroup per (dimension, group): each listing (g, i) of
//               a rank m takes part in ownership by an atomic minimum of
//               g R + i, so the rank's first listing (lowest group, then
//               lowest position) is the one that counts; a second listing
//               or a malformed range raises a status bit.
//   l2_stats    one wavefront per (step, dimension, group, 64 consecutive
//               event ids): the lanes are the events, the loop runs over the
//               group's members, so each member's 64 cells are read (and its
//               z / flags written) contiguously. Lanes whose event is routed
//               to another dimension idle. Per lane the exact sums n, S = sum
//               x, Q = sum x^2 (128-bit) give D = n Q - S^2; the CV class and
//               the z threshold are decided by exact 256-bit comparisons, the
//               reported mean / std / CV / z are one double operation each.
#include "argus_internal.h"

namespace argus {
namespace {

typedef unsigned __int128 u128;

constexpr uint64_t kDomain = 1ull << 40;  // x at or above 2^40 ns is out of the domain
constexpr uint8_t kNotEvaluated = 0xFF;

struct L2Args {
  const uint32_t* count;
  const int64_t* sum;
  int32_t R, S, E;
  const uint8_t* route;
  const int32_t* off;  // [n_dims][max_groups + 1]
  const int32_t* mem;  // [n_dims][R]
  int32_t n_dims, max_groups;
  argus_l2_params_t p;
  argus_l2_out_t o;
  uint32_t* owner;  // workspace [n_dims][R]: first listing key g R + i
};

struct U256 {
  u128 hi, lo;
};

// Full 128 x 128 -> 256-bit product.
__device__ __forceinline__ U256 mul_wide(u128 a, u128 b) {
  const uint64_t a0 = (uint64_t)a, a1 = (uint64_t)(a >> 64), b0 = (uint64_t)b, b1 = (uint64_t)(b >> 64);
  const u128 p00 = (u128)a0 * b0, p01 = (u128)a0 * b1, p10 = (u128)a1 * b0, p11 = (u128)a1 * b1;
  const u128 mid = (p00 >> 64) + (uint64_t)p01 + (uint64_t)p10;
  return U256{p11 + (p01 >> 64) + (p10 >> 64) + (mid >> 64), (mid << 64) | (uint64_t)p00};
}

__device__ __forceinline__ bool less(const U256& a, const U256& b) {
  return a.hi < b.hi || (a.hi == b.hi && a.lo < b.lo);
}

__device__ __forceinline__ void raise(int32_t* st, int32_t bit) {
  if (st) atomicOr(st, bit);
}

// ------------------------------------------------------------------- init
__global__ __launch_bounds__(256) void l2_init(L2Args a, int64_t cells, int64_t gout, int64_t owners) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < cells; i += stride) {
    a.o.z[i] = 0.0f;
    a.o.flags[i] = 0;
  }
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < gout; i += stride) {
    a.o.n[i] = 0;
    a.o.mean_ns[i] = a.o.std_ns[i] = a.o.cv[i] = 0.0;
    a.o.cls[i] = kNotEvaluated;
    a.o.n_strag[i] = 0;
  }
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < owners; i += stride) a.owner[i] = 0xFFFFFFFFu;
}

// ------------------------------------------------------------- membership
__global__ __launch_bounds__(256) void l2_owner(L2Args a) {
  const int g = blockIdx.x, d = blockIdx.y;
  const int32_t* off = a.off + (int64_t)d * (a.max_groups + 1);
  const int32_t lo = off[g], hi = off[g + 1];
  if (lo < 0 || hi < lo || hi > a.R) {
    if (threadIdx.x == 0) raise(a.o.dev_status, ARGUS_DEV_GROUPS_MALFORMED);
    return;
  }
  bool bad = false, dup = false;
  for (int32_t i = lo + (int32_t)threadIdx.x; i < hi; i += 256) {
    const int32_t m = a.mem[(int64_t)d * a.R + i];
    if (m < 0 || m >= a.R) {
      bad = true;
      continue;
    }
    const uint32_t old = atomicMin(&a.owner[(int64_t)d * a.R + m], (uint32_t)g * (uint32_t)a.R + (uint32_t)i);
    if (old != 0xFFFFFFFFu) dup = true;
  }
  if (__ballot(bad) != 0 && (threadIdx.x & 63) == 0) raise(a.o.dev_status, ARGUS_DEV_GROUPS_MALFORMED);
  if (__ballot(dup) != 0 && (threadIdx.x & 63) == 0) raise(a.o.dev_status, ARGUS_DEV_GROUPS_DUPLICATE);
}

// ----------------------------------------------------------------- stats
// x of a present, in-domain cell, else -1 (out of domain raises *dom).
__device__ __forceinline__ int64_t cell_mean(const L2Args& a, int64_t c, bool& dom) {
  const uint32_t n = a.count[c];
  if (n == 0) return -1;
  const uint64_t x = (uint64_t)a.sum[c] / n;
  if (x >= kDomain) {
    dom = true;
    return -1;
  }
  return (int64_t)x;
}

__global__ __launch_bounds__(64) void l2_stats(L2Args a) {
  const int lane = threadIdx.x;
  const int e = blockIdx.x * 64 + lane, g = blockIdx.y;
  const int s = (int)(blockIdx.z / a.n_dims), d = (int)(blockIdx.z % a.n_dims);
  const bool mine = e < a.E && a.route[e] == d;
  if (__ballot(mine) == 0) return;
  const int32_t* off = a.off + (int64_t)d * (a.max_groups + 1);
  const int32_t lo = off[g], hi = off[g + 1];
  if (lo < 0 || hi <= lo || hi > a.R) return;
  const int32_t* mem = a.mem + (int64_t)d * a.R;
  const uint32_t* own = a.owner + (int64_t)d * a.R;
  const uint32_t key0 = (uint32_t)g * (uint32_t)a.R;

  // pass 1: exact sums over the present members
  uint32_t n = 0;
  uint64_t S1 = 0;
  u128 Q = 0;
  bool dom = false;
  for (int32_t i = lo; i < hi; ++i) {
    const int32_t m = mem[i];
    if (m < 0 || m >= a.R || own[m] != key0 + (uint32_t)i) continue;
    if (!mine) continue;
    const int64_t x = cell_mean(a, ((int64_t)m * a.S + s) * a.E + e, dom);
    if (x < 0) continue;
    ++n;
    S1 += (uint64_t)x;
    Q += (u128)(uint64_t)x * (uint64_t)x;
  }
  if (__ballot(dom) != 0 && lane == 0) raise(a.o.dev_status, ARGUS_DEV_L2_DOMAIN);
  if (!mine) return;
  const int64_t go = ((int64_t)s * a.E + e) * a.max_groups + g;
  a.o.n[go] = n;
  if ((int32_t)n < a.p.min_group || n < 2) return;

  const u128 S = S1, D = (u128)n * Q - S * S;
  const double mean = (double)S1 / (double)n;
  const double var = u128_to_f64(D) / ((double)n * (double)(n - 1));
  const double sd = sqrt(var);
  a.o.mean_ns[go] = mean;
  a.o.std_ns[go] = sd;
  a.o.cv[go] = mean > 0.0 ? sd / mean : 0.0;
  uint8_t cls = 0;
  if (S > 0) {
    const U256 lhs = mul_wide((u128)n * 1000000u, D);
    const u128 S2 = S * S;
    const U256 mild = mul_wide((u128)(uint32_t)a.p.cv_mild_pm * (uint32_t)a.p.cv_mild_pm * (n - 1), S2);
    const U256 sev = mul_wide((u128)(uint32_t)a.p.cv_severe_pm * (uint32_t)a.p.cv_severe_pm * (n - 1), S2);
    if (!less(lhs, mild)) cls = less(lhs, sev) ? 1 : 2;
  }
  a.o.cls[go] = cls;

  // pass 2: z-scores and the straggler test z > z_pm / 1000
  const U256 rhs = mul_wide((u128)(uint32_t)a.p.z_pm * (uint32_t)a.p.z_pm * n, D);
  uint32_t ns = 0;
  for (int32_t i = lo; i < hi; ++i) {
    const int32_t m = mem[i];
    if (m < 0 || m >= a.R || own[m] != key0 + (uint32_t)i) continue;
    const int64_t c = ((int64_t)m * a.S + s) * a.E + e;
    bool unused = false;
    const int64_t x = cell_mean(a, c, unused);
    if (x < 0) continue;
    uint8_t f = 1;
    const u128 nx = (u128)n * (uint64_t)x;
    if (nx > S) {
      const u128 dev = nx - S;
      if (less(rhs, mul_wide(dev * dev, (u128)(n - 1) * 1000000u))) {
        f |= 2;
        ++ns;
      }
    }
    a.o.z[c] = sd > 0.0 ? (float)(((double)x - mean) / sd) : 0.0f;
    a.o.flags[c] = f;
  }
  a.o.n_strag[go] = ns;
}

}  // namespace

size_t l2_workspace_bytes(int32_t R, int32_t n_dims) {
  if (R < 0 || n_dims < 0) return 0;
  return (size_t)R * (size_t)n_dims * sizeof(uint32_t);
}

hipError_t launch_l2(const L2Launch& l, hipStream_t st) {
  L2Args a{l.count, l.sum_ns, l.R, l.S, l.E, l.g.route, l.g.group_off, l.g.members, l.g.n_dims, l.g.max_groups,
           l.p, l.o, static_cast<uint32_t*>(l.workspace)};
  const int64_t cells = (int64_t)l.R * l.S * l.E, gout = (int64_t)l.S * l.E * l.g.max_groups;
  const int64_t owners = (int64_t)l.g.n_dims * l.R;
  int64_t mx = cells > gout ? cells : gout;
  mx = mx > owners ? mx : owners;
  const int64_t blocks = (mx + 255) / 256;
  hipLaunchKernelGGL(l2_init, dim3((unsigned)(blocks < 65536 ? blocks : 65536)), dim3(256), 0, st, a, cells, gout,
                     owners);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(l2_owner, dim3(l.g.max_groups, l.g.n_dims), dim3(256), 0, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(l2_stats, dim3((l.E + 63) / 64, l.g.max_groups, (unsigned)((int64_t)l.S * l.g.n_dims)), dim3(64),
                     0, st, a);
  return hipGetLastError();
}

}  // namespace argus
