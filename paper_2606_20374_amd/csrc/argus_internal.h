// Internal helpers shared by the libargus kernels and host wrapper.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/argus.h"

namespace argus {

constexpr int NB = ARGUS_NBINS;

// Octave bin of a duration: 0 for d < 2, else floor(log2 d) saturated at 31.
__device__ __forceinline__ int octave_bin(uint64_t d) {
  if (d < 2) return 0;
  int b = 63 - __builtin_clzll(d);
  return b < NB - 1 ? b : NB - 1;
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

template <typename T>
__device__ __forceinline__ T lds_load(T* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

template <typename T>
__device__ __forceinline__ void lds_store(T* p, T v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Workgroup barrier that orders LDS only. __syncthreads() also releases
// global memory at workgroup scope, which on gfx950 waits for every vector
// memory operation of the wave (loads and stores share one counter),
// including prefetched loads still in flight. Where threads of a workgroup
// exchange data only through LDS, this barrier keeps those loads (and
// stores) in flight across it.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Work item of workgroup b of a grid of n, numbered so that the workgroups
// of one XCD take consecutive items. Workgroups are dispatched to the eight
// XCDs in turn (b mod 8), each XCD with its own L2; items whose outputs or
// inputs share cache lines (neighbouring kernel ids of one cell row) then
// meet in one L2 instead of eight. A bijection on [0, n).
__device__ __forceinline__ int64_t xcd_item(int64_t b, int64_t n) {
  constexpr int64_t kXcd = 8;
  const int64_t x = b % kXcd, i = b / kXcd, q = n / kXcd, r = n % kXcd;
  return (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + i;
}

// 64-lane wavefront reductions (gfx950 runs wave64 only).
__device__ __forceinline__ unsigned long long wave_sum_u64(unsigned long long v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ long long wave_min_i64(long long v) {
  for (int o = 32; o > 0; o >>= 1) {
    long long w = __shfl_xor(v, o, 64);
    v = w < v ? w : v;
  }
  return v;
}
__device__ __forceinline__ long long wave_max_i64(long long v) {
  for (int o = 32; o > 0; o >>= 1) {
    long long w = __shfl_xor(v, o, 64);
    v = w > v ? w : v;
  }
  return v;
}

// Launch-side entry points of each kernel file (host code).
struct SummarizeLaunch {
  const int32_t* kernel_id;
  const int32_t* stream;
  const int64_t* start_ns;
  const int64_t* end_ns;
  const int64_t* seg_off;
  int64_t n_events;
  int32_t n_seg, n_kernels, n_streams;
  int32_t keyed;  // cells keyed by (kernel id, stream): [n_seg][n_kernels][n_streams]
  uint32_t* count;
  int64_t* sum_ns;
  int64_t* min_ns;
  int64_t* max_ns;
  uint32_t* hist;
  uint32_t* n_valid;
  uint32_t* n_invalid;
  int64_t* t_first;
  int64_t* t_last;
  int64_t* step_ns;
  int64_t* busy_ns;
  int64_t* stream_busy_ns;
  int64_t* wire_bytes;
  int32_t* dev_status;
  uint32_t* queue;  // workspace word, zeroed by launch_clear before the kernel
};
hipError_t launch_summarize(const SummarizeLaunch& a, hipStream_t st);

struct CrossRankLaunch {
  const uint32_t* count;
  const int64_t* sum_ns;
  int32_t R, S, K;
  argus_xr_params_t p;
  argus_xr_out_t o;
  int64_t* xT;  // workspace [S][K][R]
};
hipError_t launch_cross_rank(const CrossRankLaunch& a, hipStream_t st);

struct IterWindowsLaunch {
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
hipError_t launch_iter_windows(const IterWindowsLaunch& a, hipStream_t st);

struct KdeLaunch {
  const int32_t* kernel_id;
  const int32_t* stream;
  const int64_t* start_ns;
  const int64_t* end_ns;
  const int64_t* seg_off;
  int64_t n_events;
  int32_t n_seg, n_kernels, n_streams;
  const uint32_t* count;
  const int64_t* min_ns;
  const int64_t* max_ns;
  const uint32_t* n_invalid;  // per segment, or null
  argus_kde_params_t p;
  argus_kde_out_t o;
  void* workspace;  // kde_workspace_bytes(n_events, n_seg, n_seg * n_kernels), 256-byte aligned
};
hipError_t launch_kde(const KdeLaunch& a, hipStream_t st);
size_t kde_workspace_bytes(int64_t n_events, int64_t n_seg, int64_t cells);

struct W1Launch {
  const uint8_t* n_clusters;
  const uint32_t* count;
  const int64_t* p50;
  const int64_t* p99;
  int32_t R, S, K;
  argus_w1_params_t p;
  argus_w1_out_t o;
  void* workspace;  // w1_workspace_bytes(R, S, K, grid)
};
hipError_t launch_w1(const W1Launch& a, hipStream_t st);
size_t w1_workspace_bytes(int32_t R, int32_t S, int32_t K, int32_t G);

struct L2Launch {
  const uint32_t* count;
  const int64_t* sum_ns;
  int32_t R, S, E;
  argus_groups_t g;
  argus_l2_params_t p;
  argus_l2_out_t o;
  void* workspace;  // l2_workspace_bytes(R, n_dims)
};
hipError_t launch_l2(const L2Launch& a, hipStream_t st);
size_t l2_workspace_bytes(int32_t R, int32_t n_dims);

struct CompactLaunch {
  const uint32_t* count;
  const int64_t* sum_ns;
  const int64_t* min_ns;
  const int64_t* max_ns;
  const uint32_t* hist;
  int32_t n_seg, n_cells, n_streams;
  uint8_t* out;
  int64_t capacity;
  int64_t* seg_byte_off;
  int32_t* dev_status;
  int64_t* sizes;  // workspace [n_seg]
};
hipError_t launch_compact(const CompactLaunch& a, hipStream_t st);

// Zero the optional device status word and the optional queue counter.
hipError_t launch_clear(int32_t* dev_status, uint32_t* queue, hipStream_t st);

constexpr size_t kSummarizeWorkspace = 256;

}  // namespace argus
