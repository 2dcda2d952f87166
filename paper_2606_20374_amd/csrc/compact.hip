// The uploaded summary stream: dense per-(rank, step, key) summaries ->
// little-endian records of the present cells (section 5.2: only compact
// statistics leave the host; section 8.3 compares their size with the raw
// trace). The record layout is defined in include/argus.h.
//
// Launches, in order:
//   compact_sizes   one workgroup per segment: the byte size of its records
//                   (33 + 5 per nonzero octave bin for every present cell).
//   compact_scan    one workgroup: exclusive prefix of the sizes in segment
//                   order -> seg_byte_off (deterministic placement).
//   compact_write   one workgroup per segment: 256 cells at a time, each
//                   thread builds its cell's record in an LDS staging area at
//                   the offset a block scan assigns, then the workgroup copies
//                   the staged bytes to their final position with aligned
//                   4-byte stores (byte stores only at the two unaligned
//                   ends). A record is written only if it lies entirely
//                   inside the caller's buffer.
#include "argus_internal.h"

namespace argus {
namespace {

constexpr int kThreads = 256;
constexpr int kRecMax = 33 + 5 * NB;  // largest record: every octave bin nonzero

struct CompactArgs {
  const uint32_t* count;
  const int64_t* sum;
  const int64_t* mn;
  const int64_t* mx;
  const uint32_t* hist;
  int32_t n_seg, n_cells, n_streams;
  uint8_t* out;
  int64_t cap;
  int64_t* seg_off;
  int32_t* dev_status;
  int64_t* sizes;
};

// nonzero-bin mask of one cell's octave histogram (16-byte loads)
__device__ __forceinline__ uint32_t bin_mask(const uint32_t* h) {
  uint32_t m = 0;
  const uint4* h4 = reinterpret_cast<const uint4*>(h);
#pragma unroll
  for (int q = 0; q < NB / 4; ++q) {
    const uint4 v = h4[q];
    m |= (v.x != 0 ? 1u : 0u) << (4 * q);
    m |= (v.y != 0 ? 1u : 0u) << (4 * q + 1);
    m |= (v.z != 0 ? 1u : 0u) << (4 * q + 2);
    m |= (v.w != 0 ? 1u : 0u) << (4 * q + 3);
  }
  return m;
}

__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* wtot, uint32_t& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t t = __shfl_up(inc, o, 64);
    if (lane >= o) inc += t;
  }
  if (lane == 63) wtot[w] = inc;
  __syncthreads();
  uint32_t base = 0;
  total = 0;
#pragma unroll
  for (int i = 0; i < kThreads / 64; ++i) {
    const uint32_t x = wtot[i];
    if (i < w) base += x;
    total += x;
  }
  __syncthreads();
  return base + inc - v;
}

// ------------------------------------------------------------------- sizes
__global__ __launch_bounds__(kThreads) void compact_sizes(CompactArgs a) {
  __shared__ unsigned long long tot;
  const int64_t g = blockIdx.x;
  if (threadIdx.x == 0) tot = 0;
  __syncthreads();
  unsigned long long s = 0;
  for (int c = threadIdx.x; c < a.n_cells; c += kThreads) {
    const int64_t i = g * a.n_cells + c;
    if (a.count[i] == 0) continue;
    s += 33u + 5u * (uint32_t)__popc(bin_mask(a.hist + i * NB));
  }
  s = wave_sum_u64(s);
  if ((threadIdx.x & 63) == 0) atomicAdd(&tot, s);
  __syncthreads();
  if (threadIdx.x == 0) a.sizes[g] = (int64_t)tot;
}

// -------------------------------------------------------------------- scan
__global__ __launch_bounds__(1024) void compact_scan(CompactArgs a) {
  __shared__ unsigned long long wtot[16];
  __shared__ unsigned long long carry;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  if (tid == 0) carry = 0;
  __syncthreads();
  for (int64_t b = 0; b < a.n_seg; b += 1024) {
    const int64_t g = b + tid;
    const unsigned long long v = g < a.n_seg ? (unsigned long long)a.sizes[g] : 0ull;
    unsigned long long inc = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const unsigned long long t = __shfl_up(inc, o, 64);
      if (lane >= o) inc += t;
    }
    if (lane == 63) wtot[w] = inc;
    __syncthreads();
    unsigned long long base = carry, total = 0;
    for (int i = 0; i < 16; ++i) {
      if (i < w) base += wtot[i];
      total += wtot[i];
    }
    if (g < a.n_seg) a.seg_off[g] = (int64_t)(base + inc - v);
    __syncthreads();
    if (tid == 0) carry += total;
    __syncthreads();
  }
  if (tid == 0) {
    a.seg_off[a.n_seg] = (int64_t)carry;
    if ((int64_t)carry > a.cap && a.dev_status) atomicOr(a.dev_status, (int32_t)ARGUS_DEV_COMPACT_CAPACITY);
  }
}

// ------------------------------------------------------------------- write
__device__ __forceinline__ void put(uint8_t* p, uint64_t v, int n) {
  for (int i = 0; i < n; ++i) p[i] = (uint8_t)(v >> (8 * i));
}

__global__ __launch_bounds__(kThreads) void compact_write(CompactArgs a) {
  __shared__ uint8_t stage[kThreads * kRecMax + 16];
  __shared__ uint32_t wtot[kThreads / 64];
  __shared__ uint32_t fit_end;
  const int64_t g = blockIdx.x;
  const int tid = threadIdx.x;
  int64_t pos = a.seg_off[g];  // global byte position of the next chunk
  if (pos >= a.cap) return;
  for (int c0 = 0; c0 < a.n_cells; c0 += kThreads) {
    const int c = c0 + tid;
    const int64_t i = g * a.n_cells + c;
    const bool present = c < a.n_cells && a.count[i] != 0;
    const uint32_t m = present ? bin_mask(a.hist + i * NB) : 0u;
    const uint32_t len = present ? 33u + 5u * (uint32_t)__popc(m) : 0u;
    uint32_t chunk = 0;
    const uint32_t at = block_excl_scan(len, wtot, chunk);
    if (chunk == 0) continue;
    if (tid == 0) fit_end = 0;
    __syncthreads();
    if (present) {
      uint8_t* p = stage + at;
      const uint32_t key = a.n_streams > 0 ? (uint32_t)(c / a.n_streams) | ((uint32_t)(c % a.n_streams) << 24)
                                           : (uint32_t)c;
      put(p, key, 4);
      put(p + 4, a.count[i], 4);
      put(p + 8, (uint64_t)a.sum[i], 8);
      put(p + 16, (uint64_t)a.mn[i], 8);
      put(p + 24, (uint64_t)a.mx[i], 8);
      p[32] = (uint8_t)__popc(m);
      int q = 33;
      const uint32_t* h = a.hist + i * NB;
      for (uint32_t mm = m; mm; mm &= mm - 1) {
        const int b = __ffs(mm) - 1;
        p[q] = (uint8_t)b;
        put(p + q + 1, h[b], 4);
        q += 5;
      }
      // records are written only when they lie entirely inside the buffer
      if (pos + at + len <= a.cap) atomicMax(&fit_end, at + len);
    }
    __syncthreads();
    // copy stage[0, fit_end) to out[pos, pos + fit_end)
    const int64_t lo = pos, hi = pos + fit_end;
    const int64_t wlo = (lo + 3) & ~(int64_t)3, whi = hi & ~(int64_t)3;
    if (wlo < whi) {
      for (int64_t wd = wlo + 4 * tid; wd < whi; wd += 4 * kThreads) {
        const uint8_t* s = stage + (wd - lo);
        const uint32_t v = (uint32_t)s[0] | ((uint32_t)s[1] << 8) | ((uint32_t)s[2] << 16) | ((uint32_t)s[3] << 24);
        *reinterpret_cast<uint32_t*>(a.out + wd) = v;
      }
      if (tid < wlo - lo) a.out[lo + tid] = stage[tid];
      if (tid < hi - whi) a.out[whi + tid] = stage[whi - lo + tid];
    } else {
      for (int64_t b = lo + tid; b < hi; b += kThreads) a.out[b] = stage[b - lo];
    }
    pos += chunk;
    __syncthreads();
    if (pos >= a.cap) return;
  }
}

}  // namespace

hipError_t launch_compact(const CompactLaunch& l, hipStream_t st) {
  CompactArgs a{l.count, l.sum_ns, l.min_ns, l.max_ns, l.hist, l.n_seg, l.n_cells, l.n_streams, l.out, l.capacity,
                l.seg_byte_off, l.dev_status, l.sizes};
  if (l.n_seg > 0) {
    hipLaunchKernelGGL(compact_sizes, dim3(l.n_seg), dim3(kThreads), 0, st, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(compact_scan, dim3(1), dim3(1024), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || l.n_seg == 0 || l.capacity == 0) return e;
  hipLaunchKernelGGL(compact_write, dim3(l.n_seg), dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace argus
