/*
 * Synthetic kernel-event trace generator: host fill, device fill and
 * per-segment checksums. Both fills evaluate the same per-event rule
 * (tg_event.h), so a trace filled on the device is byte-identical to the
 * one filled on the host. The checksums let large traces be compared
 * without copying them.
 *
 * This library is test and benchmark infrastructure shared by both sides of
 * the parity checks; it computes nothing of the summarization method.
 */
#include <hip/hip_runtime.h>

#include <stdint.h>
#include <thread>
#include <vector>

#include "tg_event.h"

extern "C" {

/* Per-segment checksum of one event: position dependent, all four fields. */
static __host__ __device__ inline uint64_t tg_mix_event(int64_t i, int32_t kid, int32_t stream, int64_t start,
                                                         int64_t end) {
  uint64_t a = tg_fmix64((uint64_t)start ^ ((uint64_t)i * TG_GOLDEN));
  uint64_t b = tg_fmix64((uint64_t)end + 0x632BE59BD9B4E019ull);
  uint64_t c = tg_fmix64(((uint64_t)(uint32_t)kid << 32) | (uint32_t)stream);
  return tg_fmix64(a ^ (b * 3u) ^ (c * 5u));
}

/* Fill segments [g_begin, g_end) on the host. Event of absolute index e is
 * written to out[e - out_base]. seg_off holds n_ranks*n_steps+1 offsets. */
int tg_fill_host(const tg_params_t* P, const tg_tables_t* Tb, const int64_t* seg_off, int32_t g_begin,
                 int32_t g_end, int64_t out_base, int32_t* kid, int32_t* stream, int64_t* start, int64_t* end,
                 int32_t n_threads) {
  if (!P || !Tb || !seg_off || !kid || !stream || !start || !end) return -1;
  if (g_begin < 0 || g_end < g_begin || g_end > P->n_ranks * P->n_steps) return -1;
  if (n_threads < 1) n_threads = 1;
  auto work = [&](int32_t t) {
    for (int32_t g = g_begin + t; g < g_end; g += n_threads) {
      int32_t r = g / P->n_steps, s = g % P->n_steps;
      int64_t b = seg_off[g], n = seg_off[g + 1] - seg_off[g];
      for (int64_t i = 0; i < n; ++i) {
        int64_t o = b + i - out_base;
        tg_event(P, Tb, r, s, i, &kid[o], &stream[o], &start[o], &end[o]);
      }
    }
  };
  if (n_threads == 1) {
    work(0);
  } else {
    std::vector<std::thread> th;
    for (int32_t t = 0; t < n_threads; ++t) th.emplace_back(work, t);
    for (auto& x : th) x.join();
  }
  return 0;
}

int tg_checksum_host(const tg_params_t* P, const int64_t* seg_off, int32_t g_begin, int32_t g_end, int64_t out_base,
                     const int32_t* kid, const int32_t* stream, const int64_t* start, const int64_t* end,
                     uint64_t* sums /* [g_end - g_begin] */) {
  if (!P || !seg_off || !sums) return -1;
  for (int32_t g = g_begin; g < g_end; ++g) {
    uint64_t h = 0;
    int64_t b = seg_off[g], n = seg_off[g + 1] - seg_off[g];
    for (int64_t i = 0; i < n; ++i) {
      int64_t o = b + i - out_base;
      h += tg_mix_event(i, kid[o], stream[o], start[o], end[o]);
    }
    sums[g - g_begin] = h;
  }
  return 0;
}

}  // extern "C"

/* One workgroup per segment, grid-stride over its events. */
__global__ __launch_bounds__(256) void tg_fill_kernel(tg_params_t P, tg_tables_t Tb, const int64_t* seg_off,
                                                      int32_t g_begin, int64_t out_base, int32_t* kid,
                                                      int32_t* stream, int64_t* start, int64_t* end) {
  const int32_t g = g_begin + (int32_t)blockIdx.x;
  const int32_t r = g / P.n_steps, s = g % P.n_steps;
  const int64_t b = seg_off[g], n = seg_off[g + 1] - seg_off[g];
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
    int64_t o = b + i - out_base;
    int32_t k, st;
    int64_t t0, t1;
    tg_event(&P, &Tb, r, s, i, &k, &st, &t0, &t1);
    kid[o] = k;
    stream[o] = st;
    start[o] = t0;
    end[o] = t1;
  }
}

__global__ __launch_bounds__(256) void tg_checksum_kernel(const int64_t* seg_off, int32_t g_begin, int64_t out_base,
                                                          const int32_t* kid, const int32_t* stream,
                                                          const int64_t* start, const int64_t* end,
                                                          unsigned long long* sums) {
  __shared__ unsigned long long acc;
  const int32_t g = g_begin + (int32_t)blockIdx.x;
  if (threadIdx.x == 0) acc = 0;
  __syncthreads();
  const int64_t b = seg_off[g], n = seg_off[g + 1] - seg_off[g];
  unsigned long long h = 0;
  for (int64_t i = threadIdx.x; i < n; i += blockDim.x) {
    int64_t o = b + i - out_base;
    h += tg_mix_event(i, kid[o], stream[o], start[o], end[o]);
  }
  atomicAdd(&acc, h);
  __syncthreads();
  if (threadIdx.x == 0) sums[blockIdx.x] = acc;
}

extern "C" {

/* Device fill: all pointers in P/Tb tables, seg_off and outputs are device
 * pointers; the caller checks that seg_off matches the output sizes. */
int tg_fill_device(const tg_params_t* P, const tg_tables_t* Tb, const int64_t* seg_off, int32_t g_begin,
                   int32_t g_end, int64_t out_base, int32_t* kid, int32_t* stream, int64_t* start, int64_t* end,
                   void* hip_stream) {
  if (!P || !Tb || g_end <= g_begin) return g_end == g_begin ? 0 : -1;
  hipLaunchKernelGGL(tg_fill_kernel, dim3(g_end - g_begin), dim3(256), 0, (hipStream_t)hip_stream, *P, *Tb,
                     seg_off, g_begin, out_base, kid, stream, start, end);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

int tg_checksum_device(const int64_t* seg_off, int32_t g_begin, int32_t g_end, int64_t out_base, const int32_t* kid,
                       const int32_t* stream, const int64_t* start, const int64_t* end, uint64_t* sums,
                       void* hip_stream) {
  if (g_end <= g_begin) return g_end == g_begin ? 0 : -1;
  hipLaunchKernelGGL(tg_checksum_kernel, dim3(g_end - g_begin), dim3(256), 0, (hipStream_t)hip_stream, seg_off,
                     g_begin, out_base, kid, stream, start, end, (unsigned long long*)sums);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

}  // extern "C"
