// Test probe (not part of libargus): evaluates the KDE's grid index and
// floating-point steps through the very functions the cell kernels call
// (kde_math.h) on given arguments, so a GPU test can compare them with the
// oracle's and the host C library's.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../paper_2606_20374_amd/csrc/kde_math.h"

namespace {

// One block per bandwidth H[i]: weights of t = 0 .. off[i+1]-off[i]-1.
__global__ void weights_kernel(const int64_t* H, const int64_t* off, int32_t nH, uint32_t* w) {
  const int i = blockIdx.x;
  if (i >= nH) return;
  const int64_t h = H[i], o = off[i], nt = off[i + 1] - off[i];
  const double H2 = (double)(h * h);
  for (int64_t t = threadIdx.x; t < nt; t += blockDim.x) w[o + t] = argus::kde_weight((int)t, H2);
}

__global__ void pow_kernel(const int64_t* n, int64_t m, double* out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < m) out[i] = argus::kde_pw((uint64_t)n[i]);
}

// H of (var, n): n^(-1/5) from pw_small (the table's values) below 65536
// durations, computed otherwise, as the cell kernels take it.
__global__ void bw_kernel(const double* var, const int64_t* n, const double* pw_small, int64_t m, int64_t* out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= m) return;
  const double pw = n[i] < 65536 ? pw_small[i] : argus::kde_pw((uint64_t)n[i]);
  out[i] = argus::kde_bw_q8(var[i], pw);
}

// Grid index of each duration, with the thresholds in LDS as the cell
// kernels hold them.
struct Thresholds {
  uint32_t th[64];
};

__global__ void grid_kernel(const uint64_t* d, int64_t m, Thresholds t, int32_t* out) {
  __shared__ uint32_t th[64];
  if (threadIdx.x < 64) th[threadIdx.x] = t.th[threadIdx.x];
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < m) out[i] = argus::kde_grid64(d[i], th);
}

// The 32-bit form the kernels use for 4-byte records (durations below 2^32).
__global__ void grid32_kernel(const uint32_t* d, int64_t m, Thresholds t, int32_t* out) {
  __shared__ uint32_t th[64];
  if (threadIdx.x < 64) th[threadIdx.x] = t.th[threadIdx.x];
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < m) out[i] = argus::kde_grid32(d[i], th);
}

int status(hipError_t e) { return e == hipSuccess ? 0 : -3; }

}  // namespace

extern "C" {

int probe_kde_weights(const int64_t* H, const int64_t* off, int32_t nH, uint32_t* w, void* stream) {
  if (nH <= 0) return 0;
  hipLaunchKernelGGL(weights_kernel, dim3(nH), dim3(256), 0, (hipStream_t)stream, H, off, nH, w);
  return status(hipGetLastError());
}

int probe_kde_root5(const int64_t* n, int64_t m, double* out, void* stream) {
  if (m <= 0) return 0;
  hipLaunchKernelGGL(pow_kernel, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, (hipStream_t)stream, n, m, out);
  return status(hipGetLastError());
}

int probe_kde_grid(const uint64_t* d, int64_t m, int32_t* out, void* stream) {
  if (m <= 0) return 0;
  Thresholds t;
  const uint32_t* th = argus::kde_thresholds();
  for (int i = 0; i < 64; ++i) t.th[i] = th[i];
  hipLaunchKernelGGL(grid_kernel, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, (hipStream_t)stream, d, m, t, out);
  return status(hipGetLastError());
}

int probe_kde_grid32(const uint32_t* d, int64_t m, int32_t* out, void* stream) {
  if (m <= 0) return 0;
  Thresholds t;
  const uint32_t* th = argus::kde_thresholds();
  for (int i = 0; i < 64; ++i) t.th[i] = th[i];
  hipLaunchKernelGGL(grid32_kernel, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, (hipStream_t)stream, d, m, t,
                     out);
  return status(hipGetLastError());
}

int probe_kde_bw_q8(const double* var, const int64_t* n, const double* pw_small, int64_t m, int64_t* out,
                    void* stream) {
  if (m <= 0) return 0;
  hipLaunchKernelGGL(bw_kernel, dim3((unsigned)((m + 255) / 256)), dim3(256), 0, (hipStream_t)stream, var, n,
                     pw_small, m, out);
  return status(hipGetLastError());
}

}  // extern "C"
