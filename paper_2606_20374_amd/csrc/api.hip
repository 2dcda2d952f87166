// C-ABI host wrapper of libargus: argument checks, workspace sizing and
// launches on the caller's stream. See include/argus.h for the contract.
#include <atomic>
#include <cstring>

#include "argus_internal.h"

namespace argus {
namespace {

__global__ void clear_kernel(int32_t* status, uint32_t* queue) {
  if (status) *status = 0;
  if (queue) *queue = 0;
}

// Per-device cache of "is gfx950": 0 unknown, 1 yes, 2 no.
std::atomic<int> g_arch_ok[64];

int check_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ARGUS_EHIP;
  if (dev < 0 || dev >= 64) return ARGUS_EUNSUPPORTED;
  int v = g_arch_ok[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, dev) != hipSuccess) return ARGUS_EHIP;
    v = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : 2;
    g_arch_ok[dev].store(v, std::memory_order_relaxed);
  }
  return v == 1 ? ARGUS_OK : ARGUS_EUNSUPPORTED;
}

int status_of(hipError_t e) { return e == hipSuccess ? ARGUS_OK : ARGUS_EHIP; }

// Scratch of argus_summarize_noalloc: the work-queue counter of the
// persistent summarize kernel, in device memory that the library never
// allocates. Each device holds its own copy until the process ends; in host
// code this name is only a handle, so kernels get the address that
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) uint8_t scratch[ARGUS_NOALLOC_SCRATCH_BYTES];

// Device address of `scratch` per device, looked up on the first call on
// that device (with it current).
std::atomic<void*> g_scratch_ptr[64];

int scratch_of_current_device(void** ptr) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return ARGUS_EHIP;
  if (dev < 0 || dev >= 64) return ARGUS_EUNSUPPORTED;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return ARGUS_EHIP;
    g_scratch_ptr[dev].store(p, std::memory_order_release);
  }
  *ptr = p;
  return ARGUS_OK;
}

}  // namespace

hipError_t launch_clear(int32_t* dev_status, uint32_t* queue, hipStream_t st) {
  if (!dev_status && !queue) return hipSuccess;
  hipLaunchKernelGGL(clear_kernel, dim3(1), dim3(1), 0, st, dev_status, queue);
  return hipGetLastError();
}

}  // namespace argus

using namespace argus;

extern "C" {

int argus_abi_version(void) { return ARGUS_ABI_VERSION; }

const char* argus_status_string(int status) {
  switch (status) {
    case ARGUS_OK: return "ok";
    case ARGUS_EINVAL: return "invalid argument";
    case ARGUS_EUNSUPPORTED: return "unsupported device (gfx950 required)";
    case ARGUS_EHIP: return "HIP launch failed";
    case ARGUS_EDEVICE: return "device-detected condition (see dev_status)";
    default: return "unknown status";
  }
}

size_t argus_summarize_workspace(const argus_events_t* ev) {
  (void)ev;
  return kSummarizeWorkspace;
}

static int summarize_impl(const argus_events_t* ev, const argus_summary_t* out, void* workspace, size_t workspace_bytes,
                   void* stream, bool keyed) {
  if (!ev || !out) return ARGUS_EINVAL;
  if (!workspace || workspace_bytes < kSummarizeWorkspace) return ARGUS_EINVAL;
  if ((reinterpret_cast<uintptr_t>(workspace) & 3u) != 0) return ARGUS_EINVAL;
  if (ev->n_ranks < 0 || ev->n_steps < 0 || ev->n_events < 0) return ARGUS_EINVAL;
  if (ev->n_kernels < 1 || ev->n_kernels > ARGUS_MAX_KERNELS) return ARGUS_EINVAL;
  if (ev->n_streams < 1 || ev->n_streams > ARGUS_MAX_STREAMS) return ARGUS_EINVAL;
  if (keyed && (int64_t)ev->n_kernels * ev->n_streams > ARGUS_MAX_KERNELS) return ARGUS_EINVAL;
  const int64_t n_seg = (int64_t)ev->n_ranks * ev->n_steps;
  if (n_seg > INT32_MAX) return ARGUS_EINVAL;
  if (!ev->seg_off) return ARGUS_EINVAL;
  if (ev->n_events > 0 && (!ev->kernel_id || !ev->stream || !ev->start_ns || !ev->end_ns)) return ARGUS_EINVAL;
  if (!out->count || !out->sum_ns || !out->min_ns || !out->max_ns || !out->hist || !out->n_valid ||
      !out->n_invalid || !out->t_first || !out->t_last || !out->step_ns || !out->busy_ns || !out->stream_busy_ns)
    return ARGUS_EINVAL;
  if ((reinterpret_cast<uintptr_t>(out->hist) & 15u) != 0) return ARGUS_EINVAL;  // 16-byte histogram stores
  int rc = check_device();
  if (rc != ARGUS_OK) return rc;
  hipStream_t st = (hipStream_t)stream;
  uint32_t* queue = static_cast<uint32_t*>(workspace);
  rc = status_of(launch_clear(out->dev_status, queue, st));
  if (rc != ARGUS_OK) return rc;
  SummarizeLaunch l{ev->kernel_id, ev->stream, ev->start_ns, ev->end_ns, ev->seg_off, ev->n_events, (int32_t)n_seg,
                    ev->n_kernels, ev->n_streams, keyed ? 1 : 0, out->count, out->sum_ns, out->min_ns, out->max_ns,
                    out->hist, out->n_valid, out->n_invalid, out->t_first, out->t_last, out->step_ns, out->busy_ns,
                    out->stream_busy_ns, out->wire_bytes, out->dev_status, queue};
  return status_of(launch_summarize(l, st));
}

int argus_summarize(const argus_events_t* ev, const argus_summary_t* out, void* workspace, size_t workspace_bytes,
                    void* stream) {
  return summarize_impl(ev, out, workspace, workspace_bytes, stream, false);
}

int argus_summarize_keyed(const argus_events_t* ev, const argus_summary_t* out, void* workspace,
                          size_t workspace_bytes, void* stream) {
  return summarize_impl(ev, out, workspace, workspace_bytes, stream, true);
}

int argus_summarize_noalloc(const argus_events_t* ev, const argus_summary_t* out, void* stream) {
  if (!ev || !out) return ARGUS_EINVAL;
  const size_t need = argus_summarize_workspace(ev);
  if (need > ARGUS_NOALLOC_SCRATCH_BYTES) return ARGUS_EINVAL;  // scratch too small for this call
  int rc = check_device();
  if (rc != ARGUS_OK) return rc;
  void* ws = nullptr;
  rc = scratch_of_current_device(&ws);
  if (rc != ARGUS_OK) return rc;
  return summarize_impl(ev, out, ws, ARGUS_NOALLOC_SCRATCH_BYTES, stream, false);
}

void argus_xr_default(argus_xr_params_t* p) {
  if (!p) return;
  p->min_ranks = 3;
  p->c_min_pair = 8;
  p->min_kernels = 8;
  p->k_mad_pm = 5189;
  p->ratio_pm = 1250;
  p->alpha_pm = 1500;
  p->tau_rank_pm = 20;
}

size_t argus_cross_rank_workspace(int32_t n_ranks, int32_t n_steps, int32_t n_kernels) {
  if (n_ranks < 0 || n_steps < 0 || n_kernels < 0) return 0;
  return (size_t)n_ranks * (size_t)n_steps * (size_t)n_kernels * sizeof(int64_t);
}

int argus_cross_rank(const uint32_t* count, const int64_t* sum_ns, int32_t n_ranks, int32_t n_steps,
                     int32_t n_kernels, const argus_xr_params_t* params, const argus_xr_out_t* out, void* workspace,
                     size_t workspace_bytes, void* stream) {
  if (!count || !sum_ns || !params || !out) return ARGUS_EINVAL;
  if (n_ranks < 1 || n_ranks > ARGUS_MAX_XR_RANKS || n_steps < 1 || n_steps > 65535 || n_kernels < 1 ||
      n_kernels > ARGUS_MAX_XR_KERNELS)
    return ARGUS_EINVAL;
  if ((int64_t)n_ranks * n_steps > INT32_MAX || (int64_t)n_steps * n_kernels > INT32_MAX) return ARGUS_EINVAL;
  const argus_xr_params_t& p = *params;
  if (p.min_ranks < 1 || p.c_min_pair < 0 || p.min_kernels < 0 || p.k_mad_pm < 0 || p.ratio_pm < 0 ||
      p.alpha_pm < 0 || p.tau_rank_pm < -1000)
    return ARGUS_EINVAL;
  const argus_xr_out_t& o = *out;
  if (!o.n_present || !o.med_ns || !o.mad_ns || !o.q1_ns || !o.q3_ns || !o.xmean_ns || !o.n_flag ||
      !o.n_degraded || !o.z || !o.flags || !o.score_pm || !o.n_eval || !o.n_flag_rank || !o.straggler)
    return ARGUS_EINVAL;
  if (!workspace || workspace_bytes < argus_cross_rank_workspace(n_ranks, n_steps, n_kernels)) return ARGUS_EINVAL;
  int rc = check_device();
  if (rc != ARGUS_OK) return rc;
  hipStream_t st = (hipStream_t)stream;
  rc = status_of(launch_clear(o.dev_status, nullptr, st));
  if (rc != ARGUS_OK) return rc;
  CrossRankLaunch l{count, sum_ns, n_ranks, n_steps, n_kernels, p, o, static_cast<int64_t*>(workspace)};
  return status_of(launch_cross_rank(l, st));
}

void argus_l1_default(argus_l1_params_t* p) {
  if (!p) return;
  p->W = 5;
  p->theta_pm = 1500;
  p->beta_pm = 1200;
  p->rho_pm = 1300;
  p->cmax_pm = 100;
  p->min_seg = 2;
}

size_t argus_iter_windows_workspace(int32_t n_ranks, int32_t n_steps) {
  (void)n_ranks;
  (void)n_steps;
  return 0;
}

int argus_iter_windows(const int64_t* step_ns, int32_t n_ranks, int32_t n_steps, const argus_l1_params_t* params,
                       uint8_t* flags, uint8_t* cls, int32_t* eff_width, int32_t* cp, float* cp_ratio,
                       int32_t* dev_status, void* workspace, size_t workspace_bytes, void* stream) {
  (void)workspace;
  (void)workspace_bytes;
  if (!params || !cls || !eff_width || !cp) return ARGUS_EINVAL;
  if (n_ranks < 0 || n_steps < 0 || n_steps > ARGUS_MAX_L1_STEPS) return ARGUS_EINVAL;
  if (n_steps > 0 && n_ranks > 0 && (!step_ns || !flags)) return ARGUS_EINVAL;
  const argus_l1_params_t& p = *params;
  if (p.W < 1 || p.theta_pm < 0 || p.beta_pm < 0 || p.rho_pm < 0 || p.cmax_pm < 0 || p.min_seg < 1)
    return ARGUS_EINVAL;
  int rc = check_device();
  if (rc != ARGUS_OK) return rc;
  hipStream_t st = (hipStream_t)stream;
  rc = status_of(launch_clear(dev_status, nullptr, st));
  if (rc != ARGUS_OK) return rc;
  IterWindowsLaunch l{step_ns, n_ranks, n_steps, p, flags, cls, eff_width, cp, cp_ratio, dev_status};
  return status_of(launch_iter_windows(l, st));
}

void argus_kde_default(argus_kde_params_t* p) {
  if (!p) return;
  p->sub_bits = 6;
  p->frac_pm = 50;
  p->min_count = 3;
  p->gap = 48;
}

size_t argus_kde_workspace(const argus_events_t* ev) {
  if (!ev || ev->n_ranks < 0 || ev->n_steps < 0 || ev->n_kernels < 0 || ev->n_events < 0) return 0;
  return kde_workspace_bytes(ev->n_events, (int64_t)ev->n_ranks * ev->n_steps,
                             (int64_t)ev->n_ranks * ev->n_steps * ev->n_kernels);
}

int argus_kde(const argus_events_t* ev, const argus_summary_t* sum, const argus_kde_params_t* params,
              const argus_kde_out_t* out, void* workspace, size_t workspace_bytes, void* stream) {
  if (!ev || !sum || !params || !out) return ARGUS_EINVAL;
  if (ev->n_ranks < 0 || ev->n_steps < 0 || ev->n_events < 0) return ARGUS_EINVAL;
  if (ev->n_kernels < 1 || ev->n_kernels > ARGUS_MAX_KDE_KERNELS) return ARGUS_EINVAL;
  if (ev->n_streams < 1 || ev->n_streams > ARGUS_MAX_STREAMS) return ARGUS_EINVAL;
  const int64_t n_seg = (int64_t)ev->n_ranks * ev->n_steps;
  if (n_seg > INT32_MAX || n_seg * ev->n_kernels > (int64_t)UINT32_MAX) return ARGUS_EINVAL;
  if (!ev->seg_off) return ARGUS_EINVAL;
  if (ev->n_events > 0 && (!ev->kernel_id || !ev->stream || !ev->start_ns || !ev->end_ns)) return ARGUS_EINVAL;
  if (!sum->count || !sum->min_ns || !sum->max_ns) return ARGUS_EINVAL;
  if (!out->n_clusters || !out->count || !out->p50_ns || !out->p99_ns) return ARGUS_EINVAL;
  if (((reinterpret_cast<uintptr_t>(out->count) | reinterpret_cast<uintptr_t>(out->p50_ns) |
        reinterpret_cast<uintptr_t>(out->p99_ns)) & 15u) != 0)
    return ARGUS_EINVAL;  // per-cell records are written with 16-byte stores
  const argus_kde_params_t& p = *params;
  if (p.sub_bits < 1 || p.sub_bits > 6 || p.frac_pm < 0 || p.frac_pm > 1000 || p.min_count < 1 || p.gap < 0)
    return ARGUS_EINVAL;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0 ||
      workspace_bytes < argus_kde_workspace(ev))
    return ARGUS_EINVAL;
  int rc = check_device();
  if (rc != ARGUS_OK) return rc;
  KdeLaunch l{ev->kernel_id, ev->stream, ev->start_ns, ev->end_ns, ev->seg_off, ev->n_events, (int32_t)n_seg,
              ev->n_kernels, ev->n_streams, sum->count, sum->min_ns, sum->max_ns, sum->n_invalid, p, *out,
              workspace};
  return status_of(launch_kde(l, (hipStream_t)stream));
}

void argus_w1_default(argus_w1_params_t* p) {
  if (!p) return;
  p->grid = 64;
  p->min_ranks = 3;
  p->alpha_pm = 1500;
}

size_t argus_w1_workspace(int32_t n_ranks, int32_t n_steps, int32_t n_kernels, int32_t grid) {
  return w1_workspace_bytes(n_ranks, n_steps, n_kernels, grid);
}

int argus_w1(const argus_kde_out_t* clusters, int32_t n_ranks, int32_t n_steps, int32_t n_kernels,
             const argus_w1_params_t* params, const argus_w1_out_t* out, void* workspace, size_t workspace_bytes,
             void* stream) {
  if (!clusters || !params || !out) return ARGUS_EINVAL;
  if (n_ranks < 1 || n_ranks > ARGUS_MAX_W1_RANKS || n_steps < 1 || n_steps > ARGUS_MAX_W1_STEPS || n_kernels < 1)
    return ARGUS_EINVAL;
  const int64_t SK = (int64_t)n_steps * n_kernels;
  if (SK > INT32_MAX || SK * n_ranks > INT32_MAX) return ARGUS_EINVAL;
  const argus_w1_params_t& p = *params;
  if (p.grid < 2 || p.grid > ARGUS_MAX_W1_GRID || p.min_ranks < 1 || p.alpha_pm < 0) return ARGUS_EINVAL;
  if (!clusters->n_clusters || !clusters->count || !clusters->p50_ns || !clusters->p99_ns) return ARGUS_EINVAL;
  auto misaligned = [](const void* q, uintptr_t m) { return (reinterpret_cast<uintptr_t>(q) & (m - 1)) != 0; };
  if (misaligned(clusters->count, 16) || misaligned(clusters->p50_ns, 16) || misaligned(clusters->p99_ns, 16))
    return ARGUS_EINVAL;
  const argus_w1_out_t& o = *out;
  if (!o.n_present || !o.lo_ns || !o.hi_ns || !o.q1 || !o.q3 || !o.fence || !o.n_flag || !o.score || !o.flag)
    return ARGUS_EINVAL;
  if (!workspace || misaligned(workspace, 256) ||
      workspace_bytes < argus_w1_workspace(n_ranks, n_steps, n_kernels, p.grid))
    return ARGUS_EINVAL;
  int rc = check_device();
  if (rc != ARGUS_OK) return rc;
  hipStream_t st = (hipStream_t)stream;
  rc = status_of(launch_clear(o.dev_status, nullptr, st));
  if (rc != ARGUS_OK) return rc;
  W1Launch l{clusters->n_clusters, clusters->count, clusters->p50_ns, clusters->p99_ns, n_ranks, n_steps,
             n_kernels, p, o, workspace};
  return status_of(launch_w1(l, st));
}

void argus_l2_default(argus_l2_params_t* p) {
  if (!p) return;
  p->min_group = 3;
  p->cv_mild_pm = 20;
  p->cv_severe_pm = 50;
  p->z_pm = 3000;
}

size_t argus_l2_workspace(int32_t n_ranks, int32_t n_dims) { return l2_workspace_bytes(n_ranks, n_dims); }

int argus_l2(const uint32_t* count, const int64_t* sum_ns, int32_t n_ranks, int32_t n_steps, int32_t n_events,
             const argus_groups_t* groups, const argus_l2_params_t* params, const argus_l2_out_t* out,
             void* workspace, size_t workspace_bytes, void* stream) {
  if (!count || !sum_ns || !groups || !params || !out) return ARGUS_EINVAL;
  if (n_ranks < 1 || n_ranks > ARGUS_MAX_L2_RANKS || n_steps < 1 || n_events < 1) return ARGUS_EINVAL;
  const argus_groups_t& g = *groups;
  if (!g.route || !g.group_off || !g.members) return ARGUS_EINVAL;
  if (g.n_dims < 1 || g.n_dims > ARGUS_MAX_L2_DIMS || g.max_groups < 1 || g.max_groups > 65535) return ARGUS_EINVAL;
  if ((int64_t)g.max_groups * n_ranks >= ((int64_t)1 << 32)) return ARGUS_EINVAL;
  if ((int64_t)n_steps * g.n_dims > 65535) return ARGUS_EINVAL;
  const int64_t cells = (int64_t)n_ranks * n_steps * n_events;
  if (cells > ((int64_t)1 << 40) || (int64_t)n_steps * n_events * g.max_groups > ((int64_t)1 << 40))
    return ARGUS_EINVAL;
  const argus_l2_params_t& p = *params;
  if (p.min_group < 2 || p.cv_mild_pm < 0 || p.cv_mild_pm > 1000000 || p.cv_severe_pm < 0 ||
      p.cv_severe_pm > 1000000 || p.z_pm < 0 || p.z_pm > 1000000)
    return ARGUS_EINVAL;
  const argus_l2_out_t& o = *out;
  if (!o.n || !o.mean_ns || !o.std_ns || !o.cv || !o.cls || !o.n_strag || !o.z || !o.flags) return ARGUS_EINVAL;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 3u) != 0 ||
      workspace_bytes < argus_l2_workspace(n_ranks, g.n_dims))
    return ARGUS_EINVAL;
  int rc = check_device();
  if (rc != ARGUS_OK) return rc;
  hipStream_t st = (hipStream_t)stream;
  rc = status_of(launch_clear(o.dev_status, nullptr, st));
  if (rc != ARGUS_OK) return rc;
  L2Launch l{count, sum_ns, n_ranks, n_steps, n_events, g, p, o, workspace};
  return status_of(launch_l2(l, st));
}

size_t argus_compact_workspace(int32_t n_ranks, int32_t n_steps) {
  if (n_ranks < 0 || n_steps < 0) return 0;
  return (size_t)n_ranks * (size_t)n_steps * sizeof(int64_t);
}

int argus_compact(const argus_summary_t* sum, int32_t n_ranks, int32_t n_steps, int32_t n_cells, int32_t n_streams,
                  uint8_t* out, int64_t capacity, int64_t* seg_byte_off, int32_t* dev_status, void* workspace,
                  size_t workspace_bytes, void* stream) {
  if (!sum || !seg_byte_off) return ARGUS_EINVAL;
  if (n_ranks < 0 || n_steps < 0 || n_cells < 1 || n_streams < 0 || n_streams > ARGUS_MAX_STREAMS) return ARGUS_EINVAL;
  if (n_streams > 0 && (n_cells % n_streams != 0 || n_cells / n_streams > (1 << 24))) return ARGUS_EINVAL;
  if (n_streams == 0 && n_cells > (1 << 24)) return ARGUS_EINVAL;
  const int64_t n_seg = (int64_t)n_ranks * n_steps;
  if (n_seg > INT32_MAX) return ARGUS_EINVAL;
  if (capacity < 0 || (capacity > 0 && !out)) return ARGUS_EINVAL;
  if (n_seg > 0 && (!sum->count || !sum->sum_ns || !sum->min_ns || !sum->max_ns || !sum->hist)) return ARGUS_EINVAL;
  if ((reinterpret_cast<uintptr_t>(sum->hist) & 15u) != 0) return ARGUS_EINVAL;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 7u) != 0 ||
      workspace_bytes < argus_compact_workspace(n_ranks, n_steps))
    return ARGUS_EINVAL;
  int rc = check_device();
  if (rc != ARGUS_OK) return rc;
  hipStream_t st = (hipStream_t)stream;
  rc = status_of(launch_clear(dev_status, nullptr, st));
  if (rc != ARGUS_OK) return rc;
  CompactLaunch l{sum->count, sum->sum_ns, sum->min_ns, sum->max_ns, sum->hist, (int32_t)n_seg, n_cells, n_streams,
                  out, capacity, seg_byte_off, dev_status, static_cast<int64_t*>(workspace)};
  return status_of(launch_compact(l, st));
}

}  // extern "C"
