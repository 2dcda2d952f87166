// Per-(rank, step, kernel id) summarization of raw kernel-event arrays.
//
// Paper: section 4.3 (kernel activity records: kernel, launch time,
// duration, stream) and section 5.2 (all raw events of each (kernel, stream,
// rank) in a time window are reduced to compact statistics; durations are
// log-transformed and evaluated on an equally spaced grid). A window here is
// one step, i.e. one seg_off segment; the grid is octaves of ns.
//
// Design (gfx950):
// * One 1024-thread workgroup owns one rank-step segment and streams its
//   structure-of-arrays events from HBM once, with coalesced non-temporal
//   loads, four events per thread in flight per iteration.
// * Per-kernel state is privatised in LDS: 64-bit sum, min and max, and an
//   8-bin window of the octave histogram anchored at the first duration seen
//   for that kernel (lognormal kernels span two or three octaves). Bins
//   outside the window go to a small pool of full 32-bin records that a
//   kernel claims on first need. If the pool runs dry the kernel is marked
//   and redone exactly in another pass over the segment, so the result is
//   exact for every input; typical traces need one pass.
// * Up to 2048 kernel ids are held per pass; larger id spaces are covered in
//   id ranges, one pass each.
// * Per-segment aggregates (valid/invalid counts, first start, last end,
//   busy time) are kept in registers and reduced once per segment; per-stream
//   busy time uses LDS atomics.
// * The flush writes every output element exactly once (identity values for
//   absent kernels), coalesced, so outputs need no clearing.
#include "argus_internal.h"

namespace argus {
namespace {

constexpr int kThreads = 1024;
constexpr int kUnroll = 4;
constexpr int kWin = 8;        // histogram bins held inline per kernel
constexpr int kPool = 32;      // full 32-bin records per pass
constexpr uint32_t kBaseUnset = 0xFFu;
constexpr uint32_t kStNone = 0, kStBusy = 0xFE, kStPoison = 0xFF;
constexpr uint32_t kDone = 1u << 16;

// meta word of a slot: bits 0-7 window base bin (0xFF unset), bits 8-15
// full-record state (0 none, 1..kPool record index + 1, 0xFE being claimed,
// 0xFF pool exhausted: redo in another pass), bit 16 already written.

template <int NSLOT>
struct Smem {
  unsigned long long sum[NSLOT];
  long long mn[NSLOT];
  long long mx[NSLOT];
  uint32_t win[NSLOT][kWin];
  uint32_t meta[NSLOT];
  uint32_t pool[kPool][NB];
  unsigned long long stream_busy[ARGUS_MAX_STREAMS];
  unsigned long long red_busy, red_wire;
  long long red_first, red_last;
  uint32_t red_valid, red_invalid;
  uint32_t npool, poison;
};

struct Args {
  const int32_t* kernel_id;
  const int32_t* stream;
  const int64_t* start_ns;
  const int64_t* end_ns;
  const int64_t* seg_off;
  int64_t n_events;
  int32_t n_kernels, n_streams;
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
};

// Count bin b of a kernel outside its inline window in a full pool record,
// claiming one for the kernel on first need. Several lanes of one wavefront
// may race for the same claim; the loser waits until the winner publishes.
// The loop only exits when no active lane of the wavefront is still pending,
// so the winner's publish always executes inside the loop body, before any
// waiting lane of its own wavefront re-reads the state (a per-lane early
// exit would let the compiler move the publish past the loop, where a
// waiting lane of the same wavefront could never observe it).
template <int NSLOT>
__device__ __forceinline__ void pool_add(Smem<NSLOT>& sm, int slot, uint32_t m, int b) {
  bool pending = true;
  while (true) {
    if (pending) {
      const uint32_t st = (m >> 8) & 0xFFu;
      if (st == kStPoison) {
        pending = false;
      } else if (st != kStNone && st != kStBusy) {
        atomicAdd(&sm.pool[st - 1][b], 1u);
        pending = false;
      } else if (st == kStNone) {
        const uint32_t claim = (m & ~0xFF00u) | (kStBusy << 8);
        const uint32_t old = atomicCAS(&sm.meta[slot], m, claim);
        if (old == m) {
          const uint32_t idx = atomicAdd(&sm.npool, 1u);
          uint32_t fin;
          if (idx < (uint32_t)kPool) {
            atomicAdd(&sm.pool[idx][b], 1u);
            fin = (m & ~0xFF00u) | ((idx + 1u) << 8);
          } else {
            fin = (m & ~0xFF00u) | (kStPoison << 8);
            lds_store(&sm.poison, 1u);
          }
          atomicExch(&sm.meta[slot], fin);
          pending = false;
        } else {
          m = old;
        }
      } else {
        m = lds_load(&sm.meta[slot]);
      }
    }
    if (!__any(pending)) break;
  }
}

template <int NSLOT>
__device__ __forceinline__ void slot_add(Smem<NSLOT>& sm, int slot, uint64_t d) {
  uint32_t m = lds_load(&sm.meta[slot]);
  if (m & kDone) return;
  const int b = octave_bin(d);
  if ((m & 0xFFu) == kBaseUnset) {
    int base = b - 3;
    base = base < 0 ? 0 : (base > NB - kWin ? NB - kWin : base);
    const uint32_t want = (m & ~0xFFu) | (uint32_t)base;
    const uint32_t old = atomicCAS(&sm.meta[slot], m, want);
    m = (old == m) ? want : old;
  }
  const int off = b - (int)(m & 0xFFu);
  if ((unsigned)off < (unsigned)kWin)
    atomicAdd(&sm.win[slot][off], 1u);
  else
    pool_add(sm, slot, m, b);
  atomicAdd(&sm.sum[slot], (unsigned long long)d);
  atomicMin(&sm.mn[slot], (long long)d);
  atomicMax(&sm.mx[slot], (long long)d);
}

template <int NSLOT>
__device__ __forceinline__ void slot_reset(Smem<NSLOT>& sm, int slot) {
  sm.sum[slot] = 0;
  sm.mn[slot] = INT64_MAX;
  sm.mx[slot] = INT64_MIN;
#pragma unroll
  for (int w = 0; w < kWin; ++w) sm.win[slot][w] = 0;
  sm.meta[slot] = kBaseUnset;
}

template <int NSLOT>
__global__ __launch_bounds__(kThreads) void summarize_kernel(Args a) {
  __shared__ Smem<NSLOT> sm;
  const int tid = threadIdx.x;
  const int64_t g = blockIdx.x;
  const int32_t K = a.n_kernels, NS = a.n_streams;

  int64_t lo = a.seg_off[g], hi = a.seg_off[g + 1];
  const bool bad = !(lo >= 0 && lo <= hi && hi <= a.n_events && hi - lo <= (int64_t)UINT32_MAX);
  if (bad) {
    lo = hi = 0;
    if (tid == 0 && a.dev_status) atomicOr(a.dev_status, (int32_t)ARGUS_DEV_BAD_SEGMENT);
  }
  if (tid < NS) sm.stream_busy[tid] = 0;
  if (tid == 0) {
    sm.red_busy = 0;
    sm.red_wire = 0;
    sm.red_first = INT64_MAX;
    sm.red_last = INT64_MIN;
    sm.red_valid = 0;
    sm.red_invalid = 0;
  }

  uint32_t nv = 0, ni = 0;
  unsigned long long busy = 0, wire = 0;
  long long tf = INT64_MAX, tl = INT64_MIN;
  bool first_scan = true;

  for (int32_t kb = 0; kb < K; kb += NSLOT) {
    const int nk = K - kb < NSLOT ? K - kb : NSLOT;
    for (int s = tid; s < nk; s += kThreads) slot_reset(sm, s);
    while (true) {
      for (int i = tid; i < kPool * NB; i += kThreads) (&sm.pool[0][0])[i] = 0;
      if (tid == 0) {
        sm.npool = 0;
        sm.poison = 0;
      }
      __syncthreads();

      for (int64_t i0 = lo; i0 < hi; i0 += (int64_t)kUnroll * kThreads) {
        int32_t kid[kUnroll], st[kUnroll];
        int64_t t0[kUnroll], t1[kUnroll];
        bool in[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int64_t i = i0 + (int64_t)u * kThreads + tid;
          in[u] = i < hi;
          if (in[u]) {
            kid[u] = __builtin_nontemporal_load(a.kernel_id + i);
            st[u] = __builtin_nontemporal_load(a.stream + i);
            t0[u] = __builtin_nontemporal_load(a.start_ns + i);
            t1[u] = __builtin_nontemporal_load(a.end_ns + i);
          }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          if (!in[u]) continue;
          const bool valid = kid[u] >= 0 && kid[u] < K && st[u] >= 0 && st[u] < NS && t0[u] >= 0 && t1[u] >= t0[u];
          const uint64_t d = (uint64_t)t1[u] - (uint64_t)t0[u];
          if (first_scan) {
            if (valid) {
              nv++;
              busy += d;
              tf = t0[u] < tf ? t0[u] : tf;
              tl = t1[u] > tl ? t1[u] : tl;
              atomicAdd(&sm.stream_busy[st[u]], (unsigned long long)d);
            } else {
              ni++;
            }
          }
          const int slot = kid[u] - kb;
          if (valid && (unsigned)slot < (unsigned)nk) slot_add(sm, slot, d);
        }
      }
      first_scan = false;
      __syncthreads();

      // flush: per-kernel scalars and wire size
      for (int s = tid; s < nk; s += kThreads) {
        const uint32_t m = sm.meta[s];
        const uint32_t pst = (m >> 8) & 0xFFu;
        if ((m & kDone) || pst == kStPoison) continue;
        uint32_t cnt = 0, nnz = 0;
#pragma unroll
        for (int w = 0; w < kWin; ++w) {
          cnt += sm.win[s][w];
          nnz += sm.win[s][w] != 0;
        }
        if (pst != kStNone) {
          for (int b = 0; b < NB; ++b) {
            cnt += sm.pool[pst - 1][b];
            nnz += sm.pool[pst - 1][b] != 0;
          }
        }
        const int64_t c = g * K + kb + s;
        a.count[c] = cnt;
        a.sum_ns[c] = (int64_t)sm.sum[s];
        a.min_ns[c] = sm.mn[s];
        a.max_ns[c] = sm.mx[s];
        if (cnt) wire += 33u + 5u * nnz;
      }
      // flush: histograms, four bins per thread, coalesced 16-byte stores
      for (int it = tid; it < nk * (NB / 4); it += kThreads) {
        const int s = it >> 3, q = it & 7;
        const uint32_t m = sm.meta[s];
        const uint32_t pst = (m >> 8) & 0xFFu;
        if ((m & kDone) || pst == kStPoison) continue;
        const int base = (int)(m & 0xFFu);
        uint32_t v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int b = 4 * q + j;
          const int off = b - base;
          v[j] = (base != (int)kBaseUnset && (unsigned)off < (unsigned)kWin) ? sm.win[s][off] : 0u;
          if (pst != kStNone) v[j] += sm.pool[pst - 1][b];
        }
        const int64_t c = g * K + kb + s;
        *reinterpret_cast<uint4*>(a.hist + c * NB + 4 * q) = make_uint4(v[0], v[1], v[2], v[3]);
      }
      __syncthreads();
      const bool again = sm.poison != 0;
      // mark written kernels done; kernels that found the pool empty start over
      for (int s = tid; s < nk; s += kThreads) {
        const uint32_t m = sm.meta[s];
        if (m & kDone) continue;
        if (((m >> 8) & 0xFFu) == kStPoison)
          slot_reset(sm, s);
        else
          sm.meta[s] = m | kDone;
      }
      __syncthreads();
      if (!again) break;
    }
  }

  // per-segment aggregates
  const unsigned long long wv = wave_sum_u64(nv), wi = wave_sum_u64(ni);
  const unsigned long long wb = wave_sum_u64(busy), ww = wave_sum_u64(wire);
  const long long wf = wave_min_i64(tf), wl = wave_max_i64(tl);
  if ((tid & 63) == 0) {
    atomicAdd(&sm.red_valid, (uint32_t)wv);
    atomicAdd(&sm.red_invalid, (uint32_t)wi);
    atomicAdd(&sm.red_busy, wb);
    atomicAdd(&sm.red_wire, ww);
    atomicMin(&sm.red_first, wf);
    atomicMax(&sm.red_last, wl);
  }
  __syncthreads();
  if (tid == 0) {
    a.n_valid[g] = sm.red_valid;
    a.n_invalid[g] = sm.red_invalid;
    a.t_first[g] = sm.red_first;
    a.t_last[g] = sm.red_last;
    a.step_ns[g] = sm.red_valid ? sm.red_last - sm.red_first : 0;
    a.busy_ns[g] = (int64_t)sm.red_busy;
    if (a.wire_bytes) a.wire_bytes[g] = (int64_t)sm.red_wire;
  }
  if (tid < NS) a.stream_busy_ns[g * NS + tid] = (int64_t)sm.stream_busy[tid];
}

template <int NSLOT>
hipError_t launch_t(const Args& args, int32_t n_seg, hipStream_t st) {
  hipLaunchKernelGGL(summarize_kernel<NSLOT>, dim3(n_seg), dim3(kThreads), 0, st, args);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_summarize(const SummarizeLaunch& l, hipStream_t st) {
  Args a{l.kernel_id, l.stream, l.start_ns, l.end_ns, l.seg_off, l.n_events, l.n_kernels, l.n_streams,
         l.count, l.sum_ns, l.min_ns, l.max_ns, l.hist, l.n_valid, l.n_invalid, l.t_first, l.t_last,
         l.step_ns, l.busy_ns, l.stream_busy_ns, l.wire_bytes, l.dev_status};
  if (l.n_seg == 0) return hipSuccess;
  if (l.n_kernels <= 64) return launch_t<64>(a, l.n_seg, st);
  if (l.n_kernels <= 512) return launch_t<512>(a, l.n_seg, st);
  return launch_t<2048>(a, l.n_seg, st);
}

}  // namespace argus
