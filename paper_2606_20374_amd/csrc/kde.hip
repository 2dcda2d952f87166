// Duration clustering per (rank, step, kernel id): valleys of a Gaussian KDE
// over log-duration, each cluster reported as (count, p50, p99) (section 5.2,
// Eq. 1; the step-by-step definition is in include/argus.h).
//
// Kernels, in launch order:
//   kde_scatter_staged_kernel / kde_scatter_kernel
//                        one workgroup per segment (persistent queue): the
//                        segment's valid durations are bucketed by kernel id
//                        into the workspace, a counting sort whose counts are
//                        argus_summarize's, so each cell's durations become
//                        contiguous. The staged variant (id spaces of up to
//                        2,048 ids) collects each id's positions in LDS and
//                        writes them as aligned 64-byte groups. HBM bound:
//                        24 B read and 8 B written per event.
//   kde_route_kernel,    every cell routed once: empty cells written, heavy
//   kde_lane_order_kernel cells to the workgroup tier, large or wide-grid
//                        cells to tier 0, the rest to the lane passes in
//                        cost-class order (grid size x duration count).
//   kde_lane_kernel<64>, one cell per lane, 64 cells per wavefront (grids of
//   kde_lane_kernel<256> up to 64 / 65-256 points, up to 255 durations).
//   kde_block_kernel     one 128-thread workgroup per cell of 2,048 or more
//                        durations.
//   kde_cell_kernel<0>   one wavefront per cell, cells claimed 64 at a time
//                        with their summaries, n^(-1/5) and (for cells of up to
//                        256 durations) the next cell's durations prefetched
//                        while the current cell is processed: grid histogram
//                        in LDS, exact bandwidth, integer-weight density
//                        (sparse over occupied grid points when that is
//                        cheaper), valleys, filters, and p50 / p99 by exact
//                        radix selection inside the target grid bin. 7.8 KB of
//                        LDS per wavefront; cells that need more go to a list.
//   kde_cell_kernel<1>   the listed cells with 20 KB per wavefront;
//   kde_cell_kernel<2>   what still does not fit, 105 KB per wavefront (any
//                        grid of the 64-bit duration range fits).
#include <atomic>
#include <cmath>
#include <mutex>
#include <vector>

#include "argus_internal.h"
#include "kde_math.h"

namespace argus {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef long long v2l __attribute__((ext_vector_type(2)));

constexpr int kScatterThreads = 512;
constexpr int kWave = 64;
constexpr int kMaxC = ARGUS_KDE_MAXC;
constexpr int kMaxT = 2 * kMaxC;  // selection targets: p50 and p99 per cluster
constexpr int kPowTab = 65536;    // n^(-1/5) tabulated for n below this
constexpr int kRegVals = 4;       // cells of up to 256 durations stay in registers
constexpr int kDigit = 6;         // radix-selection digit width (64 counters per target)

// LDS per tier: grid words (histogram, chunk offsets, occupied-point list
// and symmetric zero-padded weight table: at most 3 G + 2 T + 515 words; the
// selection lists of the wavefront tiers take 1,024) and valley capacity.
// Tier 2 holds any grid of the duration range (at most 4,032 points, T < G).
template <int TIER>
struct Tier;
template <>
struct Tier<0> {
  static constexpr int kWords = 1712, kCand = 64;
};
template <>
struct Tier<1> {
  static constexpr int kWords = 4096, kCand = 256;
};
template <>
struct Tier<2> {
  static constexpr int kWords = 20688, kCand = 2047;
};

// n^(-1/5) for small n (kde_pw), filled once per device.
__device__ double g_kde_pow[kPowTab];


struct KdeArgs {
  const int32_t* kernel_id;
  const int32_t* stream;
  const int64_t* start_ns;
  const int64_t* end_ns;
  const int64_t* seg_off;
  int64_t n_events;
  int32_t n_seg, K, NS, vec_ok;
  int32_t sub_bits, frac_pm, min_count, gap;
  const uint32_t* count;
  const int64_t* min_ns;
  const int64_t* max_ns;
  const uint32_t* n_invalid;  // per segment, or null
  uint8_t* n_clusters;
  uint32_t* cl_count;
  int64_t* p50;
  int64_t* p99;
  int32_t* bw_q8;
  int32_t* dev_status;
  // [0] scatter queue, [1] tier-0 queue, [2] list-1 length, [3] list-1 queue,
  // [4] list-2 length, [5] list-2 queue, [6] first lane pass queue, [7] list-0 length,
  // [8] wide lane pass queue, [9] wide list length, [10] workgroup tier queue, [11] heavy list length,
  // [12] lane list length
  uint32_t* counters;
  uint64_t* bucket;    // [n_events]: segment g's durations from byte 8 seg_off[g], one record per
                       // local position, of 4 bytes (seg_w4[g] = 1) or 8
  uint8_t* seg_w4;     // [n_seg]
  uint32_t* cell_end;  // [cells]: local end offset of each cell's durations
  uint32_t* list1;     // [cells]: the cells of the wide lane pass (from the bottom) and of the
                       // first lane pass (from the top), each in cost-class order; later
                       // cells handed from the workgroup tier and tier 0 to tier 1 (both lane
                       // lists are consumed first)
  uint32_t* list2;     // [cells]: cells handed from the lane tier to tier 0 (list 0, from the bottom) and
                       // to the workgroup tier (heavy list, from the top), later from tier 1 to tier 2
                       // (both are consumed before tier 1 starts)
  uint16_t* lane_key;  // [cells]: route code (a lane pass's cost class, heavy, tier 0, or none)
  uint32_t* lane_cls;  // [2 * 1024]: cells per cost class, then the classes' fill cursors
  uint32_t theta[64];  // ceil(2^(23 + t/64))
};

// ----------------------------------------------------------------- helpers

// the grid index of a duration (kde_math.h)
__device__ __forceinline__ int grid64(uint64_t d, const uint32_t* th) { return kde_grid64(d, th); }
__device__ __forceinline__ int grid32(uint32_t d, const uint32_t* th) { return kde_grid32(d, th); }

// Smallest duration whose 64-per-octave grid value is >= b.
__device__ __forceinline__ uint64_t grid64_lb(int b, const uint32_t* th) {
  if (b <= 0) return 0;
  const int e = b >> 6, t = b & 63;
  if (e >= 64) return ~0ull;
  const uint64_t m = th[t];
  return e >= 23 ? (m << (e - 23)) : ((m + (1ull << (23 - e)) - 1) >> (23 - e));
}

__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

__device__ __forceinline__ uint64_t readlane64(uint64_t v, int l) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)v, l);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(v >> 32), l);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ double readlane_f64(double v, int l) {
  return __builtin_bit_cast(double, readlane64(__builtin_bit_cast(uint64_t, v), l));
}

__device__ __forceinline__ uint64_t wave_min_u64(uint64_t v) {
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t w = __shfl_xor(v, o, kWave);
    v = w < v ? w : v;
  }
  return v;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  for (int o = 32; o > 0; o >>= 1) {
    const uint64_t w = __shfl_xor(v, o, kWave);
    v = w > v ? w : v;
  }
  return v;
}

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  const int l = lane_id();
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t t = __shfl_up(v, o, kWave);
    if (l >= o) v += t;
  }
  return v;
}

// Ordering point of the single-wavefront cell kernels. One wavefront's LDS
// operations are performed in order, so LDS data written by some lanes is
// visible to later reads of other lanes without waiting; the wavefront-scope
// fences only stop the compiler from moving memory operations across this
// point. Unlike a workgroup barrier they do not wait for outstanding global
// loads (the next cell's prefetched durations) or stores (outputs).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ void flag(const KdeArgs& a, int bit) {
  if (a.dev_status) atomicOr(a.dev_status, bit);
}

// ----------------------------------------------------------------- scatter

struct ScatterCtx {
  uint32_t* cur;
  uint64_t* out;
  uint32_t len;
  int32_t K, NS;
};

__device__ __forceinline__ void scatter_one(const ScatterCtx& s, int32_t kid, int32_t st, int64_t t0, int64_t t1) {
  if (kid >= 0 && kid < s.K && st >= 0 && st < s.NS && t0 >= 0 && t1 >= t0) {
    const uint32_t p = atomicAdd(&s.cur[kid], 1u);
    if (p < s.len) s.out[p] = (uint64_t)t1 - (uint64_t)t0;
  }
}

__global__ __launch_bounds__(kScatterThreads) void kde_scatter_kernel(KdeArgs a) {
  __shared__ uint32_t cur[ARGUS_MAX_KDE_KERNELS];
  __shared__ uint32_t wave_tot[kScatterThreads / kWave];
  __shared__ uint32_t claim;
  const int tid = threadIdx.x, K = a.K;
  const int per = (K + kScatterThreads - 1) / kScatterThreads;
  const v4i* K4 = reinterpret_cast<const v4i*>(a.kernel_id);
  const v4i* S4 = reinterpret_cast<const v4i*>(a.stream);
  const v2l* T0 = reinterpret_cast<const v2l*>(a.start_ns);
  const v2l* T1 = reinterpret_cast<const v2l*>(a.end_ns);
  while (true) {
    if (tid == 0) claim = atomicAdd(&a.counters[0], 1u);
    __syncthreads();
    const uint32_t g = claim;
    if (g >= (uint32_t)a.n_seg) break;
    if (tid == 0) a.seg_w4[g] = 0;  // 8-byte records
    // cursors = exclusive prefix of the segment's per-kernel counts
    const uint32_t* cnt = a.count + (int64_t)g * K;
    const int k0 = tid * per, k1 = min(K, k0 + per);
    uint32_t own = 0;
    for (int k = k0; k < k1; ++k) own += cnt[k];
    const uint32_t incl = wave_incl_scan(own);
    if (lane_id() == kWave - 1) wave_tot[tid / kWave] = incl;
    __syncthreads();
    uint32_t base = incl - own;
    for (int w = 0; w < tid / kWave; ++w) base += wave_tot[w];
    for (int k = k0; k < k1; ++k) {
      cur[k] = base;
      base += cnt[k];
    }
    __syncthreads();
    const int64_t lo = a.seg_off[g], hi = a.seg_off[g + 1];
    const bool bad = !(lo >= 0 && lo <= hi && hi <= a.n_events && hi - lo <= (int64_t)UINT32_MAX);
    if (!bad) {
      const ScatterCtx s{cur, a.bucket + lo, (uint32_t)(hi - lo), K, a.NS};
      int64_t a4 = hi, b4 = hi;  // aligned body [a4, b4) in groups of four events
      if (a.vec_ok) {
        const int64_t up = (lo + 3) & ~(int64_t)3, dn = hi & ~(int64_t)3;
        a4 = up < hi ? up : hi;
        b4 = dn > a4 ? dn : a4;
      }
      // head [lo, a4) (the whole segment without aligned arrays) and tail [b4, hi)
      for (int64_t i = lo + tid; i < a4; i += kScatterThreads)
        scatter_one(s, a.kernel_id[i], a.stream[i], a.start_ns[i], a.end_ns[i]);
      for (int64_t i = b4 + tid; i < hi; i += kScatterThreads)
        scatter_one(s, a.kernel_id[i], a.stream[i], a.start_ns[i], a.end_ns[i]);
      const int64_t qb = b4 >> 2;
      int64_t q = (a4 >> 2) + tid;
      v4i nk4 = 0, ns4 = 0;
      v2l na0 = 0, na1 = 0, nb0 = 0, nb1 = 0;
      if (q < qb) {
        nk4 = __builtin_nontemporal_load(K4 + q);
        ns4 = __builtin_nontemporal_load(S4 + q);
        na0 = __builtin_nontemporal_load(T0 + 2 * q);
        na1 = __builtin_nontemporal_load(T0 + 2 * q + 1);
        nb0 = __builtin_nontemporal_load(T1 + 2 * q);
        nb1 = __builtin_nontemporal_load(T1 + 2 * q + 1);
      }
      while (q < qb) {
        const v4i k4 = nk4, s4 = ns4;
        const v2l x0 = na0, x1 = na1, y0 = nb0, y1 = nb1;
        const int64_t qn = q + kScatterThreads;
        if (qn < qb) {
          nk4 = __builtin_nontemporal_load(K4 + qn);
          ns4 = __builtin_nontemporal_load(S4 + qn);
          na0 = __builtin_nontemporal_load(T0 + 2 * qn);
          na1 = __builtin_nontemporal_load(T0 + 2 * qn + 1);
          nb0 = __builtin_nontemporal_load(T1 + 2 * qn);
          nb1 = __builtin_nontemporal_load(T1 + 2 * qn + 1);
        }
        scatter_one(s, k4.x, s4.x, x0.x, y0.x);
        scatter_one(s, k4.y, s4.y, x0.y, y0.y);
        scatter_one(s, k4.z, s4.z, x1.x, y1.x);
        scatter_one(s, k4.w, s4.w, x1.y, y1.y);
        q = qn;
      }
    }
    __syncthreads();
    uint32_t* ends = a.cell_end + (int64_t)g * K;
    for (int k = tid; k < K; k += kScatterThreads) ends[k] = cur[k];
    __syncthreads();
  }
}

// ----------------------------------------------------------- staged scatter
// For id spaces of up to kStageK kernel ids. Scattering each duration with
// its own store leaves partly written cache lines for the many rare kernel
// ids, and HBM then writes about twice the durations' bytes. Here each kernel
// id keeps a window of one 64-byte group of positions (W = 8 records of 8
// bytes or 16 of 4), [done, done + W), in LDS; a duration whose position
// falls inside the window is staged, any later one (a frequent id within one
// round) is stored directly. After each round of 8,192 events the workgroup
// writes out the staged positions up to the last complete aligned 64-byte
// group, or all of them when the id overflowed its window, and advances the
// window. The rule that decides staged or direct reads only the window start,
// which changes between rounds, so the result does not depend on when the
// flushes happen. The workgroup shares only LDS state, so its barriers order
// LDS alone and the next round's loads stay in flight across them.
//
// Record width: a segment's durations are stored in 4 bytes when the segment
// takes the buffer path below and every present cell's summarized maximum is
// below 2^31, else in 8. A 4-byte record saturates at 2^32 - 1. A duration of
// 2^31 or more in such a segment can only come from summaries that do not
// match the events; it lies in a higher octave than its cell's summarized
// maximum, so on a grid of any resolution the cells' range check reports it.
constexpr int kStageThreads = 1024;
constexpr int kStageK = 2048;
constexpr int kStageD = 2;  // groups of four events per thread and round
constexpr uint64_t kW4Max = 0xFFFFFFFFull;  // saturation of a 4-byte record
constexpr uint64_t kW4Lim = 1ull << 31;     // summarized maxima below this allow 4-byte records

template <typename R>
struct StageCtx {
  static constexpr int W = 64 / (int)sizeof(R);  // positions per 64-byte group
  R (*stage)[W];
  uint32_t* cur;
  const uint32_t* done;
  R* out;
  uint32_t len, al;  // segment length; position of local 0 in its 64-byte group (in records)
  int32_t K, NS;
};

template <typename R>
__device__ __forceinline__ R to_record(uint64_t d) {
  if constexpr (sizeof(R) == 8) return d;
  else return (R)(d < kW4Max ? d : kW4Max);
}

template <typename R>
__device__ __forceinline__ void stage_one(const StageCtx<R>& s, int32_t kid, int32_t st, int64_t t0, int64_t t1) {
  constexpr int W = StageCtx<R>::W;
  if (kid >= 0 && kid < s.K && st >= 0 && st < s.NS && t0 >= 0 && t1 >= t0) {
    const uint32_t p = atomicAdd(&s.cur[kid], 1u);
    const R d = to_record<R>((uint64_t)t1 - (uint64_t)t0);
    if (p - s.done[kid] < (uint32_t)W) s.stage[kid][(p + s.al) & (W - 1)] = d;
    else if (p < s.len) s.out[p] = d;
  }
}

// Write out kernel id k's staged positions: up to the last complete aligned
// group, everything when the window overflowed, or everything (final).
template <typename R>
__device__ __forceinline__ void stage_flush(const StageCtx<R>& s, uint32_t* done, int k, bool final) {
  constexpr int W = StageCtx<R>::W;
  const uint32_t c = s.cur[k], dn = done[k];
  if (c == dn) return;
  uint32_t e, nd;
  if (c - dn > (uint32_t)W) {
    e = dn + W;
    nd = c;
  } else if (final) {
    e = nd = c;
  } else {
    const int64_t al = (int64_t)((c + s.al) & ~(uint32_t)(W - 1)) - (int64_t)s.al;
    if (al <= (int64_t)dn) return;
    e = nd = (uint32_t)al;
  }
  for (uint32_t p = dn; p < e; ++p)
    if (p < s.len) s.out[p] = s.stage[k][(p + s.al) & (W - 1)];
  done[k] = nd;
}

// Buffer-resource variants for segments below kBufEvents events. On gfx950
// stores and loads share one wait counter, so a store whose issue depends on
// data (staged or not) leaves the compiler unable to count what follows a
// prefetched load, and it waits for everything, prefetch included, before
// each use. Here every step issues a fixed set of memory instructions:
// loads past the end read zeros, and a lane with nothing to store gives an
// offset past the buffer, which the hardware drops.
typedef unsigned v2u __attribute__((ext_vector_type(2)));
typedef unsigned v4u __attribute__((ext_vector_type(4)));
constexpr uint32_t kOob = 0x80000000u;   // past every buffer below (all under 2^31 bytes)
constexpr int64_t kBufEvents = 1ll << 26;  // 2^26 events of 8 bytes: 512 MB per buffer

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, int64_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

__device__ __forceinline__ void buf_store(__amdgpu_buffer_rsrc_t r, uint32_t off, uint64_t v) {
  __builtin_amdgcn_raw_buffer_store_b64(v2u{(uint32_t)v, (uint32_t)(v >> 32)}, r, (int)off, 0, 0);
}

__device__ __forceinline__ void buf_store(__amdgpu_buffer_rsrc_t r, uint32_t off, uint32_t v) {
  __builtin_amdgcn_raw_buffer_store_b32(v, r, (int)off, 0, 0);
}

// Four events at once. Every lane takes a cursor for all four before any
// result is used, so the four LDS round trips overlap: an event that is not
// valid (or past the end) counts on the spare slot kStageK, which no flush
// reads, and stores nothing.
template <typename R>
__device__ __forceinline__ void stage_four_buf(const StageCtx<R>& s, __amdgpu_buffer_rsrc_t ro, bool ok, v4i k4,
                                               v4i s4, v2l x0, v2l x1, v2l y0, v2l y1) {
  constexpr int W = StageCtx<R>::W;
  const int32_t kid[4] = {k4.x, k4.y, k4.z, k4.w}, st[4] = {s4.x, s4.y, s4.z, s4.w};
  const int64_t t0[4] = {x0.x, x0.y, x1.x, x1.y}, t1[4] = {y0.x, y0.y, y1.x, y1.y};
  bool val[4];
  uint32_t slot[4], p[4], dn[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    val[i] = ok && kid[i] >= 0 && kid[i] < s.K && st[i] >= 0 && st[i] < s.NS && t0[i] >= 0 && t1[i] >= t0[i];
    slot[i] = val[i] ? (uint32_t)kid[i] : (uint32_t)kStageK;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) p[i] = atomicAdd(&s.cur[slot[i]], 1u);
#pragma unroll
  for (int i = 0; i < 4; ++i) dn[i] = s.done[slot[i]];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const R d = to_record<R>((uint64_t)t1[i] - (uint64_t)t0[i]);
    uint32_t off = kOob;
    if (val[i]) {
      if (p[i] - dn[i] < (uint32_t)W) s.stage[slot[i]][(p[i] + s.al) & (W - 1)] = d;
      else if (p[i] < s.len) off = p[i] * (uint32_t)sizeof(R);
    }
    buf_store(ro, off, d);
  }
}

// Flushes of the buffer path in two phases. Plan: each id with staged
// positions to write (as stage_flush decides) takes an entry of an LDS list
// of kFlushCap; ids that find the list full keep their positions staged for
// a later round (the staging rule allows any flush time). Write: one lane
// per (entry, position), kFlushCap * W / kStageThreads stores per thread
// whether used or not.
constexpr int kFlushCap = 512;

struct FlushEntry {
  uint32_t k, dn, e, nd;
};

template <typename R>
__device__ __forceinline__ void stage_plan(const StageCtx<R>& s, const uint32_t* done, int k, FlushEntry* list,
                                           uint32_t* n_list) {
  constexpr int W = StageCtx<R>::W;
  uint32_t dn = 0, e = 0, nd = 0;
  bool act = false;
  if (k < s.K) {
    const uint32_t c = s.cur[k];
    dn = done[k];
    if (c - dn > (uint32_t)W) {
      e = dn + W;
      nd = c;
      act = true;
    } else if (c != dn) {
      const int64_t al = (int64_t)((c + s.al) & ~(uint32_t)(W - 1)) - (int64_t)s.al;
      if (al > (int64_t)dn) {
        e = nd = (uint32_t)al;
        act = true;
      }
    }
  }
  // one list claim per wavefront
  const uint64_t m = __ballot(act);
  uint32_t base = 0;
  const int leader = m ? __builtin_ctzll(m) : 0;
  if (m && lane_id() == leader) base = atomicAdd(n_list, (uint32_t)__popcll(m));
  base = __builtin_amdgcn_readlane(base, leader);
  const uint32_t idx = base + (uint32_t)__popcll(m & ((1ull << lane_id()) - 1ull));
  if (act && idx < (uint32_t)kFlushCap) list[idx] = FlushEntry{(uint32_t)k, dn, e, nd};
}

template <typename R>
__device__ __forceinline__ void stage_write(const StageCtx<R>& s, __amdgpu_buffer_rsrc_t ro, uint32_t* done,
                                            const FlushEntry* list, uint32_t n_list, int tid) {
  constexpr int W = StageCtx<R>::W;
  const uint32_t n = n_list < (uint32_t)kFlushCap ? n_list : (uint32_t)kFlushCap;
#pragma unroll
  for (int j = 0; j < kFlushCap * W / kStageThreads; ++j) {
    const uint32_t slot = (uint32_t)(j * kStageThreads + tid);
    const uint32_t ent = slot / W, i = slot % W;
    uint32_t off = kOob;
    R v = 0;
    if (ent < n) {
      const FlushEntry f = list[ent];
      const uint32_t p = f.dn + i;
      if (p < f.e && p < s.len) {
        off = p * (uint32_t)sizeof(R);
        v = s.stage[f.k][(p + s.al) & (W - 1)];
      }
      if (i == 0) done[f.k] = f.nd;
    }
    buf_store(ro, off, v);
  }
}

// One well-formed segment [lo, hi) of the staged scatter, the cursors set up;
// returns with every staged position written out. Without STREAMS the stream
// array is not read and every stream counts as valid: the segment's summary
// found no invalid event, so every stream is in range (the other validity
// tests stay, as they use what is read anyway).
template <typename R, bool STREAMS>
__device__ void stage_segment(const KdeArgs& a, const StageCtx<R>& s, uint32_t* done, FlushEntry* list,
                              uint32_t* n_list, int64_t lo, int64_t hi, int tid) {
  const v4i* K4 = reinterpret_cast<const v4i*>(a.kernel_id);
  const v4i* S4 = reinterpret_cast<const v4i*>(a.stream);
  const v2l* T0 = reinterpret_cast<const v2l*>(a.start_ns);
  const v2l* T1 = reinterpret_cast<const v2l*>(a.end_ns);
  int64_t a4 = hi, b4 = hi;  // aligned body [a4, b4) in groups of four events
  if (a.vec_ok) {
    const int64_t up = (lo + 3) & ~(int64_t)3, dn = hi & ~(int64_t)3;
    a4 = up < hi ? up : hi;
    b4 = dn > a4 ? dn : a4;
  }
  // head [lo, a4) (the whole segment without aligned arrays) and tail [b4, hi)
  for (int64_t i = lo + tid; i < a4; i += kStageThreads)
    stage_one(s, a.kernel_id[i], STREAMS ? a.stream[i] : 0, a.start_ns[i], a.end_ns[i]);
  for (int64_t i = b4 + tid; i < hi; i += kStageThreads)
    stage_one(s, a.kernel_id[i], STREAMS ? a.stream[i] : 0, a.start_ns[i], a.end_ns[i]);
  const int64_t qa = a4 >> 2, qb = b4 >> 2;
  if (hi - lo <= kBufEvents) {
    // rounds of kStageD groups of four events per thread with the next
    // round's groups in flight, every step the same memory instructions;
    // staged windows are flushed after every round
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): the head / tail stores above are done
    const int64_t ng = qb - qa;
    const __amdgpu_buffer_rsrc_t rk = buf_rsrc(a.kernel_id + a4, ng * 16), rs = buf_rsrc(a.stream + a4, ng * 16);
    const __amdgpu_buffer_rsrc_t r0 = buf_rsrc(a.start_ns + a4, ng * 32), r1 = buf_rsrc(a.end_ns + a4, ng * 32);
    const __amdgpu_buffer_rsrc_t ro = buf_rsrc(s.out, (int64_t)s.len * (int64_t)sizeof(R));
    v4u bk[kStageD], bs[kStageD], ba0[kStageD], ba1[kStageD], bb0[kStageD], bb1[kStageD];
    auto load = [&](int d, int64_t rq) {
      const uint32_t o16 = rq < ng ? (uint32_t)rq * 16u : kOob, o32 = rq < ng ? (uint32_t)rq * 32u : kOob;
      bk[d] = __builtin_amdgcn_raw_buffer_load_b128(rk, (int)o16, 0, 0);
      bs[d] = STREAMS ? __builtin_amdgcn_raw_buffer_load_b128(rs, (int)o16, 0, 0) : v4u{0u, 0u, 0u, 0u};
      ba0[d] = __builtin_amdgcn_raw_buffer_load_b128(r0, (int)o32, 0, 0);
      ba1[d] = __builtin_amdgcn_raw_buffer_load_b128(r0, (int)(o32 + 16u), 0, 0);
      bb0[d] = __builtin_amdgcn_raw_buffer_load_b128(r1, (int)o32, 0, 0);
      bb1[d] = __builtin_amdgcn_raw_buffer_load_b128(r1, (int)(o32 + 16u), 0, 0);
    };
#pragma unroll
    for (int d = 0; d < kStageD; ++d) load(d, tid + (int64_t)d * kStageThreads);
    for (int64_t rb = 0; rb < ng; rb += (int64_t)kStageD * kStageThreads) {
#pragma unroll
      for (int d = 0; d < kStageD; ++d) {
        const int64_t rq = rb + tid + (int64_t)d * kStageThreads;
        const v4i k4 = __builtin_bit_cast(v4i, bk[d]), s4 = __builtin_bit_cast(v4i, bs[d]);
        const v2l x0 = __builtin_bit_cast(v2l, ba0[d]), x1 = __builtin_bit_cast(v2l, ba1[d]);
        const v2l y0 = __builtin_bit_cast(v2l, bb0[d]), y1 = __builtin_bit_cast(v2l, bb1[d]);
        load(d, rq + (int64_t)kStageD * kStageThreads);
        stage_four_buf(s, ro, rq < ng, k4, s4, x0, x1, y0, y1);
      }
      if (tid == 0) *n_list = 0;
      lds_barrier();
#pragma unroll
      for (int kk = 0; kk < kStageK / kStageThreads; ++kk) stage_plan(s, done, tid + kk * kStageThreads, list, n_list);
      lds_barrier();
      stage_write(s, ro, done, list, *n_list, tid);
      lds_barrier();
    }
  } else {
    if constexpr (sizeof(R) == 8) {
      // segments too long for 32-bit buffer offsets (8-byte records only): the
      // same rounds with global loads and stores
      v4i bk[kStageD], bs[kStageD];
      v2l ba0[kStageD], ba1[kStageD], bb0[kStageD], bb1[kStageD];
#pragma unroll
      for (int d = 0; d < kStageD; ++d) {
        const int64_t q = qa + tid + (int64_t)d * kStageThreads;
        bk[d] = bs[d] = 0;
        ba0[d] = ba1[d] = bb0[d] = bb1[d] = 0;
        if (q < qb) {
          bk[d] = __builtin_nontemporal_load(K4 + q);
          if (STREAMS) bs[d] = __builtin_nontemporal_load(S4 + q);
          ba0[d] = __builtin_nontemporal_load(T0 + 2 * q);
          ba1[d] = __builtin_nontemporal_load(T0 + 2 * q + 1);
          bb0[d] = __builtin_nontemporal_load(T1 + 2 * q);
          bb1[d] = __builtin_nontemporal_load(T1 + 2 * q + 1);
        }
      }
      for (int64_t r0 = qa; r0 < qb; r0 += (int64_t)kStageD * kStageThreads) {
#pragma unroll
        for (int d = 0; d < kStageD; ++d) {
          const int64_t q = r0 + tid + (int64_t)d * kStageThreads;
          const v4i k4 = bk[d], s4 = bs[d];
          const v2l x0 = ba0[d], x1 = ba1[d], y0 = bb0[d], y1 = bb1[d];
          const int64_t qn = q + (int64_t)kStageD * kStageThreads;
          if (qn < qb) {
            bk[d] = __builtin_nontemporal_load(K4 + qn);
            if (STREAMS) bs[d] = __builtin_nontemporal_load(S4 + qn);
            ba0[d] = __builtin_nontemporal_load(T0 + 2 * qn);
            ba1[d] = __builtin_nontemporal_load(T0 + 2 * qn + 1);
            bb0[d] = __builtin_nontemporal_load(T1 + 2 * qn);
            bb1[d] = __builtin_nontemporal_load(T1 + 2 * qn + 1);
          }
          if (q < qb) {
            stage_one(s, k4.x, s4.x, x0.x, y0.x);
            stage_one(s, k4.y, s4.y, x0.y, y0.y);
            stage_one(s, k4.z, s4.z, x1.x, y1.x);
            stage_one(s, k4.w, s4.w, x1.y, y1.y);
          }
        }
        lds_barrier();
        for (int k = tid; k < s.K; k += kStageThreads) stage_flush(s, done, k, false);
        lds_barrier();
      }
    }
  }
  // every staging write and cursor increment of the segment (the head and
  // tail, and the element-wise path, run without a round barrier after them)
  lds_barrier();
  for (int k = tid; k < s.K; k += kStageThreads) stage_flush(s, done, k, true);
}

union StageLds {
  uint64_t w8[kStageK][8];
  uint32_t w4[kStageK][16];
};

__global__ __launch_bounds__(kStageThreads) void kde_scatter_staged_kernel(KdeArgs a) {
  __shared__ StageLds stage;
  __shared__ uint32_t cur[kStageK + 1], done[kStageK + 1];  // + the spare slot
  __shared__ uint32_t wave_tot[kStageThreads / kWave];
  __shared__ uint32_t claim, n_list, wide;
  __shared__ FlushEntry list[kFlushCap];
  const int tid = threadIdx.x, K = a.K;
  const int per = (K + kStageThreads - 1) / kStageThreads;
  while (true) {
    if (tid == 0) {
      claim = atomicAdd(&a.counters[0], 1u);
      wide = 0;
    }
    lds_barrier();
    const uint32_t g = claim;
    if (g >= (uint32_t)a.n_seg) break;
    // cursors = exclusive prefix of the segment's per-kernel counts; any
    // present cell's maximum at or above kW4Lim asks for 8-byte records
    const uint32_t* cnt = a.count + (int64_t)g * K;
    const int64_t* mx = a.max_ns + (int64_t)g * K;
    const int k0 = tid * per, k1 = min(K, k0 + per);
    uint32_t own = 0;
    bool big = false;
    for (int k = k0; k < k1; ++k) {
      const uint32_t n = cnt[k];
      own += n;
      big |= n != 0 && (uint64_t)mx[k] >= kW4Lim;
    }
    const uint32_t incl = wave_incl_scan(own);
    if (lane_id() == kWave - 1) wave_tot[tid / kWave] = incl;
    if (__any(big) && lane_id() == 0) wide = 1;
    lds_barrier();
    uint32_t base = incl - own;
    for (int w = 0; w < tid / kWave; ++w) base += wave_tot[w];
    for (int k = k0; k < k1; ++k) {
      cur[k] = done[k] = base;
      base += cnt[k];
    }
    const int64_t lo = a.seg_off[g], hi = a.seg_off[g + 1];
    const bool bad = !(lo >= 0 && lo <= hi && hi <= a.n_events && hi - lo <= (int64_t)UINT32_MAX);
    const bool w4 = !bad && hi - lo <= kBufEvents && !wide;
    // a segment whose summary counted no invalid event skips the stream array
    const bool streams = !(a.n_invalid && a.n_invalid[g] == 0);
    if (tid == 0) a.seg_w4[g] = w4 ? 1 : 0;
    lds_barrier();
    if (w4) {
      const StageCtx<uint32_t> s{stage.w4, cur, done, reinterpret_cast<uint32_t*>(a.bucket + lo),
                                 (uint32_t)(hi - lo), (uint32_t)((2 * lo) & 15), K, a.NS};
      if (streams) stage_segment<uint32_t, true>(a, s, done, list, &n_list, lo, hi, tid);
      else stage_segment<uint32_t, false>(a, s, done, list, &n_list, lo, hi, tid);
    } else if (!bad) {
      const StageCtx<uint64_t> s{stage.w8, cur, done, a.bucket + lo, (uint32_t)(hi - lo), (uint32_t)(lo & 7), K,
                                 a.NS};
      if (streams) stage_segment<uint64_t, true>(a, s, done, list, &n_list, lo, hi, tid);
      else stage_segment<uint64_t, false>(a, s, done, list, &n_list, lo, hi, tid);
    }
    lds_barrier();
    uint32_t* ends = a.cell_end + (int64_t)g * K;
    for (int k = tid; k < K; k += kStageThreads) ends[k] = cur[k];
    lds_barrier();
  }
}

// -------------------------------------------------------------------- cells

template <int TIER>
struct CellLds {
  static constexpr int W = Tier<TIER>::kWords, CA = Tier<TIER>::kCand;
  // first, so that its LDS address is a multiple of 256 bytes and the weight
  // reads' constant offsets fold into the instructions' offset fields
  alignas(256) uint32_t buf[W];  // grid histogram (then its prefix) | analysis data; later selection data
  uint64_t cval[CA];    // valley depth f
  uint64_t tlb[kMaxT];  // target bin: smallest duration
  uint64_t tub[kMaxT];  // target bin: one past the largest duration
  uint64_t tpre[kMaxT]; // digits selected so far
  uint64_t trank[kMaxT];
  uint32_t tpop[kMaxT];  // durations in the target bin
  uint32_t tdone[kMaxT]; // target already resolved
  uint32_t tcnt[kMaxT];  // durations gathered for the target so far
  int32_t cpos[CA];     // valley grid index
  uint32_t th[64];
};

// One cell's inputs, checked against the bucketed durations.
struct CellMeta {
  uint32_t n;
  uint32_t w4;  // records of 4 bytes (1) or 8 (0)
  int64_t mn, mx;
  int64_t off;  // byte offset of the first duration in the bucket, or -1 when the summary does not match
  double pw;    // n^(-1/5) from the table (0 when n is outside it)
};

typedef unsigned v4u_a4 __attribute__((ext_vector_type(4), aligned(4)));
typedef unsigned long long v2ul __attribute__((ext_vector_type(2)));
typedef unsigned long long v2ul_a8 __attribute__((ext_vector_type(2), aligned(8)));

// A cell's bucketed durations, records of 4 or 8 bytes. Reads take the
// width's own loads (one branch per group of loads, uniform when the
// wavefront works on one cell).
struct Durs {
  const void* p;
  bool w4;
  // v[u] = record i0 + u * stride where that is below n, else dflt
  template <int N>
  __device__ __forceinline__ void get(uint64_t i0, uint32_t stride, uint32_t n, uint64_t (&v)[N],
                                      uint64_t dflt) const {
    if (w4) {
      const uint32_t* q = static_cast<const uint32_t*>(p);
#pragma unroll
      for (int u = 0; u < N; ++u) {
        const uint64_t i = i0 + (uint64_t)u * stride;
        v[u] = i < n ? (uint64_t)q[i] : dflt;
      }
    } else {
      const uint64_t* q = static_cast<const uint64_t*>(p);
#pragma unroll
      for (int u = 0; u < N; ++u) {
        const uint64_t i = i0 + (uint64_t)u * stride;
        v[u] = i < n ? q[i] : dflt;
      }
    }
  }
  // v[u] = record i0 + u (u < 8) where that is below n, else dflt: one lane's
  // run of eight records in 16-byte loads. The loads may reach up to seven
  // records past the cell; those bytes lie inside the workspace (a segment of
  // 4-byte records fills half its area, and the bucket is followed by the
  // cell-end array) and are discarded.
  __device__ __forceinline__ void run8(uint32_t i0, uint32_t n, uint64_t (&v)[8], uint64_t dflt) const {
    if (w4) {
      const v4u_a4* q = reinterpret_cast<const v4u_a4*>(static_cast<const uint32_t*>(p) + i0);
      const v4u x = q[0], y = q[1];
      const uint32_t r[8] = {x.x, x.y, x.z, x.w, y.x, y.y, y.z, y.w};
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = i0 + u < n ? (uint64_t)r[u] : dflt;
    } else {
      const v2ul_a8* q = reinterpret_cast<const v2ul_a8*>(static_cast<const uint64_t*>(p) + i0);
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const v2ul x = q[h];
        v[2 * h] = i0 + 2 * h < n ? (uint64_t)x.x : dflt;
        v[2 * h + 1] = i0 + 2 * h + 1 < n ? (uint64_t)x.y : dflt;
      }
    }
  }
  __device__ __forceinline__ uint64_t nt(uint32_t i) const {  // streaming (nontemporal) read
    return w4 ? (uint64_t)__builtin_nontemporal_load(static_cast<const uint32_t*>(p) + i)
              : __builtin_nontemporal_load(static_cast<const uint64_t*>(p) + i);
  }
};

__device__ __forceinline__ Durs durs_of(const KdeArgs& a, const CellMeta& m) {
  return Durs{reinterpret_cast<const char*>(a.bucket) + m.off, m.w4 != 0};
}

template <int TIER>
__device__ void remove_valley(CellLds<TIER>& L, int idx, int m) {
  const int l = lane_id();
  for (int qb = idx; qb < m - 1; qb += kWave) {
    const int q = qb + l;
    int32_t p = 0;
    uint64_t v = 0;
    if (q < m - 1) {
      p = L.cpos[q + 1];
      v = L.cval[q + 1];
    }
    wave_sync();
    if (q < m - 1) {
      L.cpos[q] = p;
      L.cval[q] = v;
    }
    wave_sync();
  }
}

__device__ void write_empty(const KdeArgs& a, int64_t c) {
  const int l = lane_id();
  if (l < kMaxC) {
    a.cl_count[c * kMaxC + l] = 0;
    a.p50[c * kMaxC + l] = 0;
    a.p99[c * kMaxC + l] = 0;
  }
  if (l == 0) {
    a.n_clusters[c] = 0;
    if (a.bw_q8) a.bw_q8[c] = 0;
  }
}

// Load a small cell's durations into registers (lane l holds l, l + 64, ...).
__device__ __forceinline__ void load_small(const KdeArgs& a, const CellMeta& m, uint64_t (&rv)[kRegVals]) {
  const int l = lane_id();
  const bool small = m.off >= 0 && m.n <= (uint32_t)(kWave * kRegVals);
  const Durs vals = durs_of(a, m);
#pragma unroll
  for (int r = 0; r < kRegVals; ++r) {
    const uint32_t i = (uint32_t)(l + r * kWave);
    rv[r] = small && i < m.n ? vals.nt(i) : 0ull;
  }
}

// Zero padding of the symmetric weight table beyond T: the density loop
// takes occupied grid points by whole histogram chunks of 64 for pairs of
// chunks, so it meets distances up to T + 190.
constexpr int kWPad = 192;  // >= 190 (see density_pair)
constexpr int kListPad = 32;  // readable pairs past the list's end (a step reads 8)
static_assert((2 * kListPad + kWPad) % 64 == 0 && kListPad >= 8 && kWPad >= 190, "weight table layout");

// f(j) = sum_b c(b) w(|j - b|) for this lane's grid points j = jb + lane
// (fa) and j + 64 (fb), in registers, over the occupied grid points
// list[k0, k1) (pairs (4 b, c(b)), read with wavefront-uniform addresses): one
// pass over the list serves both 64-point chunks. ws is the symmetric weight
// table, ws[d] = w(|d|), zero from T + 1 to T + kWPad; the list range is
// whole 64-point chunks covering the reach of both, [jb - T, jb + 127 + T],
// so it starts at most 63 points lower and ends at most 63 higher, and every
// |j - b| and |j + 64 - b| read is at most T + 190. Eight points per step, so sixteen
// weight reads are in flight; the list holds kListPad readable pairs past its
// end. Acc = uint32_t is exact while the cell has fewer than 65,536
// durations (f <= 65536 n) and multiplies in 24 bits (c < 2^24, w <= 2^16).
template <typename Acc>
__device__ __forceinline__ void density_pair(const uint32_t* ws, const uint2* list, int k0, int k1, int jb, Acc& fa,
                                             Acc& fb) {
  const int j = jb + lane_id();
  const char* wj = reinterpret_cast<const char*>(ws + j);
  fa = fb = 0;
  auto step = [&](int k, bool tail) {
    uint32_t cb[8], wa[8], wb[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint2 e = list[k + u];  // (4 b, c(b)): the byte offset of ws[j - b] below ws + j
      const bool in = !tail || k + u < k1;  // wavefront-uniform
      cb[u] = in ? e.y : 0u;
      const uint32_t ob = in ? e.x : 4u * (uint32_t)j;
      wa[u] = *reinterpret_cast<const uint32_t*>(wj - ob);
      wb[u] = *reinterpret_cast<const uint32_t*>(wj + 4 * kWave - ob);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if constexpr (sizeof(Acc) == 4) {
        fa += __umul24(cb[u], wa[u]);
        fb += __umul24(cb[u], wb[u]);
      } else {
        fa += (uint64_t)cb[u] * wa[u];
        fb += (uint64_t)cb[u] * wb[u];
      }
    }
  };
  // whole steps of eight listed points need no bounds test; one tail step
  int k = k0;
  for (; k + 8 <= k1; k += 8) step(k, false);
  if (k < k1) step(k, true);
}

// Rank of this lane's element e (lane < k) among list[0, k) in ascending
// order, ties broken by position; list has 64 readable slots.
__device__ __forceinline__ uint32_t rank_in_list(const uint64_t* list, int k, uint64_t e) {
  const int l = lane_id();
  uint32_t rank = 0;
  for (int j0 = 0; j0 < k; j0 += 8) {
    uint64_t ej[8];  // eight reads in flight
#pragma unroll
    for (int u = 0; u < 8; ++u) ej[u] = list[j0 + u];
#pragma unroll
    for (int u = 0; u < 8; ++u) rank += (j0 + u < k && (ej[u] < e || (ej[u] == e && j0 + u < l))) ? 1u : 0u;
  }
  return rank;
}

// Steps 2 - 8 on one wavefront, the grid histogram of the cell being in
// L.buf[0, G): bandwidth, density, valleys, filters, cap, per-cluster counts
// and the selection targets (L.tlb / tub / trank / tpop, L.tpre = 0).
// Returns false when the cell needs a larger tier (only for TIER < 2).
struct Analysis {
  int ncl, NT;
  int64_t H;
  uint32_t ccount[kMaxC];
};

template <int TIER>
__device__ bool kde_analyze(const KdeArgs& a, CellLds<TIER>& L, const CellMeta& cm, int lo, int G, Analysis& res) {
  constexpr int WORDS = CellLds<TIER>::W, CAND = CellLds<TIER>::CA;
  const int l = lane_id();
  const uint32_t n = cm.n;
  const int sh = 6 - a.sub_bits;
  uint32_t* cgrid = L.buf;
  // 2. bandwidth from the exact first and second moments of the grid index;
  // the occupied grid points are listed on the way, in ascending order, as
  // (4 b, c(b)) pairs, with cs[i] = pairs before histogram chunk i. LDS words:
  // [0, G) histogram | cs | list (+ kListPad pairs) | weight table; 2 kListPad + kWPad
  // is a multiple of 64 words, so the weight reads' constant part is a multiple of
  // 256 bytes and folds into the instructions' offsets
  const int NCH = (G + kWave - 1) / kWave + 1;
  uint32_t* cs = L.buf + G;
  const int lofs = (G + NCH + 1) & ~1;
  uint2* list = reinterpret_cast<uint2*>(L.buf + lofs);
  uint64_t s1 = 0, s2 = 0;
  int nnz = 0;
  for (int jb = 0, ch = 0; jb < G; jb += kWave, ++ch) {
    const int j = jb + l;
    const uint32_t k = j < G ? cgrid[j] : 0u;
    s1 += (uint64_t)k * (uint64_t)j;
    s2 += (uint64_t)k * (uint64_t)j * (uint64_t)j;
    const uint64_t occ = __ballot(k != 0);
    if (l == 0) cs[ch] = (uint32_t)nnz;
    if (k != 0) {
      const int idx = nnz + __popcll(occ & ((1ull << l) - 1ull));
      if (TIER == 2 || lofs + 2 * idx + 1 < WORDS) list[idx] = make_uint2(4u * (uint32_t)j, k);  // (4 b, c(b))
    }
    nnz += __popcll(occ);
  }
  if (l == 0) cs[NCH - 1] = (uint32_t)nnz;
  const int tofs = lofs + 2 * (nnz + kListPad);
  if (TIER < 2 && tofs > WORDS) return false;
  s1 = wave_sum_u64(s1);
  s2 = wave_sum_u64(s2);
  int64_t H = 0;
  if (n >= 2) {
    // n * s2 - s1^2 exactly: in 64 bits when it fits (the usual case), else 128
    uint64_t ns2;
    double vnum;
    if (!__builtin_mul_overflow((uint64_t)n, s2, &ns2) && s1 < (1ull << 32)) vnum = (double)(ns2 - s1 * s1);
    else vnum = u128_to_f64((unsigned __int128)n * s2 - (unsigned __int128)s1 * s1);
    const double var = vnum / ((double)n * (double)(n - 1));
    double pw = cm.pw;
    if (n >= (uint32_t)kPowTab) {
      // tier 0 is routed fewer than 2,048 durations; should a larger cell come
      // here, it goes on to tier 1 rather than carry the exact root's
      // registers in the hottest kernel
      if (TIER == 0) return false;
      pw = kde_pw(n);
    }
    H = kde_bw_q8(var, pw);
  }

  // 3-4. weights, density and valleys
  int m = 0;
  if (H > 0 && G >= 3) {
    // weights straight into the symmetric table ws[-C .. C]: w(t) rounds to
    // 0 once 32768 t^2 / H^2 > ln(131072), i.e. t > 0.018963 H, so every
    // nonzero weight has t <= Tb = floor(0.019 H) + 2 (and t < G)
    const int64_t Tb = (H * 19) / 1000 + 2;
    const int C = (Tb < (int64_t)G - 1 ? (int)Tb : G - 1) + kWPad;
    if (TIER < 2 && tofs + 2 * C + 1 > WORDS) return false;
    uint32_t* ws = L.buf + tofs + C;
    const double H2 = (double)(H * H);
    int T = -1;
    bool past = false;  // a chunk with a zero weight has been seen: the rest are zero
    for (int tb = 0; tb <= C; tb += kWave) {
      const int t = tb + l;
      uint32_t wt = 0;
      if (!past && t < G) wt = kde_weight(t, H2);
      const int cnt = __popcll(__ballot(wt != 0));  // weights are non-increasing in t
      if (!past) T = tb + cnt - 1;
      past = past || cnt < kWave;
      if (t <= C) {
        ws[t] = wt;
        ws[-t] = wt;
      }
    }
    wave_sync();
    int carry_start = -1, carry_drop = 0;
    uint64_t prev_last = 0;
    for (int jp = 0; jp < G; jp += 2 * kWave) {
      // densities of the chunks at jp and jp + 64 in one pass over the list
      const int kb0 = (jp - T > 0 ? jp - T : 0) / kWave;
      const int kb1 = (jp + 2 * kWave - 1 + T < G - 1 ? jp + 2 * kWave - 1 + T : G - 1) / kWave;
      const int k0 = (int)__builtin_amdgcn_readfirstlane(cs[kb0]), k1 = (int)__builtin_amdgcn_readfirstlane(cs[kb1 + 1]);
      uint64_t fpair[2];
      if (n < 65536u) {
        uint32_t fa, fb;
        density_pair<uint32_t>(ws, list, k0, k1, jp, fa, fb);
        fpair[0] = fa;
        fpair[1] = fb;
      } else {
        density_pair<uint64_t>(ws, list, k0, k1, jp, fpair[0], fpair[1]);
      }
      // valleys chunk by chunk, in grid order
      for (int h = 0; h < 2; ++h) {
        const int jb = jp + h * kWave;
        if (jb >= G) break;
        const int j = jb + l;
        const bool valid = j < G;
        uint64_t fj = valid ? fpair[h] : 0ull;
        uint64_t fl = __shfl_up(fj, 1, kWave);
        if (l == 0) fl = prev_last;
        const bool start = valid && (j == 0 || fj != fl);
        const bool drop = start && j > 0 && fl > fj;
        const bool rise = start && j > 0 && fl < fj;
        const uint64_t S = __ballot(start), D = __ballot(drop);
        int a_idx = carry_start, a_drop = carry_drop;
        const uint64_t below = S & ((1ull << l) - 1ull);
        if (below) {
          const int al = 63 - __builtin_clzll(below);
          a_idx = jb + al;
          a_drop = (int)((D >> al) & 1ull);
        }
        const bool is_valley = rise && a_drop;
        const uint64_t Vb = __ballot(is_valley);
        if (is_valley) {
          const int idx = m + __popcll(Vb & ((1ull << l) - 1ull));
          if (idx < CAND) {
            L.cpos[idx] = (a_idx + j - 1) / 2;
            L.cval[idx] = fl;
          }
        }
        m += __popcll(Vb);
        if (TIER < 2 && m > CAND) return false;
        if (S) {
          const int ls = 63 - __builtin_clzll(S);
          carry_start = jb + ls;
          carry_drop = (int)((D >> ls) & 1ull);
        }
        const int last = G - 1 - jb < kWave - 1 ? G - 1 - jb : kWave - 1;
        prev_last = readlane64(fj, last);
      }
    }
    if (m > CAND) m = CAND;  // cannot happen in tier 2: a grid of G points has < G / 2 valleys
    wave_sync();
  }

  // grid histogram -> inclusive prefix counts (in place)
  {
    uint32_t carry = 0;
    for (int jb = 0; jb < G; jb += kWave) {
      const int j = jb + l;
      const uint32_t v = j < G ? cgrid[j] : 0u;
      const uint32_t incl = wave_incl_scan(v) + carry;
      if (j < G) cgrid[j] = incl;
      carry = __builtin_amdgcn_readlane(incl, kWave - 1);
    }
    wave_sync();
  }
  const uint32_t* P = cgrid;
  auto bound = [&](int q, int mm) -> int { return q < mm ? L.cpos[q] : G - 1; };

  // 5. cluster-level filter
  uint64_t need = ((uint64_t)a.frac_pm * n + 999u) / 1000u;
  if (need < (uint64_t)a.min_count) need = (uint64_t)a.min_count;
  while (m > 0) {
    uint64_t best = ~0ull;  // size * 4096 + q: smallest size, then lowest q
    for (int qb = 0; qb <= m; qb += kWave) {
      const int q = qb + l;
      if (q <= m) {
        const uint64_t hiP = P[bound(q, m)];
        const uint64_t loP = q > 0 ? P[L.cpos[q - 1]] : 0;
        const uint64_t key = ((hiP - loP) << 12) | (uint64_t)q;
        best = key < best ? key : best;
      }
    }
    best = wave_min_u64(best);
    if ((best >> 12) >= need) break;
    const int q = (int)(best & 4095u);
    int idx;
    if (q == 0) idx = 0;
    else if (q == m) idx = m - 1;
    else idx = L.cval[q - 1] > L.cval[q] ? q - 1 : q;
    remove_valley(L, idx, m);
    --m;
  }

  // 6. spacing filter over [0, valleys..., G - 1]
  while (m > 0) {
    int hit = -1;
    for (int qb = 0; qb <= m && hit < 0; qb += kWave) {
      const int q = qb + l;
      bool close = false;
      if (q <= m) {
        const int lo_b = q > 0 ? L.cpos[q - 1] : 0;
        close = bound(q, m) - lo_b < a.gap;
      }
      const uint64_t bm = __ballot(close);
      if (bm) hit = qb + __builtin_ctzll(bm);
    }
    if (hit < 0) break;
    int idx;
    if (hit == 0) idx = 0;
    else if (hit == m) idx = m - 1;
    else idx = L.cval[hit - 1] > L.cval[hit] ? hit - 1 : hit;
    remove_valley(L, idx, m);
    --m;
  }

  // 7. cluster cap: drop the largest-f valley (the upper one on ties)
  while (m > kMaxC - 1) {
    uint64_t best_v = 0;
    int best_q = -1;
    for (int qb = 0; qb < m; qb += kWave) {
      const int q = qb + l;
      const bool on = q < m;
      const uint64_t v = on ? L.cval[q] : 0ull;
      const uint64_t mv = wave_max_u64(v);
      const uint64_t bm = __ballot(on && v == mv);
      if (bm && (best_q < 0 || mv >= best_v)) {
        best_v = mv;
        best_q = qb + 63 - __builtin_clzll(bm);
      }
    }
    remove_valley(L, best_q, m);
    --m;
  }

  // 8. counts and selection targets (ranks in the cell's sorted order):
  // cluster q holds the ranks [hiP(q - 1), hiP(q)) of the sorted durations
  const int ncl = m + 1, NT = 2 * ncl;
  uint64_t hiP[kMaxC], tr[kMaxT];
  uint32_t ccount[kMaxC];
#pragma unroll
  for (int q = 0; q < kMaxC; ++q) hiP[q] = q < ncl ? (uint64_t)P[bound(q, m)] : 0ull;
#pragma unroll
  for (int q = 0; q < kMaxC; ++q) {
    const uint64_t before = q > 0 ? hiP[q - 1] : 0ull;
    const uint64_t size = q < ncl ? hiP[q] - before : 1ull;  // >= 1 for a kept cluster (min_count >= 1)
    ccount[q] = q < ncl ? (uint32_t)size : 0u;
    tr[2 * q] = before + (size - 1) / 2;
    tr[2 * q + 1] = before + (99 * size + 99) / 100 - 1;
  }
  // target grid bin: the smallest j with P[j] > rank (P is non-decreasing
  // and P[G - 1] = n exceeds every rank), one ballot per target and chunk
  int tj[kMaxT];
#pragma unroll
  for (int t = 0; t < kMaxT; ++t) tj[t] = G - 1;
  uint32_t open = (1u << NT) - 1u;
  for (int jb = 0; jb < G && open; jb += kWave) {
    const int j = jb + l;
    const uint64_t pj = j < G ? (uint64_t)P[j] : ~0ull;
#pragma unroll
    for (int t = 0; t < kMaxT; ++t) {
      if ((open >> t) & 1u) {
        const uint64_t bm = __ballot(pj > tr[t]);
        if (bm) {
          tj[t] = jb + __builtin_ctzll(bm);
          open &= ~(1u << t);
        }
      }
    }
  }
  {
    int j = 0;
    uint64_t r = 0;
#pragma unroll
    for (int t = 0; t < kMaxT; ++t)
      if (t == l) {
        j = tj[t];
        r = tr[t];
      }
    if (l < NT) {
      const uint64_t below = j > 0 ? P[j - 1] : 0;
      L.tlb[l] = grid64_lb((lo + j) << sh, L.th);
      L.tub[l] = grid64_lb((lo + j + 1) << sh, L.th);
      L.tpre[l] = 0;
      L.trank[l] = r - below;
      L.tpop[l] = P[j] - below;
    }
  }
  wave_sync();

  res.ncl = ncl;
  res.NT = NT;
  res.H = H;
#pragma unroll
  for (int q = 0; q < kMaxC; ++q) res.ccount[q] = ccount[q];
  return true;
}

// One cell on one wavefront. Returns false when the cell needs a larger
// tier (only for TIER < 2; nothing has been written for it then).
template <int TIER>
__device__ bool kde_one_cell(const KdeArgs& a, CellLds<TIER>& L, int64_t c, const CellMeta& cm,
                             const uint64_t (&rv)[kRegVals]) {
  constexpr int WORDS = CellLds<TIER>::W;
  const int l = lane_id();
  const uint32_t n = cm.n;
  const Durs vals = durs_of(a, cm);
  const int sh = 6 - a.sub_bits;
  const int lo = grid64((uint64_t)cm.mn, L.th) >> sh;
  const int G = (grid64((uint64_t)cm.mx, L.th) >> sh) - lo + 1;
  if (TIER < 2 && G > WORDS) return false;
  uint32_t* cgrid = L.buf;
  const bool in_regs = n <= (uint32_t)(kWave * kRegVals);

  // 1. grid histogram
  for (int j = l; j < G; j += kWave) cgrid[j] = 0;
  wave_sync();
  bool out_of_range = false;
  // 4-byte records (the cell's flag is wavefront-uniform): grid indices
  // from 32-bit operations
  auto add = [&](int x) {
    if (x >= 0 && x < G) atomicAdd(&cgrid[x], 1u);
    else out_of_range = true;
  };
  if (in_regs) {
    if (vals.w4) {
#pragma unroll
      for (int r = 0; r < kRegVals; ++r)
        if ((uint32_t)(l + r * kWave) < n) add((grid32((uint32_t)rv[r], L.th) >> sh) - lo);
    } else {
#pragma unroll
      for (int r = 0; r < kRegVals; ++r)
        if ((uint32_t)(l + r * kWave) < n) add((grid64(rv[r], L.th) >> sh) - lo);
    }
  } else {
    // four loads in flight per lane
    for (uint64_t i0 = l; i0 < n; i0 += 4 * kWave) {
      uint64_t v[4];
      vals.get(i0, kWave, n, v, 0ull);
      if (vals.w4) {
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (i0 + u * kWave < n) add((grid32((uint32_t)v[u], L.th) >> sh) - lo);
      } else {
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (i0 + u * kWave < n) add((grid64(v[u], L.th) >> sh) - lo);
      }
    }
  }
  wave_sync();
  if (__any(out_of_range)) {  // durations outside the summarized [min, max]
    if (l == 0) flag(a, ARGUS_DEV_KDE_SUMMARY);
    write_empty(a, c);
    return true;
  }

  Analysis an;
  if (!kde_analyze<TIER>(a, L, cm, lo, G, an)) return false;
  const int ncl = an.ncl, NT = an.NT;
  const int64_t H = an.H;
  uint32_t ccount[kMaxC];
#pragma unroll
  for (int q = 0; q < kMaxC; ++q) ccount[q] = an.ccount[q];

  // 9a. a target bin with at most 64 durations is gathered into LDS (from
  // registers, or in one pass over the cell's durations for all such targets
  // at once) and its element of the wanted rank found by counting
  {
    int ndirect = 0;
    for (int t = 0; t < NT; ++t) ndirect += L.tpop[t] <= (uint32_t)kWave ? 1 : 0;
    if (l < kMaxT) {
      L.tdone[l] = 0;
      L.tcnt[l] = 0;
    }
    wave_sync();
    if (ndirect > 0) {
      uint64_t* lists = reinterpret_cast<uint64_t*>(L.buf);  // kMaxT lists of kWave durations
      // four durations of the lane against each target in turn: a target's
      // (wavefront-uniform) bin is read from LDS once per four durations
      auto gather4 = [&](const uint64_t (&v)[4], const bool (&ok)[4]) {
        for (int t = 0; t < NT; ++t) {
          if (L.tpop[t] > (uint32_t)kWave) continue;
          const uint64_t lb = L.tlb[t], ub = L.tub[t];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            if (ok[u] && v[u] >= lb && v[u] < ub) {
              const uint32_t slot = atomicAdd(&L.tcnt[t], 1u);
              if (slot < (uint32_t)kWave) lists[t * kWave + slot] = v[u];
            }
          }
        }
      };
      if (in_regs) {
        bool ok[4];
#pragma unroll
        for (int r = 0; r < kRegVals; ++r) ok[r] = (uint32_t)(l + r * kWave) < n;
        gather4(rv, ok);
      } else {
        for (uint64_t i0 = l; i0 < n; i0 += 4 * kWave) {
          uint64_t v[4];
          bool ok[4];
          vals.get(i0, kWave, n, v, 0ull);
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            ok[u] = i0 + u * kWave < n;
          }
          gather4(v, ok);
        }
      }
      wave_sync();
      for (int t = 0; t < NT; ++t) {
        if (L.tpop[t] > (uint32_t)kWave) continue;
        const int k = (int)L.tpop[t];
        const uint64_t* list = lists + t * kWave;
        const uint64_t e = l < k ? list[l] : 0ull;
        uint32_t rank = 0;
        if (k <= 16) {
          // few elements: compare against each one read from its lane
          for (int i = 0; i < k; ++i) {
            const uint64_t ei = readlane64(e, i);
            rank += (ei < e || (ei == e && i < l)) ? 1u : 0u;
          }
        } else {
          rank = rank_in_list(list, k, e);
        }
        const uint64_t hit = __ballot(l < k && (uint64_t)rank == L.trank[t]);
        const uint64_t val = readlane64(e, hit ? __builtin_ctzll(hit) : 0);
        if (l == 0) {
          L.tpre[t] = val - L.tlb[t];
          L.tdone[t] = 1;
        }
      }
      wave_sync();
    }
  }

  // 9b. exact selection inside the remaining target bins, kDigit bits per pass
  int nbits = 0;
  for (int t = 0; t < NT; ++t) {
    if (L.tdone[t]) continue;
    const uint64_t width = L.tub[t] - L.tlb[t];
    const int b = width > 1 ? 64 - __builtin_clzll(width - 1) : 0;
    nbits = b > nbits ? b : nbits;
  }
  const int npass = (nbits + kDigit - 1) / kDigit;
  constexpr int R = 1 << kDigit;
  uint32_t* hist = L.buf;  // NT x R counters; the prefix counts are no longer needed
  for (int p = 0; p < npass; ++p) {
    const int shift = kDigit * (npass - 1 - p);
    for (int i = l; i < NT * R; i += kWave) hist[i] = 0;
    wave_sync();
    // as in 9a: four durations against each open target in turn
    auto consider4 = [&](const uint64_t (&v)[4], const bool (&ok)[4]) {
      for (int t = 0; t < NT; ++t) {
        if (L.tdone[t]) continue;
        const uint64_t lb = L.tlb[t], ub = L.tub[t], pre = L.tpre[t];
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          if (ok[w] && v[w] >= lb && v[w] < ub) {
            const uint64_t u = v[w] - lb;
            const uint64_t hi_part = shift + kDigit >= 64 ? 0 : u >> (shift + kDigit);
            if (hi_part == pre) atomicAdd(&hist[t * R + (int)((u >> shift) & (R - 1))], 1u);
          }
        }
      }
    };
    if (in_regs) {
      bool ok[4];
#pragma unroll
      for (int r = 0; r < kRegVals; ++r) ok[r] = (uint32_t)(l + r * kWave) < n;
      consider4(rv, ok);
    } else {
      for (uint64_t i0 = l; i0 < n; i0 += 4 * kWave) {
        uint64_t v[4];
        bool ok[4];
        vals.get(i0, kWave, n, v, 0ull);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          ok[u] = i0 + u * kWave < n;
        }
        consider4(v, ok);
      }
    }
    wave_sync();
    for (int t = 0; t < NT; ++t) {
      if (L.tdone[t]) continue;
      // the digit holding the target rank: one counter per lane, a wave scan
      const uint32_t v = hist[t * R + l];
      const uint32_t incl = wave_incl_scan(v);
      const uint64_t r = L.trank[t];
      const uint64_t bm = __ballot((uint64_t)(incl - v) <= r && r < (uint64_t)incl);
      const int owner = bm ? __builtin_ctzll(bm) : 0;
      const uint32_t excl = __builtin_amdgcn_readlane(incl - v, owner);
      if (l == 0) {
        L.trank[t] = r - excl;
        L.tpre[t] = (L.tpre[t] << kDigit) | (uint64_t)owner;
      }
      wave_sync();
    }
  }

  // outputs
  if (l < kMaxC) {
    const int64_t o = c * kMaxC + l;
    uint32_t cnt = 0;
#pragma unroll
    for (int q = 0; q < kMaxC; ++q)
      if (q == l) cnt = ccount[q];
    a.cl_count[o] = l < ncl ? cnt : 0u;
    a.p50[o] = l < ncl ? (int64_t)(L.tlb[2 * l] + L.tpre[2 * l]) : 0;
    a.p99[o] = l < ncl ? (int64_t)(L.tlb[2 * l + 1] + L.tpre[2 * l + 1]) : 0;
  }
  if (l == 0) {
    a.n_clusters[c] = (uint8_t)ncl;
    if (a.bw_q8) a.bw_q8[c] = (int32_t)H;
  }
  wave_sync();
  return true;
}

// Summary of cell c checked against the bucketed durations (cell_end chain).
__device__ CellMeta load_meta(const KdeArgs& a, int64_t c) {
  CellMeta m{};
  m.off = -1;
  m.n = a.count[c];
  if (m.n == 0) return m;
  m.mn = a.min_ns[c];
  m.mx = a.max_ns[c];
  const uint32_t end = a.cell_end[c];
  const uint32_t prev = c % a.K ? a.cell_end[c - 1] : 0u;
  const int64_t g = c / a.K;
  const int64_t lo = a.seg_off[g], hi = a.seg_off[g + 1];
  const bool seg_ok = lo >= 0 && lo <= hi && hi <= a.n_events && hi - lo <= (int64_t)UINT32_MAX;
  m.w4 = a.seg_w4[g];
  if (seg_ok && end >= m.n && end - m.n == prev && (int64_t)end <= hi - lo && m.mn >= 0 && m.mn <= m.mx)
    m.off = 8 * lo + (int64_t)(end - m.n) * (m.w4 ? 4 : 8);
  m.pw = m.n < (uint32_t)kPowTab ? g_kde_pow[m.n] : 0.0;
  return m;
}

__device__ CellMeta meta_from_lane(const CellMeta& m, int i) {
  CellMeta r;
  r.n = __builtin_amdgcn_readlane(m.n, i);
  r.w4 = __builtin_amdgcn_readlane(m.w4, i);
  r.mn = (int64_t)readlane64((uint64_t)m.mn, i);
  r.mx = (int64_t)readlane64((uint64_t)m.mx, i);
  r.off = (int64_t)readlane64((uint64_t)m.off, i);
  r.pw = readlane_f64(m.pw, i);
  return r;
}

template <int TIER>
__device__ void finish_or_hand_on(const KdeArgs& a, CellLds<TIER>& L, int64_t c, const CellMeta& m,
                                  const uint64_t (&rv)[kRegVals]) {
  const int l = lane_id();
  if (m.n == 0) {
    write_empty(a, c);
    return;
  }
  if (m.off < 0) {
    if (l == 0) flag(a, ARGUS_DEV_KDE_SUMMARY);
    write_empty(a, c);
    return;
  }
  if (!kde_one_cell<TIER>(a, L, c, m, rv)) {
    if (TIER == 0 && l == 0) a.list1[atomicAdd(&a.counters[2], 1u)] = (uint32_t)c;
    if (TIER == 1 && l == 0) a.list2[atomicAdd(&a.counters[4], 1u)] = (uint32_t)c;
    wave_sync();
  }
}

template <int TIER>
__global__ __launch_bounds__(kWave, TIER == 0 ? 4 : 1) void kde_cell_kernel(KdeArgs a) {
  __shared__ CellLds<TIER> L;
  const int l = lane_id();
  L.th[l] = a.theta[l];
  wave_sync();
  while (true) {
    uint32_t claim = 0;
    if (l == 0) claim = atomicAdd(&a.counters[TIER == 0 ? 1 : (TIER == 1 ? 3 : 5)], 1u);
    claim = __builtin_amdgcn_readfirstlane(claim);
    if constexpr (TIER == 0) {
      const uint32_t len0 = __builtin_amdgcn_readfirstlane(
          __hip_atomic_load(&a.counters[7], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      const int64_t i0 = (int64_t)claim * kWave;
      if (i0 >= (int64_t)len0) break;
      const int ncells = (int64_t)len0 - i0 < kWave ? (int)((int64_t)len0 - i0) : kWave;
      // every lane fetches one listed cell's summary; the wave then walks the
      // cells, loading the next small cell's durations while it works on this one
      CellMeta mine{};
      mine.off = -1;
      int64_t cell = 0;
      if (l < ncells) {
        cell = a.list2[i0 + l];
        mine = load_meta(a, cell);
      }
      // cur is only ever a copy of nxt, taken once its loads are complete,
      // and the first cell's loads are waited for right away: at the loop
      // head no load is pending into cur on either path, so the next cell's
      // loads stay in flight while this one is processed
      uint64_t cur[kRegVals], nxt[kRegVals];
      CellMeta mn = meta_from_lane(mine, 0);
      load_small(a, mn, nxt);
      __builtin_amdgcn_s_waitcnt(0);
      for (int i = 0; i < ncells; ++i) {
        const CellMeta m = mn;
#pragma unroll
        for (int r = 0; r < kRegVals; ++r) cur[r] = nxt[r];
        mn = CellMeta{};
        mn.off = -1;
        if (i + 1 < ncells) mn = meta_from_lane(mine, i + 1);
        load_small(a, mn, nxt);
        finish_or_hand_on<TIER>(a, L, (int64_t)readlane64((uint64_t)cell, i), m, cur);
      }
    } else {
      const uint32_t len = __builtin_amdgcn_readfirstlane(
          __hip_atomic_load(&a.counters[TIER == 1 ? 2 : 4], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
      if (claim >= len) break;
      const int64_t c = (TIER == 1 ? a.list1 : a.list2)[claim];
      CellMeta mine{};
      mine.off = -1;
      if (l == 0) mine = load_meta(a, c);
      const CellMeta m = meta_from_lane(mine, 0);
      uint64_t cur[kRegVals];
      load_small(a, m, cur);
      finish_or_hand_on<TIER>(a, L, c, m, cur);
    }
  }
}

// --------------------------------------------------------- workgroup tier
// Cells of at least kBlockMin durations, one two-wavefront workgroup per
// cell: both wavefronts stream the durations (kBlockDepth loads in flight
// per lane) into the LDS grid histogram, wavefront 0 runs the analysis, and
// the p50 / p99 targets are then resolved by selection passes in which both
// stream the durations once more. Each target owns a region of kSelRegion
// LDS words per pass: a histogram of the next kSelDigit bits of its
// candidate range while more than kSelCap durations remain in it, else the
// list of those durations, whose element of the wanted rank is found by
// counting. Wavefront w resolves targets w, w + 2, ... after each pass.
// Cells whose grid or valleys do not fit go to tier 1 unchanged. While
// wavefront 0 analyses a cell its partner waits, so the workgroup is kept
// small: eight workgroups share a CU (LDS bound), and their streaming passes
// fill the time (workgroups of 512 / 256 threads: 20.6 / 15.6 ms on the
// cluster step, 128: 13.6 ms).
constexpr int kBlockThreads = 128;
constexpr int kBlockWaves = kBlockThreads / kWave;
constexpr int kBlockDepth = 8;  // duration loads in flight per thread in the streaming passes
constexpr uint32_t kBlockMin = 2048;
constexpr int kSelRegion = 512;                      // words per target, within the tier-1 grid words
constexpr int kSelDigit = 9;                         // log2(kSelRegion)
constexpr int kSelCap = 64;        // gathered durations per target (8-byte entries)
constexpr int kSelCap32 = 256;     // gathered offsets per target (4-byte entries, bins narrower than 2^32)
static_assert(kMaxT % kBlockWaves == 0, "selection targets shared out over the wavefronts");
static_assert((1 << kSelDigit) == kSelRegion && 2 * kSelCap <= kSelRegion && kMaxT * kSelRegion <= Tier<1>::kWords,
              "selection regions");
static_assert(kSelCap32 + 256 <= kSelRegion && kSelCap32 == 4 * kWave, "offset list and its digit histogram");

// Element of rank r among the k <= kSelCap32 offsets of list (one wavefront,
// four entries per lane): MSD radix selection with 8-bit digits over the
// nb-bit offsets, the digit histogram in hist (256 words). Sets ok = false
// when r >= k.
__device__ __forceinline__ uint32_t select_offsets(const uint32_t* list, uint32_t* hist, int k, int nb, uint64_t r,
                                                   bool& ok) {
  const int l = lane_id();
  ok = r < (uint64_t)k;
  uint32_t e[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) e[j] = l + kWave * j < k ? list[l + kWave * j] : 0u;
  uint32_t prefix = 0, rr = ok ? (uint32_t)r : 0u;
  for (int sh = ((nb + 7) / 8 - 1) * 8; sh >= 0; sh -= 8) {
#pragma unroll
    for (int j = 0; j < 4; ++j) hist[l + kWave * j] = 0;
    wave_sync();
#pragma unroll
    for (int j = 0; j < 4; ++j)
      if (l + kWave * j < k && (sh + 8 >= 32 || (e[j] >> (sh + 8)) == (prefix >> (sh + 8))))
        atomicAdd(&hist[(e[j] >> sh) & 255u], 1u);
    wave_sync();
    const uint4 hv = reinterpret_cast<const uint4*>(hist)[l];  // bins 4l .. 4l + 3
    const uint32_t sum = hv.x + hv.y + hv.z + hv.w;
    const uint32_t incl = wave_incl_scan(sum), excl = incl - sum;
    const uint64_t bm = __ballot(excl <= rr && rr < incl);
    const int owner = bm ? __builtin_ctzll(bm) : 0;
    uint32_t d = 0, x = rr - excl;
    if (x >= hv.x) {
      x -= hv.x;
      d = 1;
      if (x >= hv.y) {
        x -= hv.y;
        d = 2;
        if (x >= hv.z) {
          x -= hv.z;
          d = 3;
        }
      }
    }
    const uint32_t digit = 4u * (uint32_t)owner + __builtin_amdgcn_readlane(d, owner);
    rr = __builtin_amdgcn_readlane(x, owner);
    prefix |= digit << sh;
    wave_sync();
  }
  return prefix;
}

__global__ __launch_bounds__(kBlockThreads, 4) void kde_block_kernel(KdeArgs a) {
  __shared__ CellLds<1> L;
  __shared__ uint32_t s_claim, s_nt, s_ok, s_bad;
  const int tid = threadIdx.x, l = lane_id(), wv = tid / kWave;
  if (tid < 64) L.th[tid] = a.theta[tid];
  const int64_t cells = (int64_t)a.n_seg * a.K;
  const uint32_t n_heavy = __hip_atomic_load(&a.counters[11], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int sh = 6 - a.sub_bits;
  uint32_t* cgrid = L.buf;
  while (true) {
    if (tid == 0) {
      s_claim = atomicAdd(&a.counters[10], 1u);
      s_bad = 0;
    }
    __syncthreads();
    const uint32_t claim = __builtin_amdgcn_readfirstlane(s_claim);
    if (claim >= n_heavy) break;
    const int64_t c = (int64_t)__builtin_amdgcn_readfirstlane(a.list2[cells - 1 - (int64_t)claim]);
    const CellMeta cm = load_meta(a, c);  // checked when the cell was listed: off >= 0, n >= kBlockMin
    const uint64_t n = cm.n;
    const Durs vals = durs_of(a, cm);
    const int lo = grid64((uint64_t)cm.mn, L.th) >> sh;
    const int G = (grid64((uint64_t)cm.mx, L.th) >> sh) - lo + 1;
    if (G > Tier<1>::kWords) {
      if (tid == 0) a.list1[atomicAdd(&a.counters[2], 1u)] = (uint32_t)c;
      __syncthreads();
      continue;
    }

    // 1. grid histogram, all wavefronts
    for (int j = tid; j < G; j += kBlockThreads) cgrid[j] = 0;
    __syncthreads();
    bool out_of_range = false;
    if (vals.w4) {
      // 4-byte records: 32-bit loads and grid indices
      const uint32_t* q = static_cast<const uint32_t*>(vals.p);
      const uint32_t n32 = (uint32_t)n;
      for (uint32_t i0 = (uint32_t)tid; i0 < n32; i0 += kBlockDepth * kBlockThreads) {
        uint32_t v[kBlockDepth];
#pragma unroll
        for (int u = 0; u < kBlockDepth; ++u) {
          const uint32_t i = i0 + (uint32_t)(u * kBlockThreads);
          v[u] = i < n32 ? q[i] : 0u;
        }
#pragma unroll
        for (int u = 0; u < kBlockDepth; ++u) {
          if (i0 + (uint32_t)(u * kBlockThreads) >= n32) break;
          const int x = (grid32(v[u], L.th) >> sh) - lo;
          if (x >= 0 && x < G) atomicAdd(&cgrid[x], 1u);
          else out_of_range = true;
        }
      }
    } else {
      for (uint64_t i0 = tid; i0 < n; i0 += kBlockDepth * kBlockThreads) {
        uint64_t v[kBlockDepth];
        vals.get(i0, kBlockThreads, n, v, 0ull);
#pragma unroll
        for (int u = 0; u < kBlockDepth; ++u) {
          if (i0 + u * kBlockThreads >= n) break;
          const int x = (grid64(v[u], L.th) >> sh) - lo;
          if (x >= 0 && x < G) atomicAdd(&cgrid[x], 1u);
          else out_of_range = true;
        }
      }
    }
    if (out_of_range) s_bad = 1;
    __syncthreads();
    if (s_bad) {  // durations outside the summarized [min, max]
      if (wv == 0) {
        if (l == 0) flag(a, ARGUS_DEV_KDE_SUMMARY);
        write_empty(a, c);
      }
      __syncthreads();
      continue;
    }

    // 2-8. analysis on wavefront 0
    Analysis an{};
    if (wv == 0) {
      const bool ok = kde_analyze<1>(a, L, cm, lo, G, an);
      if (l == 0) {
        s_ok = ok ? 1u : 0u;
        s_nt = (uint32_t)an.NT;
      }
    }
    __syncthreads();
    if (!s_ok) {
      if (tid == 0) a.list1[atomicAdd(&a.counters[2], 1u)] = (uint32_t)c;
      __syncthreads();
      continue;
    }
    const int NT = (int)__builtin_amdgcn_readfirstlane(s_nt);

    // 9. selection passes: target t's candidates are the durations in
    // [tlb, tub), of which tpop are there and the one of rank trank is wanted
    if (tid < kMaxT) L.tdone[tid] = tid < NT && L.tub[tid] - L.tlb[tid] <= 1 ? 1u : 0u;
    __syncthreads();
    while (true) {
      // per target, uniform: range start, width (0 once resolved), digit
      // shift (-1: gather); bit t of narrow: offsets in the range fit 32 bits
      // (gathered as 4-byte offsets, up to kSelCap32 of them)
      uint64_t tlo[kMaxT], twd[kMaxT];
      int tsh[kMaxT];
      uint32_t live = 0, narrow = 0;
#pragma unroll
      for (int t = 0; t < kMaxT; ++t) {
        tlo[t] = 0;
        twd[t] = 0;
        tsh[t] = -1;
        if (t < NT && !L.tdone[t]) {
          tlo[t] = readlane64(L.tlb[t], 0);
          twd[t] = readlane64(L.tub[t] - L.tlb[t], 0);
          const int bits = 64 - __builtin_clzll(twd[t] - 1);  // width >= 2
          const bool nar = bits <= 32;
          const uint32_t cap = nar ? (uint32_t)kSelCap32 : (uint32_t)kSelCap;
          tsh[t] = (int)__builtin_amdgcn_readfirstlane(
              L.tpop[t] <= cap ? -1 : (bits > kSelDigit ? bits - kSelDigit : 0));
          live |= 1u << t;
          narrow |= (nar ? 1u : 0u) << t;
        }
      }
      live = __builtin_amdgcn_readfirstlane(live);
      narrow = __builtin_amdgcn_readfirstlane(narrow);
      if (live == 0) break;
      for (int i = tid; i < kMaxT * kSelRegion; i += kBlockThreads) L.buf[i] = 0;
      if (tid < kMaxT) L.tcnt[tid] = 0;
      __syncthreads();
      // 4-byte records whose live target ranges all end at or below 2^32:
      // the same tests on 32-bit offsets (every such range is narrow, so its
      // candidates are gathered as offsets), half the arithmetic per test
      bool t32 = vals.w4;
#pragma unroll
      for (int t = 0; t < kMaxT; ++t)
        if ((live >> t) & 1u)
          t32 = t32 && tlo[t] < (1ull << 32) && twd[t] < (1ull << 32) && twd[t] <= (1ull << 32) - tlo[t];
      if (t32) {
        const uint32_t* q = static_cast<const uint32_t*>(vals.p);
        const uint32_t n32 = (uint32_t)n;
        for (uint32_t i0 = (uint32_t)tid; i0 < n32; i0 += kBlockDepth * kBlockThreads) {
          uint32_t v[kBlockDepth];
#pragma unroll
          for (int k = 0; k < kBlockDepth; ++k) {
            const uint32_t i = i0 + (uint32_t)(k * kBlockThreads);
            v[k] = i < n32 ? q[i] : 0u;
          }
#pragma unroll
          for (int t = 0; t < kMaxT; ++t) {
            if (!((live >> t) & 1u)) continue;
            const uint32_t lo32 = (uint32_t)tlo[t], wd32 = (uint32_t)twd[t];
#pragma unroll
            for (int k = 0; k < kBlockDepth; ++k) {
              const uint32_t u = v[k] - lo32;
              if (i0 + (uint32_t)(k * kBlockThreads) < n32 && u < wd32) {
                if (tsh[t] < 0) {
                  const uint32_t slot = atomicAdd(&L.tcnt[t], 1u);
                  if (slot < (uint32_t)kSelCap32) L.buf[t * kSelRegion + (int)slot] = u;
                } else {
                  atomicAdd(&L.buf[t * kSelRegion + (int)(u >> tsh[t])], 1u);
                }
              }
            }
          }
        }
      } else {
        // live targets outer (a uniform test each), the loaded durations inner
        for (uint64_t i0 = tid; i0 < n; i0 += kBlockDepth * kBlockThreads) {
          uint64_t v[kBlockDepth];
          vals.get(i0, kBlockThreads, n, v, 0ull);
#pragma unroll
          for (int t = 0; t < kMaxT; ++t) {
            if (!((live >> t) & 1u)) continue;
#pragma unroll
            for (int k = 0; k < kBlockDepth; ++k) {
              const uint64_t u = v[k] - tlo[t];
              if (i0 + k * kBlockThreads < n && u < twd[t]) {
                if (tsh[t] < 0) {
                  const uint32_t slot = atomicAdd(&L.tcnt[t], 1u);
                  if ((narrow >> t) & 1u) {
                    if (slot < (uint32_t)kSelCap32) L.buf[t * kSelRegion + (int)slot] = (uint32_t)u;
                  } else if (slot < (uint32_t)kSelCap) {
                    reinterpret_cast<uint64_t*>(L.buf + t * kSelRegion)[slot] = v[k];
                  }
                } else {
                  atomicAdd(&L.buf[t * kSelRegion + (int)(u >> tsh[t])], 1u);
                }
              }
            }
          }
        }
      }
      __syncthreads();
      // wavefront wv resolves targets wv, wv + kBlockWaves, ...
      for (int t = wv; t < kMaxT; t += kBlockWaves) {
        if (!((live >> t) & 1u)) continue;
        const uint64_t r = readlane64(L.trank[t], 0);
        const uint64_t base = readlane64(L.tlb[t], 0);
        if (tsh[t] < 0 && ((narrow >> t) & 1u)) {
          // radix selection among the gathered offsets
          const uint32_t got = L.tcnt[t];
          const int k = got < (uint32_t)kSelCap32 ? (int)got : kSelCap32;
          bool ok;
          const uint32_t off = select_offsets(L.buf + t * kSelRegion, L.buf + t * kSelRegion + kSelCap32, k,
                                              64 - __builtin_clzll(twd[t] - 1), r, ok);
          if (l == 0) {
            L.tlb[t] = ok ? base + off : base;
            L.tdone[t] = 1;
          }
        } else if (tsh[t] < 0) {
          // counting rank among the gathered durations
          const uint64_t* list = reinterpret_cast<const uint64_t*>(L.buf + t * kSelRegion);
          const uint32_t got = L.tcnt[t];
          const int k = got < (uint32_t)kSelCap ? (int)got : kSelCap;
          const uint64_t e = l < k ? list[l] : 0ull;
          const uint32_t rank = rank_in_list(list, k, e);
          const uint64_t hit = __ballot(l < k && (uint64_t)rank == r);
          const uint64_t val = readlane64(e, hit ? __builtin_ctzll(hit) : 0);
          if (l == 0) {
            L.tlb[t] = hit ? val : base;
            L.tdone[t] = 1;
          }
        } else {
          // the digit holding rank r: 8 counters per lane, a wave scan
          constexpr int PER = kSelRegion / kWave;
          const uint32_t* h = L.buf + t * kSelRegion + l * PER;
          uint32_t cnt[PER], sum = 0;
#pragma unroll
          for (int k = 0; k < PER; ++k) {
            cnt[k] = h[k];
            sum += cnt[k];
          }
          const uint32_t incl = wave_incl_scan(sum);
          const bool mine = (uint64_t)(incl - sum) <= r && r < (uint64_t)incl;
          const uint64_t bm = __ballot(mine);
          const int owner = bm ? __builtin_ctzll(bm) : 0;
          uint32_t sub = 0, pop = 0;
          uint64_t rr = 0;
          if (l == owner) {
            rr = bm ? r - (incl - sum) : 0;
            int k = 0;
#pragma unroll
            for (int q = 0; q < PER - 1; ++q)
              if (k == q && rr >= cnt[q]) {
                rr -= cnt[q];
                k = q + 1;
              }
            uint32_t pk = 0;
#pragma unroll
            for (int q = 0; q < PER; ++q)
              if (q == k) pk = cnt[q];
            sub = (uint32_t)(owner * PER + k);
            pop = pk;
          }
          sub = __builtin_amdgcn_readlane(sub, owner);
          pop = __builtin_amdgcn_readlane(pop, owner);
          rr = readlane64(rr, owner);
          const uint64_t nlo = base + ((uint64_t)sub << tsh[t]);
          const uint64_t span = 1ull << tsh[t];
          const uint64_t end = base + twd[t];
          const uint64_t nhi = end - nlo < span ? end : nlo + span;
          if (l == 0) {
            L.tlb[t] = nlo;
            L.tub[t] = nhi;
            L.trank[t] = rr;
            L.tpop[t] = pop;
            L.tdone[t] = (nhi - nlo <= 1 || pop == 0) ? 1u : 0u;
          }
        }
      }
      __syncthreads();
    }

    // outputs (wavefront 0 holds the analysis)
    if (wv == 0) {
      if (l < kMaxC) {
        const int64_t o = c * kMaxC + l;
        uint32_t cnt = 0;
#pragma unroll
        for (int q = 0; q < kMaxC; ++q)
          if (q == l) cnt = an.ccount[q];
        a.cl_count[o] = l < an.ncl ? cnt : 0u;
        a.p50[o] = l < an.ncl ? (int64_t)L.tlb[2 * l] : 0;
        a.p99[o] = l < an.ncl ? (int64_t)L.tlb[2 * l + 1] : 0;
      }
      if (l == 0) {
        a.n_clusters[c] = (uint8_t)an.ncl;
        if (a.bw_q8) a.bw_q8[c] = (int32_t)an.H;
      }
    }
    __syncthreads();
  }
}

// -------------------------------------------------------------- lane tier
// Cells of at most kLaneN durations whose grid has at most kLaneG points
// (nine cells in ten in the benchmark workloads; the median holds 40
// durations) are processed one per lane, 64 cells per wavefront, each lane
// running every step of the definition on its own cell: a wavefront per
// such cell would spend most of its instructions on per-cell fixed costs.
// Per-lane arrays live in LDS with the lane as the fastest index, so lanes
// at the same step touch consecutive words. A lane that finds more valleys
// than kLaneCand, or more durations in a target grid bin than kLaneList,
// writes nothing and hands its cell to the wavefront tiers, like every cell
// outside these limits. The per-lane arrays are kept small (weights and
// target-bin offsets in 16 bits where they fit) because the lane passes are
// latency bound: every kilobyte of LDS per wavefront is resident wavefronts
// per CU.
constexpr int kLaneN = 255;     // durations per cell (counts fit in 8 bits, densities in 24)
constexpr int kLaneG = 64;      // grid points per cell, first lane pass (over every cell)
constexpr int kLaneGW = 256;    // grid points per cell, second lane pass (listed wide cells)
constexpr int kLaneT = 32;      // kernel weights (t < 32)
constexpr int kLaneCand = 8;    // valleys before filtering
constexpr int kLaneList = 16;   // durations of one target grid bin
static_assert(2 * kLaneList <= kLaneT, "two target lists in the weight words");

template <int GC>
struct LaneLds {
  alignas(4) uint8_t cp[GC][kWave];  // grid counts, then inclusive prefix counts (8 bits: n <= 255)
  // kernel weights w(t) for 1 <= t < kLaneT (w(0) = 65536 is implicit; a cell
  // whose w(1) needs 17 bits goes to the wavefront tiers); later the
  // durations of a cluster's target bins as offsets from the bin start: two
  // bins of 16-bit offsets, or one bin of 32-bit offsets
  union {
    uint16_t w[kLaneT][kWave];
    uint16_t off16[2 * kLaneList][kWave];
    uint32_t off32[kLaneList][kWave];
  };
  uint32_t cand[kLaneCand][kWave]; // valleys: density << 8 | grid index
  uint32_t th[64];
};

template <int GC>
__device__ __forceinline__ uint32_t lane_cnt(const LaneLds<GC>& L, int j, int l) {
  return L.cp[j][l];
}

template <int GC>
__device__ __forceinline__ void lane_drop(LaneLds<GC>& L, int i, int& m, int l) {
  for (int q = i; q + 1 < m; ++q) L.cand[q][l] = L.cand[q + 1][l];
  --m;
}

// Per-lane empty record (count 0, or a summary that does not match).
__device__ __forceinline__ void lane_write(const KdeArgs& a, int64_t c, int ncl, const uint32_t (&cnt)[kMaxC],
                                           const uint64_t (&p50)[kMaxC], const uint64_t (&p99)[kMaxC], int64_t H) {
  *reinterpret_cast<uint4*>(a.cl_count + c * kMaxC) = make_uint4(cnt[0], cnt[1], cnt[2], cnt[3]);
  v2l* q50 = reinterpret_cast<v2l*>(a.p50 + c * kMaxC);
  v2l* q99 = reinterpret_cast<v2l*>(a.p99 + c * kMaxC);
  q50[0] = v2l{(long long)p50[0], (long long)p50[1]};
  q50[1] = v2l{(long long)p50[2], (long long)p50[3]};
  q99[0] = v2l{(long long)p99[0], (long long)p99[1]};
  q99[1] = v2l{(long long)p99[2], (long long)p99[3]};
  a.n_clusters[c] = (uint8_t)ncl;
  if (a.bw_q8) a.bw_q8[c] = (int32_t)H;
}

// One cell on one lane. Returns false (nothing written) when the cell does
// not fit the lane limits found on the way.
template <int GC>
__device__ bool lane_cell(const KdeArgs& a, LaneLds<GC>& L, int64_t c, const CellMeta& cm) {
  const int l = lane_id();
  const uint32_t n = cm.n;
  const Durs vals = durs_of(a, cm);
  const int sh = 6 - a.sub_bits;
  const int lo = grid64((uint64_t)cm.mn, L.th) >> sh;
  const int G = (grid64((uint64_t)cm.mx, L.th) >> sh) - lo + 1;

  // 1. grid histogram; eight loads in flight per lane, and LDS adds that
  // return nothing, so no iteration waits on the previous one
  for (int j = 0; j < G; ++j) L.cp[j][l] = 0;
  bool out_of_range = false;
  // the lane's count byte lives in a word shared with three other lanes
  auto add = [&](int x) {
    if (x >= 0 && x < G) atomicAdd(reinterpret_cast<uint32_t*>(&L.cp[x][l & ~3]), 1u << ((l & 3) * 8));
    else out_of_range = true;
  };
  for (uint32_t i0 = 0; i0 < n; i0 += 8) {
    uint64_t d[8];
    vals.run8(i0, n, d, 0ull);
    // 4-byte records: grid indices from 32-bit operations
    if (vals.w4) {
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (i0 + u < n) add((grid32((uint32_t)d[u], L.th) >> sh) - lo);
    } else {
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (i0 + u < n) add((grid64(d[u], L.th) >> sh) - lo);
    }
  }
  uint32_t cnt[kMaxC] = {0, 0, 0, 0};
  uint64_t p50[kMaxC] = {0, 0, 0, 0}, p99[kMaxC] = {0, 0, 0, 0};
  if (out_of_range) {  // durations outside the summarized [min, max]
    flag(a, ARGUS_DEV_KDE_SUMMARY);
    lane_write(a, c, 0, cnt, p50, p99, 0);
    return true;
  }

  // 2. bandwidth (exact integer moments: n <= 255, x < 64)
  int64_t H = 0;
  if (n >= 2) {
    uint64_t s1 = 0, s2 = 0;
    for (int j = 0; j < G; ++j) {
      const uint64_t k = lane_cnt(L, j, l);
      s1 += k * (uint64_t)j;
      s2 += k * (uint64_t)j * (uint64_t)j;
    }
    const double var = (double)(n * s2 - s1 * s1) / ((double)n * (double)(n - 1));
    H = kde_bw_q8(var, cm.pw);
  }

  // 3-4. weights, then the density in one pass with its valleys: a run of
  // equal values entered from above and left upwards is a valley, placed at
  // the middle of the run
  int m = 0;
  if (H > 0 && G >= 3) {
    const double H2 = (double)(H * H);
    int T = -1;
    for (int t = 0; t < G; ++t) {
      const uint32_t wt = kde_weight(t, H2);
      if (wt == 0) break;
      if (t == kLaneT) return false;  // kernel wider than the lane's weight table
      if (t > 0) {
        if (wt > 0xFFFFu) return false;  // w(1) = 65536: a bandwidth far beyond the table's reach
        L.w[t][l] = (uint16_t)wt;
      }
      T = t;
    }
    uint32_t v = 0, pv = 0;
    int r0 = 0;
    for (int j = 0; j < G; ++j) {
      const int b0 = j - T > 0 ? j - T : 0, b1 = j + T < G - 1 ? j + T : G - 1;
      // left of j the distance falls to 1, right of it it rises from 1: two
      // loops walk the weight column by pointer (counts < 256, weights
      // < 2^16); j itself weighs w(0) = 65536
      uint32_t f = 0;
      const uint16_t* wl = &L.w[j - b0][l];
      const uint8_t* cl = &L.cp[b0][l];
#pragma unroll 4
      for (int b = b0; b < j; ++b, wl -= kWave, cl += kWave) f += __umul24(*cl, *wl);
      f += (uint32_t)*cl << 16;
      cl += kWave;
      const uint16_t* wr = &L.w[1][l];
#pragma unroll 4
      for (int b = j + 1; b <= b1; ++b, wr += kWave, cl += kWave) f += __umul24(*cl, *wr);
      if (j == 0) {
        v = f;
      } else if (f != v) {
        if (r0 >= 1 && pv > v && f > v) {
          if (m == kLaneCand) return false;
          L.cand[m][l] = (v << 8) | (uint32_t)((r0 + j - 1) / 2);
          ++m;
        }
        pv = v;
        v = f;
        r0 = j;
      }
    }
  }

  // grid counts -> inclusive prefix counts (at most n <= 255), in place
  {
    uint32_t run = 0;
    for (int j = 0; j < G; ++j) {
      run += L.cp[j][l];
      L.cp[j][l] = (uint8_t)run;
    }
  }
  auto P = [&](int j) -> uint32_t { return j < 0 ? 0u : lane_cnt(L, j, l); };
  auto pos = [&](int q) -> int { return (int)(L.cand[q][l] & 0xFFu); };
  auto val = [&](int q) -> uint32_t { return L.cand[q][l] >> 8; };
  auto hi_of = [&](int q, int mm) -> int { return q < mm ? pos(q) : G - 1; };

  // 5. cluster-level filter
  uint32_t need = (uint32_t)(((uint64_t)a.frac_pm * n + 999u) / 1000u);
  if (need < (uint32_t)a.min_count) need = (uint32_t)a.min_count;
  while (m > 0) {
    int best = 0;
    uint32_t best_size = 0;
    for (int q = 0; q <= m; ++q) {
      const uint32_t sz = P(hi_of(q, m)) - (q > 0 ? P(pos(q - 1)) : 0u);
      if (q == 0 || sz < best_size) {
        best = q;
        best_size = sz;
      }
    }
    if (best_size >= need) break;
    lane_drop(L, best == 0 ? 0 : (best == m ? m - 1 : (val(best - 1) > val(best) ? best - 1 : best)), m, l);
  }

  // 6. spacing filter over [0, valleys..., G - 1]
  while (m > 0) {
    int hit = -1;
    for (int q = 0; q <= m && hit < 0; ++q)
      if (hi_of(q, m) - (q > 0 ? pos(q - 1) : 0) < a.gap) hit = q;
    if (hit < 0) break;
    lane_drop(L, hit == 0 ? 0 : (hit == m ? m - 1 : (val(hit - 1) > val(hit) ? hit - 1 : hit)), m, l);
  }

  // 7. cluster cap: drop the largest-density valley (the upper one on ties)
  while (m > kMaxC - 1) {
    int s = 0;
    for (int q = 1; q < m; ++q)
      if (val(q) >= val(s)) s = q;
    lane_drop(L, s, m, l);
  }

  // 8. per cluster: count, then p50 / p99 as the element of the wanted rank
  // inside its grid bin, found among the bin's durations gathered in LDS. The
  // targets' ranks increase, so the bin search goes on from the last bin. A
  // cluster's two bins are gathered in one pass over the durations, as 16-bit
  // offsets from the bin start, when both bins are at most 2^16 ns wide (bins
  // of durations below about 6 ms); otherwise one bin per pass as 32-bit
  // offsets, and bins wider than 2^32 ns hand the cell to the wavefront tiers.
  const int ncl = m + 1;
  uint32_t before = 0;
  int jc = 0;
  for (int q = 0; q < ncl; ++q) {
    const uint32_t hiP = P(hi_of(q, m)), size = hiP - before;
    for (int qq = 0; qq < kMaxC; ++qq)
      if (qq == q) cnt[qq] = size;
    uint32_t rr[2], k[2];
    uint64_t lb[2], ub[2];
    bool narrow = true;
    for (int t2 = 0; t2 < 2; ++t2) {
      const uint32_t r = t2 == 0 ? before + (size - 1) / 2 : before + (99 * size + 99) / 100 - 1;
      while (P(jc) <= r) ++jc;  // smallest grid index whose prefix count passes r
      const uint32_t below = P(jc - 1);
      k[t2] = P(jc) - below;
      if (k[t2] > (uint32_t)kLaneList) return false;
      rr[t2] = r - below;
      lb[t2] = grid64_lb((lo + jc) << sh, L.th);
      ub[t2] = grid64_lb((lo + jc + 1) << sh, L.th);
      narrow = narrow && ub[t2] - lb[t2] <= (1ull << 16);
    }
    const bool same = lb[1] == lb[0];
    uint64_t pick[2] = {0, 0};
    if (narrow) {
      // list t at entries [16 t, 16 t + k[t]): 16-bit offsets from lb[t]
      uint32_t got0 = 0, got1 = same ? k[1] : 0u;
      for (uint32_t i0 = 0; i0 < n && (got0 < k[0] || got1 < k[1]); i0 += 8) {
        uint64_t d[8];
        vals.run8(i0, n, d, ~0ull);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          if (d[u] >= lb[0] && d[u] < ub[0] && got0 < k[0]) L.off16[got0++][l] = (uint16_t)(d[u] - lb[0]);
          if (!same && d[u] >= lb[1] && d[u] < ub[1] && got1 < k[1])
            L.off16[kLaneList + got1++][l] = (uint16_t)(d[u] - lb[1]);
        }
      }
      for (int t2 = 0; t2 < 2; ++t2) {
        const int base = same ? 0 : t2 * kLaneList;
        uint32_t off = 0;
        for (uint32_t i = 0; i < k[t2]; ++i) {
          const uint32_t e = L.off16[base + i][l];
          uint32_t rank = 0;
          for (uint32_t x = 0; x < k[t2]; ++x) {
            const uint32_t y = L.off16[base + x][l];
            rank += (y < e || (y == e && x < i)) ? 1u : 0u;
          }
          if (rank == rr[t2]) off = e;
        }
        pick[t2] = lb[t2] + off;
      }
    } else {
      for (int t2 = 0; t2 < 2; ++t2) {
        if (ub[t2] - lb[t2] > (1ull << 32)) return false;
        uint32_t got = 0;
        for (uint32_t i0 = 0; i0 < n && got < k[t2]; i0 += 8) {
          uint64_t d[8];
          vals.run8(i0, n, d, ~0ull);
#pragma unroll
          for (int u = 0; u < 8; ++u)
            if (d[u] >= lb[t2] && d[u] < ub[t2] && got < k[t2]) L.off32[got++][l] = (uint32_t)(d[u] - lb[t2]);
        }
        uint32_t off = 0;
        for (uint32_t i = 0; i < k[t2]; ++i) {
          const uint32_t e = L.off32[i][l];
          uint32_t rank = 0;
          for (uint32_t x = 0; x < k[t2]; ++x) {
            const uint32_t y = L.off32[x][l];
            rank += (y < e || (y == e && x < i)) ? 1u : 0u;
          }
          if (rank == rr[t2]) off = e;
        }
        pick[t2] = lb[t2] + off;
      }
    }
    for (int qq = 0; qq < kMaxC; ++qq) {
      if (qq != q) continue;
      p50[qq] = pick[0];
      p99[qq] = pick[1];
    }
    before = hiP;
  }
  lane_write(a, c, ncl, cnt, p50, p99, H);
  return true;
}

// ------------------------------------------------------------------ routing
// Before the lane passes every cell is routed once, one thread per cell:
// empty cells (and cells whose summary does not match the buckets) are
// written, heavy cells go to the workgroup tier's list, cells too large for
// either lane pass to tier 0's list, and the rest to one of the two lane
// passes, ordered by a cost class. A lane pass runs 64 cells in lockstep, so
// a wavefront takes as long as its costliest cell, and cells in kernel-id
// order mix grids of 10 and 64 points and 10 and 255 durations. The class
// groups cells of similar grid size and duration count, whose loops run
// similar trip counts: ((G - 1) / 2, (n - 1) / 16) for the first lane pass
// (G <= 64), kLaneClasses + ((G - 65) / 8, (n - 1) / 16) for the wide pass
// (65 <= G <= 256). A counting sort over the classes (counts here,
// positions in kde_lane_order_kernel) lays each lane list out in class
// order. Each workgroup routes a contiguous range of cells and claims its
// list ranges with one atomic per list and class.
constexpr int kRouteThreads = 512;
constexpr int kLaneClasses = 512;                          // 32 grid-size x 16 duration-count classes
constexpr int kWideClasses = 384;                          // 24 x 16 for the wide pass
constexpr int kClasses = 1024;                             // both, padded to two per thread
constexpr uint16_t kNoClass = 0xFFFF, kHeavy = 0xFFFE, kTier0 = 0xFFFD;
constexpr int kOrderPer = 16;  // cells per thread and round in kde_lane_order_kernel
static_assert(kClasses == 2 * kRouteThreads && kLaneClasses + kWideClasses <= kClasses, "class scan");
static_assert(((kLaneG - 1) >> 1) * 16 + ((kLaneN - 1) >> 4) < kLaneClasses, "lane classes");
static_assert(((kLaneGW - 65) >> 3) * 16 + ((kLaneN - 1) >> 4) < kWideClasses, "wide classes");

// Route code of a cell from its checked summary: a class, kHeavy, kTier0, or
// kNoClass (nothing left to do: the empty record is written by the caller).
__device__ __forceinline__ uint16_t route_code(const CellMeta& m, const uint32_t* th, int sh) {
  if (m.n == 0 || m.off < 0) return kNoClass;
  if (m.n >= kBlockMin) return kHeavy;
  if (m.n > (uint32_t)kLaneN) return kTier0;
  const int G = (grid64((uint64_t)m.mx, th) >> sh) - (grid64((uint64_t)m.mn, th) >> sh) + 1;
  const int nq = (int)((m.n - 1) >> 4);
  if (G <= kLaneG) return (uint16_t)(((G - 1) >> 1) * 16 + nq);
  if (G <= kLaneGW) return (uint16_t)(kLaneClasses + ((G - 65) >> 3) * 16 + nq);
  return kTier0;
}

// Index for each lane with pred among the new entries of an LDS list
// counter: one atomic per wavefront. Called by every lane of the wavefront.
__device__ __forceinline__ uint32_t wave_append(uint32_t* counter, bool pred) {
  const uint64_t m = __ballot(pred);
  if (m == 0) return 0;
  const int leader = __builtin_ctzll(m);
  uint32_t base = 0;
  if (lane_id() == leader) base = atomicAdd(counter, (uint32_t)__popcll(m));
  base = __builtin_amdgcn_readlane(base, leader);
  return base + (uint32_t)__popcll(m & ((1ull << lane_id()) - 1ull));
}

// Contiguous range of cells of workgroup b out of nb.
__device__ __forceinline__ void cell_range(int64_t C, int64_t b, int64_t nb, int64_t& c0, int64_t& c1) {
  const int64_t per = (C + nb - 1) / nb;
  c0 = b * per < C ? b * per : C;
  c1 = c0 + per < C ? c0 + per : C;
}

__global__ __launch_bounds__(kRouteThreads) void kde_route_kernel(KdeArgs a) {
  __shared__ uint32_t hist[kClasses];
  __shared__ uint32_t th[64];
  __shared__ uint32_t n_heavy, n_tier0, base_heavy, base_tier0;
  const int tid = threadIdx.x;
  if (tid < 64) th[tid] = a.theta[tid];
  hist[tid] = hist[tid + kRouteThreads] = 0;
  if (tid == 0) n_heavy = n_tier0 = 0;
  __syncthreads();
  const int64_t C = (int64_t)a.n_seg * a.K;
  int64_t c0, c1;
  cell_range(C, blockIdx.x, gridDim.x, c0, c1);
  const int sh = 6 - a.sub_bits;
  // 1. route codes; empty records; per-workgroup counts
  for (int64_t cb = c0; cb < c1; cb += kRouteThreads) {
    const int64_t c = cb + tid;
    uint16_t code = kNoClass;
    if (c < c1) {
      const CellMeta m = load_meta(a, c);
      code = route_code(m, th, sh);
      if (code == kNoClass) {
        if (m.n != 0) flag(a, ARGUS_DEV_KDE_SUMMARY);
        const uint32_t z[kMaxC] = {0, 0, 0, 0};
        const uint64_t zz[kMaxC] = {0, 0, 0, 0};
        lane_write(a, c, 0, z, zz, zz, 0);
      } else if (code < kClasses) {
        atomicAdd(&hist[code], 1u);
      }
      a.lane_key[c] = code;
    }
    wave_append(&n_heavy, code == kHeavy);
    wave_append(&n_tier0, code == kTier0);
  }
  __syncthreads();
  // 2. list ranges of this workgroup
  if (tid == 0) {
    uint32_t nl = 0, nw = 0;
    for (int k = 0; k < kLaneClasses; ++k) nl += hist[k];
    for (int k = kLaneClasses; k < kClasses; ++k) nw += hist[k];
    if (nl) atomicAdd(&a.counters[12], nl);
    if (nw) atomicAdd(&a.counters[9], nw);
    base_heavy = n_heavy ? atomicAdd(&a.counters[11], n_heavy) : 0u;
    base_tier0 = n_tier0 ? atomicAdd(&a.counters[7], n_tier0) : 0u;
    n_heavy = n_tier0 = 0;
  }
  for (int k = tid; k < kClasses; k += kRouteThreads)
    if (hist[k]) atomicAdd(&a.lane_cls[k], hist[k]);
  __syncthreads();
  // 3. heavy and tier-0 entries (the lane lists are laid out by the next kernel)
  for (int64_t cb = c0; cb < c1; cb += kRouteThreads) {
    const int64_t c = cb + tid;
    const uint16_t code = c < c1 ? a.lane_key[c] : kNoClass;
    const uint32_t ih = wave_append(&n_heavy, code == kHeavy);
    if (code == kHeavy) a.list2[C - 1 - (int64_t)(base_heavy + ih)] = (uint32_t)c;
    const uint32_t i0 = wave_append(&n_tier0, code == kTier0);
    if (code == kTier0) a.list2[base_tier0 + i0] = (uint32_t)c;
  }
}

// Positions of the lane passes' cells: class offsets from an exclusive scan
// of the class counts, a range per class and round claimed with one atomic,
// ranks inside the round from LDS atomics. First-pass cells of position p
// go to list1[C - 1 - p], wide cells to list1[p - (first-pass total)].
__global__ __launch_bounds__(kRouteThreads) void kde_lane_order_kernel(KdeArgs a) {
  __shared__ uint32_t off[kClasses], lcnt[kClasses], lbase[kClasses];
  __shared__ uint32_t wsum[kRouteThreads / kWave];
  const int tid = threadIdx.x, wv = tid / kWave;
  {
    const uint32_t v0 = a.lane_cls[2 * tid], v1 = a.lane_cls[2 * tid + 1];
    const uint32_t incl = wave_incl_scan(v0 + v1);
    if (lane_id() == kWave - 1) wsum[wv] = incl;
    __syncthreads();
    uint32_t base = incl - v0 - v1;
    for (int w = 0; w < wv; ++w) base += wsum[w];
    off[2 * tid] = base;
    off[2 * tid + 1] = base + v0;
  }
  __syncthreads();
  const uint32_t n_first = off[kLaneClasses];
  const int64_t C = (int64_t)a.n_seg * a.K;
  int64_t c0, c1;
  cell_range(C, blockIdx.x, gridDim.x, c0, c1);
  for (int64_t cb = c0; cb < c1; cb += (int64_t)kOrderPer * kRouteThreads) {
    lcnt[tid] = lcnt[tid + kRouteThreads] = 0;
    __syncthreads();
    uint16_t key[kOrderPer];
    uint32_t rank[kOrderPer];
#pragma unroll
    for (int u = 0; u < kOrderPer; ++u) {
      const int64_t c = cb + (int64_t)u * kRouteThreads + tid;
      key[u] = c < c1 ? a.lane_key[c] : kNoClass;
      rank[u] = key[u] < kClasses ? atomicAdd(&lcnt[key[u]], 1u) : 0u;
    }
    __syncthreads();
    for (int k = tid; k < kClasses; k += kRouteThreads)
      if (lcnt[k]) lbase[k] = atomicAdd(&a.lane_cls[kClasses + k], lcnt[k]);
    __syncthreads();
#pragma unroll
    for (int u = 0; u < kOrderPer; ++u) {
      if (key[u] >= kClasses) continue;
      const int64_t c = cb + (int64_t)u * kRouteThreads + tid;
      const int64_t p = (int64_t)off[key[u]] + lbase[key[u]] + rank[u];
      if (key[u] < kLaneClasses) a.list1[C - 1 - p] = (uint32_t)c;
      else a.list1[p - n_first] = (uint32_t)c;
    }
    __syncthreads();
  }
}

// Lane passes. GC = kLaneG: the routed cells in class order, 64 list
// entries per claim; GC = kLaneGW: the wide list. A cell that does not fit
// the lane limits goes to list 0 (tier 0).
template <int GC>
__global__ __launch_bounds__(kWave) void kde_lane_kernel(KdeArgs a) {
  constexpr bool kFirst = GC == kLaneG;
  __shared__ LaneLds<GC> L;
  const int l = lane_id();
  L.th[l] = a.theta[l];
  wave_sync();
  const int64_t Ctot = (int64_t)a.n_seg * a.K;
  const int64_t C = (int64_t)__builtin_amdgcn_readfirstlane(
      __hip_atomic_load(&a.counters[kFirst ? 12 : 9], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  const int sh = 6 - a.sub_bits;
  while (true) {
    uint32_t claim = 0;
    if (l == 0) claim = atomicAdd(&a.counters[kFirst ? 6 : 8], 1u);
    claim = __builtin_amdgcn_readfirstlane(claim);
    if ((int64_t)claim * kWave >= C) break;
    const int64_t i = (int64_t)claim * kWave + l;
    if (i < C) {
      const int64_t c = kFirst ? (int64_t)a.list1[Ctot - 1 - i] : (int64_t)a.list1[i];
      const CellMeta m = load_meta(a, c);
      bool done = false;
      if (m.off >= 0 && m.n <= (uint32_t)kLaneN) {
        const int G = (grid64((uint64_t)m.mx, L.th) >> sh) - (grid64((uint64_t)m.mn, L.th) >> sh) + 1;
        if (G <= GC) done = lane_cell<GC>(a, L, c, m);
      }
      if (!done) a.list2[atomicAdd(&a.counters[7], 1u)] = (uint32_t)c;
    }
  }
}

// ---------------------------------------------------------------- host side

__global__ void kde_pow_table_kernel() {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n < kPowTab) g_kde_pow[n] = n > 0 ? kde_pw((uint64_t)n) : 0.0;
}

// Fill g_kde_pow on the current device once (before its first KDE call).
hipError_t ensure_pow_table() {
  static std::mutex mu;
  static bool done[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  if (done[dev]) return hipSuccess;
  hipLaunchKernelGGL(kde_pow_table_kernel, dim3(kPowTab / 256), dim3(256), 0, nullptr);
  e = hipGetLastError();
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e == hipSuccess) done[dev] = true;
  return e;
}

template <typename Kern>
int resident(Kern kern, int threads) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, threads, 0) != hipSuccess) return 0;
  return cus * (per_cu > 0 ? per_cu : 1);
}

__global__ void kde_clear_kernel(uint32_t* counters, uint32_t* lane_cls, int32_t* dev_status) {
  if (threadIdx.x < 16) counters[threadIdx.x] = 0;
  for (int i = threadIdx.x; i < 2 * kClasses; i += blockDim.x) lane_cls[i] = 0;
  if (threadIdx.x == 0 && dev_status) *dev_status = 0;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }

}  // namespace

size_t kde_workspace_bytes(int64_t n_events, int64_t n_seg, int64_t cells) {
  return 256 + al256((size_t)n_events * 8) + 3 * al256((size_t)cells * 4) + al256((size_t)cells * 2) +
         al256((size_t)2 * kClasses * 4) + al256((size_t)n_seg);
}

hipError_t launch_kde(const KdeLaunch& l, hipStream_t st) {
  hipError_t e = ensure_pow_table();
  if (e != hipSuccess) return e;
  const int64_t cells = (int64_t)l.n_seg * l.n_kernels;
  char* ws = static_cast<char*>(l.workspace);
  KdeArgs a{};
  a.kernel_id = l.kernel_id;
  a.stream = l.stream;
  a.start_ns = l.start_ns;
  a.end_ns = l.end_ns;
  a.seg_off = l.seg_off;
  a.n_events = l.n_events;
  a.n_seg = l.n_seg;
  a.K = l.n_kernels;
  a.NS = l.n_streams;
  a.vec_ok = aligned16(l.kernel_id) && aligned16(l.stream) && aligned16(l.start_ns) && aligned16(l.end_ns);
  a.sub_bits = l.p.sub_bits;
  a.frac_pm = l.p.frac_pm;
  a.min_count = l.p.min_count;
  a.gap = l.p.gap;
  a.count = l.count;
  a.min_ns = l.min_ns;
  a.max_ns = l.max_ns;
  a.n_invalid = l.n_invalid;
  a.n_clusters = l.o.n_clusters;
  a.cl_count = l.o.count;
  a.p50 = l.o.p50_ns;
  a.p99 = l.o.p99_ns;
  a.bw_q8 = l.o.bw_q8;
  a.dev_status = l.o.dev_status;
  a.counters = reinterpret_cast<uint32_t*>(ws);
  size_t off = 256;
  a.bucket = reinterpret_cast<uint64_t*>(ws + off);
  off += al256((size_t)l.n_events * 8);
  a.cell_end = reinterpret_cast<uint32_t*>(ws + off);
  off += al256((size_t)cells * 4);
  a.list1 = reinterpret_cast<uint32_t*>(ws + off);
  off += al256((size_t)cells * 4);
  a.list2 = reinterpret_cast<uint32_t*>(ws + off);
  off += al256((size_t)cells * 4);
  a.lane_key = reinterpret_cast<uint16_t*>(ws + off);
  off += al256((size_t)cells * 2);
  a.lane_cls = reinterpret_cast<uint32_t*>(ws + off);
  off += al256((size_t)2 * kClasses * 4);
  a.seg_w4 = reinterpret_cast<uint8_t*>(ws + off);
  const uint32_t* th = kde_thresholds();
  for (int t = 0; t < 64; ++t) a.theta[t] = th[t];

  hipLaunchKernelGGL(kde_clear_kernel, dim3(1), dim3(256), 0, st, a.counters, a.lane_cls, a.dev_status);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (cells == 0) return hipSuccess;

  // resident workgroups per kernel, cached per device
  static std::atomic<int> grids[64][8];
  int dev = 0;
  if ((e = hipGetDevice(&dev)) != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  int g[8];
  for (int i = 0; i < 8; ++i) g[i] = grids[dev][i].load();
  if (g[0] == 0) grids[dev][0].store(g[0] = resident(kde_scatter_kernel, kScatterThreads));
  if (g[1] == 0) grids[dev][1].store(g[1] = resident(kde_cell_kernel<0>, kWave));
  if (g[2] == 0) grids[dev][2].store(g[2] = resident(kde_cell_kernel<1>, kWave));
  if (g[3] == 0) grids[dev][3].store(g[3] = resident(kde_cell_kernel<2>, kWave));
  if (g[4] == 0) grids[dev][4].store(g[4] = resident(kde_lane_kernel<kLaneG>, kWave));
  if (g[5] == 0) grids[dev][5].store(g[5] = resident(kde_lane_kernel<kLaneGW>, kWave));
  if (g[6] == 0) grids[dev][6].store(g[6] = resident(kde_block_kernel, kBlockThreads));
  if (g[7] == 0) grids[dev][7].store(g[7] = resident(kde_scatter_staged_kernel, kStageThreads));
  for (int i = 0; i < 8; ++i)
    if (g[i] <= 0) return hipErrorInvalidDevice;
  if (l.n_kernels <= kStageK)
    hipLaunchKernelGGL(kde_scatter_staged_kernel, dim3(l.n_seg < g[7] ? l.n_seg : g[7]), dim3(kStageThreads), 0, st, a);
  else
    hipLaunchKernelGGL(kde_scatter_kernel, dim3(l.n_seg < g[0] ? l.n_seg : g[0]), dim3(kScatterThreads), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  // routing and the class order of the lane passes: contiguous ranges of
  // at least 16,384 cells per workgroup, at most 512 workgroups
  const int64_t route_wg = (cells + 16383) / 16384 < 512 ? (cells + 16383) / 16384 : 512;
  hipLaunchKernelGGL(kde_route_kernel, dim3((unsigned)route_wg), dim3(kRouteThreads), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(kde_lane_order_kernel, dim3((unsigned)route_wg), dim3(kRouteThreads), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const int64_t chunks = (cells + kWave - 1) / kWave;
  hipLaunchKernelGGL(kde_lane_kernel<kLaneG>, dim3(chunks < g[4] ? (int)chunks : g[4]), dim3(kWave), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(kde_lane_kernel<kLaneGW>, dim3(g[5]), dim3(kWave), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(kde_block_kernel, dim3(g[6]), dim3(kBlockThreads), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(kde_cell_kernel<0>, dim3(g[1]), dim3(kWave), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(kde_cell_kernel<1>, dim3(g[2]), dim3(kWave), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL(kde_cell_kernel<2>, dim3(g[3]), dim3(kWave), 0, st, a);
  return hipGetLastError();
}

}  // namespace argus
