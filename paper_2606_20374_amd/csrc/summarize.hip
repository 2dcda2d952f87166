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
//   structure-of-arrays events from HBM exactly once: 16-byte non-temporal
//   loads of four consecutive events per thread, software pipelined so the
//   next group is in flight while the current one is processed.
// * Per-kernel state is privatised in LDS: 64-bit sum, min and max, and a
//   WIN-bin window of the octave histogram anchored at the first duration
//   seen for that kernel (a lognormal mode spans two or three octaves; ten
//   bins also hold kernels whose positions run at 1x, 3x and 9x). Bins
//   outside the window go to a small pool of full 32-bin records that a
//   kernel claims on first need.
// * Keys (kernel ids, or (kernel id, stream) pairs as id * n_streams +
//   stream: section 5.2 groups per kernel and stream) map to LDS slots
//   directly when the key space fits (dense), or through an LDS key->slot
//   map that hands out slots on first sight (mapped), so a large, sparse key
//   space takes one pass per 16,384 keys.
// * Whenever the pool or the slots run out, the kernels concerned are
//   marked and redone exactly in another pass over the segment: the result
//   is exact for every input; typical traces need one pass.
// * Per-segment aggregates (valid/invalid counts, first start, last end,
//   busy time) are kept in registers and reduced once per segment; per-stream
//   busy time uses LDS atomics.
// * The flush writes each present cell once and the count of every cell
//   (0 for absent kernels); an absent cell's other fields are not written,
//   so a large, sparse key space costs 4 bytes per absent cell.
#include <atomic>

#include "argus_internal.h"

namespace argus {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef long long v2l __attribute__((ext_vector_type(2)));

constexpr int kThreads = 1024;
constexpr int kPool = 32;  // full 32-bin records per pass
constexpr uint32_t kBaseUnset = 0xFFu;
constexpr uint32_t kStNone = 0, kStBusy = 0xFE, kStPoison = 0xFF;
constexpr uint32_t kDone = 1u << 16;
constexpr int kMapIds = 16384;  // ids per pass in mapped mode
// Bound on the iterations of one claim wait, and on the passes over one key
// range that may end with a wait cut short. A claim's owner publishes after
// a fixed number of its own instructions, so no wait comes near the bound
// unless the code around it is compiled wrongly; the bounds make the kernel
// exit (and report) in that case instead of hanging.
constexpr int kSpinCap = 1 << 16;
constexpr int kMaxStuckPasses = 4;
constexpr uint32_t kMapEmpty = 0xFFFF, kMapBusy = 0xFFFE, kMapDefer = 0xFFFD, kMapDone = 0xFFFC;

// meta word of a slot: bits 0-7 window base bin (0xFF unset), bits 8-15
// full-record state (0 none, 1..kPool record index + 1, 0xFE being claimed,
// 0xFF pool exhausted: redo in another pass), bit 16 already written.
//
// map entry (mapped mode, 16 bits, two per 32-bit word): a slot index, or
// empty / being claimed / deferred to another pass / already written.

template <int NSLOT, int WIN, bool MAPPED>
struct Smem {
  unsigned long long sum[NSLOT];
  long long mm[NSLOT][2];  // min, max (one 16-byte read per event)
  uint32_t win[NSLOT][WIN];
  uint32_t meta[NSLOT];
  uint32_t pool[kPool][NB];
  unsigned long long stream_busy[ARGUS_MAX_STREAMS];
  uint32_t map[MAPPED ? kMapIds / 2 : 1];
  uint16_t slot_kid[MAPPED ? NSLOT : 1];
  unsigned long long red_busy, red_wire;
  long long red_first, red_last;
  uint32_t red_valid, red_invalid;
  uint32_t npool, poison, nslots, stuck;
};

struct Args {
  const int32_t* kernel_id;
  const int32_t* stream;
  const int64_t* start_ns;
  const int64_t* end_ns;
  const int64_t* seg_off;
  int64_t n_events;
  int32_t n_kernels, n_streams;
  int32_t key_ns;  // 0: cells keyed by kernel id; else n_streams: keyed by (kernel id, stream)
  int32_t n_keys;  // cells per segment: n_kernels, or n_kernels * n_streams
  int32_t vec_ok;  // event arrays 16-byte aligned: vector loads allowed
  int32_t n_seg;
  uint32_t* queue;  // next segment to take (zeroed before the launch)
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

template <int NSLOT, int WIN, bool MAPPED>
struct Seg {
  using S = Smem<NSLOT, WIN, MAPPED>;
  S& sm;

  __device__ __forceinline__ uint16_t map_get(int lk) const {
    return reinterpret_cast<const uint16_t*>(sm.map)[lk];
  }
  __device__ __forceinline__ void map_set(int lk, uint16_t v) { reinterpret_cast<uint16_t*>(sm.map)[lk] = v; }

  // Slot of local id lk, claiming one on first sight (mapped mode); -1 when
  // the id is already written or deferred to another pass. Lanes of one
  // wavefront may race for the same claim; the loop exits only when no
  // active lane is still pending, so a winner's publish executes inside the
  // loop, before a waiting lane of its own wavefront re-reads the entry.
  __device__ int map_claim(int lk, uint32_t e) {
    uint32_t* w = &sm.map[lk >> 1];
    const int sh = (lk & 1) * 16;
    int res = -2;
    // the trip count is the same for every lane (the loop exits on __any):
    // the bound costs one scalar register
    for (int it = 0;; ++it) {
      if (res == -2 && it >= kSpinCap) {
        // the wait is cut short: this event is dropped and the pass redone
        lds_store(&sm.stuck, 1u);
        res = -1;
      }
      if (res == -2) {
        if (e < (uint32_t)NSLOT) {
          res = (int)e;
        } else if (e == kMapDone || e == kMapDefer) {
          res = -1;
        } else if (e == kMapEmpty) {
          const uint32_t word = lds_load(w);
          if (((word >> sh) & 0xFFFFu) == kMapEmpty) {
            const uint32_t want = (word & ~(0xFFFFu << sh)) | (kMapBusy << sh);
            if (atomicCAS(w, word, want) == word) {
              const uint32_t s = atomicAdd(&sm.nslots, 1u);
              uint32_t fin;
              if (s < (uint32_t)NSLOT) {
                sm.slot_kid[s] = (uint16_t)lk;
                fin = s;
                res = (int)s;
              } else {
                fin = kMapDefer;
                lds_store(&sm.poison, 1u);
                res = -1;
              }
              // our half is BUSY and only we change it: flip it to fin
              atomicXor(w, (kMapBusy ^ fin) << sh);
            }
          }
          if (res == -2) e = (lds_load(w) >> sh) & 0xFFFFu;
        } else {  // being claimed by another lane
          e = (lds_load(w) >> sh) & 0xFFFFu;
        }
      }
      if (!__any(res == -2)) break;
    }
    return res;
  }

  // Count bin b outside the inline window in a full pool record, claiming
  // one for the slot on first need (same exit discipline as map_claim).
  __device__ void pool_add(int slot, uint32_t m, int b) {
    bool pending = true;
    for (int it = 0;; ++it) {
      if (pending && it >= kSpinCap) {
        lds_store(&sm.stuck, 1u);
        pending = false;
      }
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
            // only the state field changes (it is ours while BUSY)
            atomicXor(&sm.meta[slot], (fin ^ claim) & 0xFF00u);
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

  // mmv: min and max of the slot as read before this event (possibly stale:
  // min only falls and max only rises, so a stale read can only cause an
  // extra atomic, never a missed one)
  __device__ __forceinline__ void slot_add(int slot, uint32_t m, uint64_t d, const v2l& mmv) {
    if (m & kDone) return;
    const int b = octave_bin(d);
    if ((m & 0xFFu) == kBaseUnset) {
      int base = b - WIN / 2 + 1;
      base = base < 0 ? 0 : (base > NB - WIN ? NB - WIN : base);
      const uint32_t want = (m & ~0xFFu) | (uint32_t)base;
      const uint32_t old = atomicCAS(&sm.meta[slot], m, want);
      m = (old == m) ? want : old;
    }
    const int off = b - (int)(m & 0xFFu);
    if ((unsigned)off < (unsigned)WIN)
      atomicAdd(&sm.win[slot][off], 1u);
    else
      pool_add(slot, m, b);
    atomicAdd(&sm.sum[slot], (unsigned long long)d);
    if ((long long)d < mmv.x) atomicMin(&sm.mm[slot][0], (long long)d);
    if ((long long)d > mmv.y) atomicMax(&sm.mm[slot][1], (long long)d);
  }

  __device__ __forceinline__ void slot_reset(int s) {
    sm.sum[s] = 0;
    sm.mm[s][0] = INT64_MAX;
    sm.mm[s][1] = INT64_MIN;
#pragma unroll
    for (int w = 0; w < WIN; ++w) sm.win[s][w] = 0;
    sm.meta[s] = kBaseUnset;
  }
};

// Four events of one thread: validity and per-segment aggregates, then the
// per-kernel updates.
template <int NSLOT, int WIN, bool MAPPED>
__device__ __forceinline__ void process4(Seg<NSLOT, WIN, MAPPED>& sg, const Args& a, const int32_t (&kid)[4],
                                         const int32_t (&st)[4], const int64_t (&t0)[4], const int64_t (&t1)[4],
                                         int n, bool first_scan, int kb, int nk, uint32_t& nv, uint32_t& ni,
                                         unsigned long long& busy, long long& tf, long long& tl) {
  uint64_t d[4];
  int lk[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const bool valid =
        j < n && kid[j] >= 0 && kid[j] < a.n_kernels && st[j] >= 0 && st[j] < a.n_streams && t0[j] >= 0 && t1[j] >= t0[j];
    d[j] = (uint64_t)t1[j] - (uint64_t)t0[j];
    if (first_scan && j < n) {
      if (valid) {
        nv++;
        busy += d[j];
        tf = t0[j] < tf ? t0[j] : tf;
        tl = t1[j] > tl ? t1[j] : tl;
        atomicAdd(&sg.sm.stream_busy[st[j]], (unsigned long long)d[j]);
      } else {
        ni++;
      }
    }
    const uint32_t key = a.key_ns ? (uint32_t)kid[j] * (uint32_t)a.key_ns + (uint32_t)st[j] : (uint32_t)kid[j];
    lk[j] = valid && key - (uint32_t)kb < (uint32_t)nk ? (int)(key - (uint32_t)kb) : -1;
  }
  // per-kernel updates two events at a time: their LDS lookups are issued
  // together, and the live register set stays small enough that nothing
  // spills around the scan loop
#pragma unroll
  for (int h = 0; h < 4; h += 2) {
    int slot[2];
    if (MAPPED) {
      uint32_t e[2];
#pragma unroll
      for (int j = 0; j < 2; ++j) e[j] = lk[h + j] >= 0 ? sg.map_get(lk[h + j]) : kMapDone;
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        slot[j] = e[j] < (uint32_t)NSLOT ? (int)e[j] : -1;
        if (lk[h + j] >= 0 && e[j] >= (uint32_t)NSLOT && e[j] != kMapDone && e[j] != kMapDefer)
          slot[j] = sg.map_claim(lk[h + j], e[j]);
      }
    } else {
#pragma unroll
      for (int j = 0; j < 2; ++j) slot[j] = lk[h + j];
    }
    uint32_t m[2];
    v2l mmv[2];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      m[j] = slot[j] >= 0 ? sg.sm.meta[slot[j]] : 0u;
      mmv[j] = slot[j] >= 0 ? *reinterpret_cast<const v2l*>(&sg.sm.mm[slot[j]][0]) : v2l{0, 0};
    }
#pragma unroll
    for (int j = 0; j < 2; ++j)
      if (slot[j] >= 0) sg.slot_add(slot[j], m[j], d[h + j], mmv[j]);
  }
}

template <int NSLOT, int WIN, bool MAPPED>
__global__ __launch_bounds__(kThreads) void summarize_kernel(Args a) {
  __shared__ Smem<NSLOT, WIN, MAPPED> sm;
  __shared__ int64_t g_next;
  Seg<NSLOT, WIN, MAPPED> sg{sm};
  const int tid = threadIdx.x;
  const int32_t K = a.n_keys, NS = a.n_streams;

  // Persistent workgroups pull segments from a queue, so the output stores
  // of one segment drain while the loads of the next are already in flight.
  // Threads share only LDS state, so every barrier orders LDS alone: no
  // barrier waits for the outputs' stores.
  while (true) {
  if (tid == 0) g_next = (int64_t)atomicAdd(a.queue, 1u);
  lds_barrier();
  // the segment index is wave-uniform: keep it (and what derives from it:
  // bounds, loop limits) in scalar registers
  const int64_t g = (int64_t)__builtin_amdgcn_readfirstlane((int)g_next);
  if (g >= a.n_seg) break;

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

  // aligned part [a4, b4) in 4-event groups; head [lo, a4) and tail [b4, hi)
  int64_t a4 = lo, b4 = lo;
  if (a.vec_ok) {
    const int64_t up = (lo + 3) & ~(int64_t)3, dn = hi & ~(int64_t)3;
    a4 = up < hi ? up : hi;
    b4 = dn > a4 ? dn : a4;
  }
  const int64_t qa = a4 >> 2, qb = b4 >> 2;
  const v4i* K4 = reinterpret_cast<const v4i*>(a.kernel_id);
  const v4i* S4 = reinterpret_cast<const v4i*>(a.stream);
  const v2l* T0 = reinterpret_cast<const v2l*>(a.start_ns);
  const v2l* T1 = reinterpret_cast<const v2l*>(a.end_ns);

  uint32_t nv = 0, ni = 0;
  unsigned long long busy = 0, wire = 0;
  long long tf = INT64_MAX, tl = INT64_MIN;
  bool first_scan = true;
  int n_stuck = 0;  // passes of this segment that ended with a wait cut short
  constexpr int kRange = MAPPED ? kMapIds : NSLOT;

  for (int32_t kb = 0; kb < K; kb += kRange) {
    const int nk = K - kb < kRange ? K - kb : kRange;
    if (MAPPED)
      for (int i = tid; i < kMapIds / 2; i += kThreads) sm.map[i] = 0xFFFFFFFFu;
    else
      for (int s = tid; s < nk; s += kThreads) sg.slot_reset(s);
    while (true) {
      // mapped mode hands out slots afresh in every pass
      if (MAPPED)
        for (int s = tid; s < NSLOT; s += kThreads) sg.slot_reset(s);
      for (int i = tid; i < kPool * NB; i += kThreads) (&sm.pool[0][0])[i] = 0;
      if (tid == 0) {
        sm.npool = 0;
        sm.poison = 0;
        sm.nslots = 0;
        sm.stuck = 0;
      }
      lds_barrier();

      // unaligned head and tail: at most 3 events each, on the first threads
      if (a.vec_ok) {
        int32_t kid[4], st[4];
        int64_t t0[4], t1[4];
        int n = 0;
        const int64_t h = a4 - lo, t = hi - b4;
        const int64_t i = tid < h ? lo + tid : (tid - h < t ? b4 + (tid - h) : -1);
        if (i >= 0) {
          kid[0] = a.kernel_id[i];
          st[0] = a.stream[i];
          t0[0] = a.start_ns[i];
          t1[0] = a.end_ns[i];
          n = 1;
        }
        for (int j = n; j < 4; ++j) {
          kid[j] = -1;
          st[j] = 0;
          t0[j] = t1[j] = 0;
        }
        if (n) process4(sg, a, kid, st, t0, t1, n, first_scan, kb, nk, nv, ni, busy, tf, tl);
      }
      if (!a.vec_ok) {
        // scalar fallback for unaligned arrays: four strided events per thread
        for (int64_t i0 = lo + tid; i0 < hi; i0 += 4ll * kThreads) {
          int32_t kid[4], st[4];
          int64_t t0[4], t1[4];
          int n = 0;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const int64_t i = i0 + (int64_t)j * kThreads;  // in range for a prefix of j
            const bool in = i < hi;
            kid[j] = in ? a.kernel_id[i] : -1;
            st[j] = in ? a.stream[i] : 0;
            t0[j] = in ? a.start_ns[i] : 0;
            t1[j] = in ? a.end_ns[i] : 0;
            n += in;
          }
          process4(sg, a, kid, st, t0, t1, n, first_scan, kb, nk, nv, ni, busy, tf, tl);
        }
      }
      // aligned body: group q holds events 4q..4q+3; the next group's loads
      // are issued before the current group is processed
      {
        int64_t q = qa + tid;
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
          const int32_t kid[4] = {nk4.x, nk4.y, nk4.z, nk4.w};
          const int32_t st[4] = {ns4.x, ns4.y, ns4.z, ns4.w};
          const int64_t t0[4] = {na0.x, na0.y, na1.x, na1.y};
          const int64_t t1[4] = {nb0.x, nb0.y, nb1.x, nb1.y};
          const int64_t qn = q + kThreads;
          if (qn < qb) {
            nk4 = __builtin_nontemporal_load(K4 + qn);
            ns4 = __builtin_nontemporal_load(S4 + qn);
            na0 = __builtin_nontemporal_load(T0 + 2 * qn);
            na1 = __builtin_nontemporal_load(T0 + 2 * qn + 1);
            nb0 = __builtin_nontemporal_load(T1 + 2 * qn);
            nb1 = __builtin_nontemporal_load(T1 + 2 * qn + 1);
          }
          process4(sg, a, kid, st, t0, t1, 4, first_scan, kb, nk, nv, ni, busy, tf, tl);
          q = qn;
        }
      }
      first_scan = false;
      lds_barrier();

      // A claim wait cut short dropped an update: every kernel of this pass is
      // redone (the per-segment aggregates were complete in the first scan).
      // After kMaxStuckPasses such passes the results are flushed as they are
      // and the condition is reported.
      const bool stuck = sm.stuck != 0;
      const bool redo_pass = stuck && n_stuck < kMaxStuckPasses;
      if (stuck) {
        if (!redo_pass && tid == 0 && a.dev_status) atomicOr(a.dev_status, (int32_t)ARGUS_DEV_SUMMARY_STALLED);
        ++n_stuck;
      }

      // flush: the count of every slot; sum, min, max and wire size of the
      // present ones
      const int nslot = MAPPED ? (int)(sm.nslots < (uint32_t)NSLOT ? sm.nslots : NSLOT) : nk;
      for (int s = tid; s < (redo_pass ? 0 : nslot); s += kThreads) {
        const uint32_t m = sm.meta[s];
        const uint32_t pst = (m >> 8) & 0xFFu;
        if ((m & kDone) || pst == kStPoison) continue;
        uint32_t cnt = 0, nnz = 0;
#pragma unroll
        for (int w = 0; w < WIN; ++w) {
          cnt += sm.win[s][w];
          nnz += sm.win[s][w] != 0;
        }
        if (pst != kStNone) {
          for (int b = 0; b < NB; ++b) {
            cnt += sm.pool[pst - 1][b];
            nnz += sm.pool[pst - 1][b] != 0;
          }
        }
        const int64_t c = g * K + kb + (MAPPED ? (int)sm.slot_kid[s] : s);
        a.count[c] = cnt;
        if (cnt) {
          a.sum_ns[c] = (int64_t)sm.sum[s];
          a.min_ns[c] = sm.mm[s][0];
          a.max_ns[c] = sm.mm[s][1];
          wire += 33u + 5u * nnz;
        }
      }
      // flush: histograms of the present slots (their window base is set),
      // four bins per thread, 16-byte stores
      for (int it = tid; it < (redo_pass ? 0 : nslot) * (NB / 4); it += kThreads) {
        const int s = it >> 3, q = it & 7;
        const uint32_t m = sm.meta[s];
        const uint32_t pst = (m >> 8) & 0xFFu;
        const int base = (int)(m & 0xFFu);
        if ((m & kDone) || pst == kStPoison || base == (int)kBaseUnset) continue;
        uint32_t v[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int b = 4 * q + j;
          const int off = b - base;
          v[j] = (unsigned)off < (unsigned)WIN ? sm.win[s][off] : 0u;
          if (pst != kStNone) v[j] += sm.pool[pst - 1][b];
        }
        const int64_t c = g * K + kb + (MAPPED ? (int)sm.slot_kid[s] : s);
        *reinterpret_cast<uint4*>(a.hist + c * NB + 4 * q) = make_uint4(v[0], v[1], v[2], v[3]);
      }
      lds_barrier();
      const bool again = sm.poison != 0 || redo_pass;
      // mark what was written; kernels that ran out of room start over
      for (int s = tid; s < nslot; s += kThreads) {
        const uint32_t m = sm.meta[s];
        if (m & kDone) continue;
        const bool redo = redo_pass || ((m >> 8) & 0xFFu) == kStPoison;
        if (MAPPED) {
          sg.map_set(sm.slot_kid[s], redo ? (uint16_t)kMapEmpty : (uint16_t)kMapDone);
        } else if (redo) {
          sg.slot_reset(s);
        } else {
          sm.meta[s] = m | kDone;
        }
      }
      if (MAPPED)
        for (int i = tid; i < nk; i += kThreads)
          if (sg.map_get(i) == kMapDefer) sg.map_set(i, (uint16_t)kMapEmpty);
      lds_barrier();
      if (!again) break;
    }
    if (MAPPED) {
      // keys of this range that never occurred: count 0 (their other fields
      // are not written)
      for (int i = tid; i < nk; i += kThreads)
        if (sg.map_get(i) == kMapEmpty) a.count[g * K + kb + i] = 0;
      lds_barrier();
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
  lds_barrier();
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
  lds_barrier();
  }
}

// Workgroups resident at once (one per CU for the large tables): the grid
// of the persistent kernel. Cached per device and instantiation.
template <int NSLOT, int WIN, bool MAPPED>
int resident_groups() {
  static std::atomic<int> cache[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, summarize_kernel<NSLOT, WIN, MAPPED>, kThreads, 0) !=
        hipSuccess)
      return 0;
    v = cus * (per_cu > 0 ? per_cu : 1);
    cache[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

template <int NSLOT, int WIN, bool MAPPED>
hipError_t launch_t(const Args& args, int32_t n_seg, hipStream_t st) {
  const int groups = resident_groups<NSLOT, WIN, MAPPED>();
  if (groups <= 0) return hipErrorInvalidDevice;
  const int grid = n_seg < groups ? n_seg : groups;
  hipLaunchKernelGGL((summarize_kernel<NSLOT, WIN, MAPPED>), dim3(grid), dim3(kThreads), 0, st, args);
  return hipGetLastError();
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

hipError_t launch_summarize(const SummarizeLaunch& l, hipStream_t st) {
  const int32_t vec_ok =
      aligned16(l.kernel_id) && aligned16(l.stream) && aligned16(l.start_ns) && aligned16(l.end_ns) ? 1 : 0;
  const int32_t n_keys = l.keyed ? l.n_kernels * l.n_streams : l.n_kernels;
  Args a{l.kernel_id, l.stream, l.start_ns, l.end_ns, l.seg_off, l.n_events, l.n_kernels, l.n_streams,
         l.keyed ? l.n_streams : 0, n_keys, vec_ok, l.n_seg, l.queue, l.count, l.sum_ns, l.min_ns, l.max_ns, l.hist, l.n_valid, l.n_invalid, l.t_first, l.t_last,
         l.step_ns, l.busy_ns, l.stream_busy_ns, l.wire_bytes, l.dev_status};
  if (l.n_seg == 0) return hipSuccess;
  if (n_keys <= 64) return launch_t<64, 10, false>(a, l.n_seg, st);
  if (n_keys <= 512) return launch_t<512, 10, false>(a, l.n_seg, st);
  if (n_keys <= 2048) return launch_t<2048, 10, false>(a, l.n_seg, st);
  return launch_t<2048, 6, true>(a, l.n_seg, st);
}

}  // namespace argus
