// Block-wide selection helpers shared by the cross-rank kernels: exact MSD
// radix selection of order statistics among register-resident keys, and the
// block-size dispatch that keeps those keys in registers.
#pragma once

#include <type_traits>

#include "argus_internal.h"

namespace argus {

// hist[bin] += 1 for every active lane. Each of ROUNDS rounds counts all
// active lanes sharing the first remaining lane's bin with one atomic (the
// bin is read with readlane, no LDS round trip); the rest add individually.
// Must be reached by every lane of the wavefront.
template <int ROUNDS = 2>
__device__ __forceinline__ void hist_add(uint32_t* hist, uint32_t bin, bool active) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int it = 0; it < ROUNDS; ++it) {
    const unsigned long long act = __ballot(active);
    if (act == 0) return;
    const int leader = __ffsll((long long)act) - 1;
    const uint32_t lb = __builtin_amdgcn_readlane(bin, leader);
    const bool mine = active && bin == lb;
    const unsigned long long same = __ballot(mine);
    // the leader's own bin (equal to lb) as the address: a divergent address
    // keeps the compiler from wrapping the single-lane atomic in another
    // wave-wide aggregation of its own
    if (lane == leader) atomicAdd(&hist[bin], (uint32_t)__popcll(same));
    if (mine) active = false;
  }
  if (active) atomicAdd(&hist[bin], 1u);
}

// Shared state of a selection of T ranks with DB-bit digits (2^DB bins per
// target); at most 16 wavefronts per block.
template <int T, int DB = 8>
struct SelShared {
  uint32_t hist[T][1 << DB];
  uint32_t wave_tot[T * 16];
  uint32_t digit[T], before[T];
};

// MSD radix select of the ranks k[0..T) among the valid register keys of
// the whole block of NT >= 256 threads (bit j of vm: key[j] valid), all keys
// <= range, DB bits per pass (wider digits: fewer passes over the keys, each
// with a larger histogram to clear and scan), HR aggregation rounds per
// histogram add. Every thread of the block must call it.
template <int NT, int V, int T, int DB = 8, int HR = 2, typename KeyT>
__device__ void select_ranks(const KeyT (&key)[V], uint64_t vm, uint64_t range, const uint32_t (&k)[T],
                             uint64_t (&out)[T], SelShared<T, DB>& sh) {
  constexpr int NB = 1 << DB;
  constexpr int BPT = NB > NT ? NB / NT : 1;  // bins per scanning thread
  constexpr int NSCAN = NB / BPT;             // scanning threads
  static_assert(NT >= 256 && NT <= 1024 && NB % NSCAN == 0, "block size and digit width");
  uint64_t prefix[T];
  uint32_t kk[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    prefix[t] = 0;
    kk[t] = k[t];
  }
  if (range != 0) {
    const int nbits = 64 - __builtin_clzll(range);
    const int passes = (nbits + DB - 1) / DB;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    for (int p = passes - 1; p >= 0; --p) {
      const int shift = p * DB;
      const bool top = p == passes - 1;
      for (int i = tid; i < T * NB; i += NT) (&sh.hist[0][0])[i] = 0;
      __syncthreads();
      // targets with equal prefixes share one histogram: rep[t] is the first
      int rep[T];
#pragma unroll
      for (int t = 0; t < T; ++t) {
        rep[t] = t;
#pragma unroll
        for (int q = T - 1; q >= 0; --q)
          if (q < t && prefix[q] == prefix[t]) rep[t] = q;
      }
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const uint64_t kj = (uint64_t)key[j];
        const bool ok = (vm >> j) & 1u;
        const uint32_t digit = (uint32_t)(kj >> shift) & (uint32_t)(NB - 1);
        const uint64_t hi = top || shift + DB >= 64 ? 0 : kj >> (shift + DB);
#pragma unroll
        for (int t = 0; t < T; ++t)
          if (rep[t] == t) hist_add<HR>(sh.hist[t], digit, ok && (top || hi == prefix[t]));
      }
      __syncthreads();
      // per-target inclusive scan over the bins, BPT consecutive bins per
      // scanning thread
      uint32_t h[T][BPT], v[T];
      if (tid < NSCAN) {
#pragma unroll
        for (int t = 0; t < T; ++t) {
          uint32_t sum = 0;
#pragma unroll
          for (int b = 0; b < BPT; ++b) {
            h[t][b] = sh.hist[rep[t]][tid * BPT + b];
            sum += h[t][b];
          }
          v[t] = sum;
          for (int o = 1; o < 64; o <<= 1) {
            const uint32_t n = __shfl_up(v[t], o, 64);
            if (lane >= o) v[t] += n;
          }
          if (lane == 63) sh.wave_tot[t * 16 + w] = v[t];
        }
      }
      __syncthreads();
      if (tid < NSCAN) {
#pragma unroll
        for (int t = 0; t < T; ++t) {
          uint32_t run = v[t];
          for (int ww = 0; ww < w; ++ww) run += sh.wave_tot[t * 16 + ww];
#pragma unroll
          for (int b = BPT - 1; b >= 0; --b) run -= h[t][b];
          // run: bins before this thread's first bin
#pragma unroll
          for (int b = 0; b < BPT; ++b) {
            if (run <= kk[t] && kk[t] < run + h[t][b]) {
              sh.digit[t] = (uint32_t)(tid * BPT + b);
              sh.before[t] = run;
            }
            run += h[t][b];
          }
        }
      }
      __syncthreads();
#pragma unroll
      for (int q = 0; q < T; ++q) {
        prefix[q] = DB >= 64 ? sh.digit[q] : (prefix[q] << DB) | sh.digit[q];
        kk[q] -= sh.before[q];
      }
      __syncthreads();
    }
  }
#pragma unroll
  for (int t = 0; t < T; ++t) out[t] = prefix[t];
}

// Call f(std::integral_constant<int, NT>, std::integral_constant<int, V>)
// with a block size NT and the smallest instantiated per-thread count V such
// that NT * V >= n (n <= 16384): at most 24 values per thread stay in
// registers without spilling.
template <typename F>
void dispatch_block(int n, F&& f) {
  using std::integral_constant;
  auto pick = [&](auto nt) {
    constexpr int NT = decltype(nt)::value;
    const int v = (n + NT - 1) / NT;
    if (v <= 1) return f(nt, integral_constant<int, 1>{});
    if (v <= 2) return f(nt, integral_constant<int, 2>{});
    if (v <= 4) return f(nt, integral_constant<int, 4>{});
    if (v <= 8) return f(nt, integral_constant<int, 8>{});
    if (v <= 12) return f(nt, integral_constant<int, 12>{});
    if (v <= 16) return f(nt, integral_constant<int, 16>{});
    if (v <= 20) return f(nt, integral_constant<int, 20>{});
    return f(nt, integral_constant<int, 24>{});
  };
  if (n <= 24 * 256) return pick(integral_constant<int, 256>{});
  if (n <= 24 * 512) return pick(integral_constant<int, 512>{});
  return pick(integral_constant<int, 1024>{});
}


}  // namespace argus
