// Work-group-wide radix select and ordered scans on 32-bit order keys, used by
// the TSG gate (k-th smallest rho) and by the flat top-B (k-th largest S).
// One work-group of kSelThreads threads owns one (unit, sequence) segment.
#pragma once

#include "stlite_internal.h"

namespace stlite {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;

struct SelectShared {
  uint32_t hist[256];
  int32_t wave_tot[kSelWaves];
  int32_t wave_tot2[kSelWaves];
  uint32_t prefix;
  int32_t k;
};

// hist[digit] += 1 for every lane with pred, aggregating the lanes of a wave
// that share a digit (up to two rounds) before the per-lane LDS atomics, so
// that long runs of equal keys do not serialise on one LDS address.
__device__ __forceinline__ void hist_add(uint32_t* hist, bool pred, uint32_t digit) {
  const int lane = threadIdx.x & 63;
  uint64_t act = __ballot(pred);
#pragma unroll
  for (int round = 0; round < 2; ++round) {
    if (act == 0) break;
    const int leader = __ffsll((unsigned long long)act) - 1;
    const uint32_t ld = __shfl(digit, leader);
    const uint64_t same = __ballot(pred && digit == ld);
    if (lane == leader) atomicAdd(&hist[ld], uint32_t(__popcll(same)));
    if (pred && digit == ld) pred = false;
    act &= ~same;
  }
  if (pred) atomicAdd(&hist[digit], 1u);
}

// Inclusive scan of x over the work-group (all kSelThreads threads call it).
// Returns the inclusive prefix; *total receives the group total.
__device__ __forceinline__ int32_t block_inclusive_scan(int32_t x, int32_t* wave_tot, int32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t y = __shfl_up(x, off);
    if (lane >= off) x += y;
  }
  if (lane == 63) wave_tot[wave] = x;
  __syncthreads();
  int32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kSelWaves; ++w) {
    const int32_t t = wave_tot[w];
    before += (w < wave) ? t : 0;
    all += t;
  }
  __syncthreads();
  *total = all;
  return x + before;
}

// Exact k-th smallest key (1 <= k <= n) of keys[0..n) by four 8-bit digit
// passes.  Returns the key value T; *need receives how many keys equal to T
// belong to the k smallest (the lowest-index ones are taken by the caller).
__device__ inline uint32_t block_radix_select(const uint32_t* keys, int32_t n, int32_t k, SelectShared& sh,
                                              int32_t* need) {
  const int tid = threadIdx.x, lane = tid & 63;
  uint32_t prefix = 0, mask = 0;
  for (int shift = 24; shift >= 0; shift -= 8) {
    for (int i = tid; i < 256; i += kSelThreads) sh.hist[i] = 0;
    __syncthreads();
    for (int32_t base = 0; base < n; base += kSelThreads) {
      const int32_t i = base + tid;
      uint32_t key = 0;
      bool pred = false;
      if (i < n) {
        key = keys[i];
        pred = (key & mask) == prefix;
      }
      hist_add(sh.hist, pred, (key >> shift) & 255u);
    }
    __syncthreads();
    if (tid < 64) {
      // lane owns bins 4*lane .. 4*lane+3
      uint32_t c[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = sh.hist[4 * lane + j];
      int32_t local = int32_t(c[0] + c[1] + c[2] + c[3]);
      int32_t incl = local;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int32_t y = __shfl_up(incl, off);
        if (lane >= off) incl += y;
      }
      int32_t before = incl - local;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (before < k && k <= before + int32_t(c[j])) {
          sh.prefix = prefix | (uint32_t(4 * lane + j) << shift);
          sh.k = k - before;
        }
        before += int32_t(c[j]);
      }
    }
    __syncthreads();
    prefix = sh.prefix;
    k = sh.k;
    mask |= 255u << shift;
    __syncthreads();
  }
  *need = k;
  return prefix;
}

}  // namespace stlite
