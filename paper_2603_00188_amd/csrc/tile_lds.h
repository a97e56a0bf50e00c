// 64-key tiles of bf16 key rows staged in LDS by direct global->LDS DMA
// (global_load_lds_dwordx4: lane j of a wave-load lands at LDS base + 16 j, no
// VGPRs involved), shared by the window-score and rho GEMM kernels.
//
// Layout: 64 keys x 256 bytes, no padding.  The 16-byte chunk c (dims 8c..8c+7)
// of local key k sits at slot c ^ (k & 15), so that the MFMA B-operand read --
// sixteen consecutive keys, one chunk each -- touches sixteen different bank
// groups.
#pragma once

#include "stlite_internal.h"

namespace stlite {

typedef __attribute__((address_space(3))) void* lds_void_t;

constexpr int kTileKeys = 64;
constexpr int kTileElems = kTileKeys * kHeadDim;  // 16 KB of bf16

// Issue the DMA of keys first .. first+63 of `rows` ([.][128] bf16) into `tile`;
// key indices past `last_valid` repeat key `last_valid`.  Every wave issues
// 16 / NW wave-loads (4 keys each); wait for them with wait_vmcnt (and a
// barrier for the other waves' rows) before reading the tile.  The LDS
// address reaches the instruction through an opaque copy: the compiler then
// inserts none of its own (full) waits before tile reads, which it would
// otherwise add wherever it cannot count the loads still in flight.
template <int NW>
__device__ inline void tile_dma(const uint16_t* rows, int32_t first, int32_t last_valid, uint16_t* tile) {
  constexpr int kLoads = 16 / NW;
  // The wave index selects the LDS rows through M0: keep it scalar.
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
#pragma unroll
  for (int m = 0; m < kLoads; ++m) {
    const int grp = wave * kLoads + m;
    const int kl = grp * 4 + (lane >> 4);
    const int chunk = (lane & 15) ^ (kl & 15);
    const int32_t key = min(first + kl, last_valid);
    uint32_t dst = uint32_t(reinterpret_cast<uintptr_t>(tile + grp * 4 * kHeadDim));
    asm volatile("" : "+s"(dst));
    __builtin_amdgcn_global_load_lds(rows + size_t(key) * kHeadDim + chunk * 8, (lds_void_t)(uintptr_t)dst, 16, 0, 0);
  }
}

// 16x16x32 MFMA B operand for sub-tile t and k-step kk: lane l supplies dims
// 32 kk + 8 (l >> 4) .. +7 of key 16 t + (l & 15).
__device__ inline bf16x8_t tile_b_operand(const uint16_t* tile, int t, int kk) {
  const int lane = threadIdx.x & 63;
  const int key = t * 16 + (lane & 15);
  const int chunk = kk * 4 + (lane >> 4);
  return *reinterpret_cast<const bf16x8_t*>(tile + key * kHeadDim + ((chunk ^ (key & 15)) << 3));
}

// Wait until at most N of this wave's vector-memory operations are outstanding.
template <int N>
__device__ inline void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Work-group barrier without the memory fence of __syncthreads, which would
// wait for every outstanding global load -- including the tile DMA that is
// meant to stay in flight.  Pending LDS reads and writes are completed first.
__device__ inline void barrier_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

}  // namespace stlite
