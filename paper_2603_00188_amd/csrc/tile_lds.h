// 64-key tiles of bf16 key rows staged in LDS by direct memory->LDS DMA
// (buffer_load_dwordx4 ... lds: lane j of a wave-load lands at LDS base + 16 j, no
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
// Buffer descriptor flags of a raw (unswizzled, stride 0) buffer on gfx950.
constexpr int kBufferFlags = 0x00020000;

// DMA of 64-key tiles: keys first .. first+63 of `rows` ([.][128] bf16) into
// an LDS tile; key indices past `last_valid` repeat key `last_valid`.  A tile
// is 16 wave-loads of 4 keys; wave w of NW issues wave-loads w, w + NW, ...
// (16 / NW of them when NW divides 16).  Wait for them with wait_vmcnt (and a
// barrier for the other waves' rows) before reading the tile.
//
// The loads are buffer loads with the LDS bit (MUBUF encoding): the compiler
// tracks them with the vector-memory counter only, so LDS reads issued while
// they are in flight keep exact lgkmcnt waits (the flat-encoded global->LDS
// form makes it wait for every LDS read instead).  The buffer's range ends at
// key last_valid, so no load can reach past it.  Per-lane byte offsets are
// computed once; a wave-load costs a clamp and an add.  The LDS address
// reaches the instruction through an opaque copy: the compiler then inserts
// none of its own (full) waits before tile reads, which it would otherwise
// add wherever it cannot count the loads still in flight.
template <int NW>
struct TileDma {
  static constexpr int kLoads = (16 + NW - 1) / NW;
  uint32_t row[kLoads];    // local key * 256 (the clamped part)
  uint32_t chunk[kLoads];  // swizzled 16-byte slot * 16

  // The wave index selects the LDS rows through M0: keep it scalar.
  __device__ static int wave() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }
  __device__ static int group(int m) { return min(wave() + m * NW, 15); }

  __device__ TileDma() {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int m = 0; m < kLoads; ++m) {
      const int kl = group(m) * 4 + (lane >> 4);
      row[m] = uint32_t(kl) * (kHeadDim * 2);
      chunk[m] = uint32_t((lane & 15) ^ (kl & 15)) * 16u;
    }
  }

  // The descriptor covers keys first .. min(first + 63, last_valid) only (at
  // most 16 KB), so offsets stay small whatever the sequence length.
  __device__ void issue(const uint16_t* rows, int32_t first, int32_t last_valid, uint16_t* tile) const {
    const int32_t n_valid = min(last_valid - first + 1, kTileKeys);
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint16_t*>(rows + size_t(first) * kHeadDim), 0, n_valid * (kHeadDim * 2), kBufferFlags);
    const uint32_t bound = uint32_t(n_valid - 1) * (kHeadDim * 2);
#pragma unroll
    for (int m = 0; m < kLoads; ++m) {
      if (16 % NW != 0 && wave() + m * NW >= 16) break;
      const uint32_t off = min(row[m], bound) + chunk[m];
      uint32_t dst = uint32_t(reinterpret_cast<uintptr_t>(tile)) + uint32_t(group(m) * 4 * kHeadDim * 2);
      asm volatile("" : "+s"(dst));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t)(uintptr_t)dst, 16, off, 0, 0, 0);
    }
  }
};

// 16x16x32 MFMA B operand for sub-tile t and k-step kk: lane l supplies dims
// 32 kk + 8 (l >> 4) .. +7 of key 16 t + (l & 15).
__device__ inline bf16x8_t tile_b_operand(const uint16_t* tile, int t, int kk) {
  const int lane = threadIdx.x & 63;
  const int key = t * 16 + (lane & 15);
  const int chunk = kk * 4 + (lane >> 4);
  return *reinterpret_cast<const bf16x8_t*>(tile + key * kHeadDim + ((chunk ^ (key & 15)) << 3));
}

// 32x32x16 MFMA B operand for key block kb (keys 32 kb .. 32 kb + 31) and
// k-step kk: lane l supplies dims 16 kk + 8 (l >> 5) .. +7 of key 32 kb + (l & 31).
// Each group of 16 consecutive lanes reads one chunk of 16 consecutive keys:
// sixteen different slots, so the read is bank-conflict free.
__device__ inline bf16x8_t tile_b32_operand(const uint16_t* tile, int kb, int kk) {
  const int lane = threadIdx.x & 63;
  const int key = kb * 32 + (lane & 31);
  const int chunk = kk * 2 + (lane >> 5);
  return *reinterpret_cast<const bf16x8_t*>(tile + key * kHeadDim + ((chunk ^ (key & 15)) << 3));
}

// Row of register i of a 32x32 MFMA accumulator held by lane l (its column
// is l & 31): rows come in groups of four, alternating between the two lane
// halves.
__device__ inline int acc32_row(int i, int lane) { return (i & 3) + 4 * (lane >> 5) + 8 * (i >> 2); }

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
