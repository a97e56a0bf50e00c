// Segmented exact k-smallest selection on 32-bit order keys, spread over the
// whole GPU.  A segment is one (unit, sequence) pair; its n keys live at
// keys[unit * total_tokens + cu_seqlens[seq] + i], i < n, and it selects the k
// keys first in (key ascending, index ascending) order.  Used by the TSG gate
// (rho ascending) and by the flat top-B (S descending, as inverted keys).
//
// Passes (each over 4096-key chunks, grid = chunks x units, except pivot and
// offsets which run one work-group per segment):
//   keys + level-0 histogram (call-specific producer, uses hist_chunk)
//   pivot<0>   refine<1>   pivot<1>   refine<2>   pivot<2>   -> exact T, need
//   count      (keys < T, keys == T per chunk)
//   offsets    (per segment: output offset and equal-key rank base per chunk)
//   emit       (call-specific consumer, uses take_chunk)
// Level digits: bits 31..21, 20..10, 9..0 (2048, 2048, 1024 bins).
#pragma once

#include "stlite_internal.h"

namespace stlite {

constexpr int kSegThreads = 256;
constexpr int kSegPer = kSegChunk / kSegThreads;  // 16 keys per thread
constexpr int kSegBins = 2048;

struct ChunkRef {
  int32_t seq, c, begin, end;  // sequence, chunk index within it, key range [begin, end) within the segment
};

__device__ inline ChunkRef seg_chunk(const SegSel& s, int32_t x) {
  int32_t lo = 0, hi = s.n_seqs - 1;
  while (lo < hi) {  // last sequence whose chunk_begin <= x
    const int32_t mid = (lo + hi + 1) >> 1;
    if (s.info[mid].chunk_begin <= x) lo = mid; else hi = mid - 1;
  }
  ChunkRef r;
  r.seq = lo;
  r.c = x - s.info[lo].chunk_begin;
  r.begin = r.c * kSegChunk;
  r.end = min(r.begin + kSegChunk, s.info[lo].n);
  return r;
}

__device__ inline uint32_t* seg_keys(const SegSel& s, int unit, int32_t seq) {
  return s.keys + size_t(unit) * s.total_tokens + s.cu_seqlens[seq];
}

__device__ inline uint32_t* seg_hist(const SegSel& s, int unit, int32_t seq, int level) {
  return s.hist + ((size_t(unit) * s.n_seqs + seq) * 3 + level) * kSegBins;
}

// hist[digit] += 1 for every lane with pred; lanes of a wave that share a
// digit are aggregated (two rounds) before the per-lane LDS atomics, so long
// runs of equal keys do not serialise on one LDS address.
__device__ __forceinline__ void seg_hist_add(uint32_t* hist, bool pred, uint32_t digit) {
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

__device__ __forceinline__ void seg_hist_zero(uint32_t* lh) {
  for (int i = threadIdx.x; i < kSegBins; i += blockDim.x) lh[i] = 0;
}

// Add a work-group's LDS histogram into the segment's global one.
__device__ __forceinline__ void seg_hist_flush(const uint32_t* lh, uint32_t* gh) {
  for (int i = threadIdx.x; i < kSegBins; i += blockDim.x) {
    const uint32_t v = lh[i];
    if (v) atomicAdd(&gh[i], v);
  }
}

// Exclusive scan over the work-group (kSegThreads threads); *total gets the sum.
__device__ __forceinline__ int32_t seg_block_exscan(int32_t x, int32_t* scratch, int32_t* total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int32_t incl = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int32_t y = __shfl_up(incl, off);
    if (lane >= off) incl += y;
  }
  if (lane == 63) scratch[wave] = incl;
  __syncthreads();
  int32_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kSegThreads / 64; ++w) {
    const int32_t t = scratch[w];
    before += (w < wave) ? t : 0;
    all += t;
  }
  __syncthreads();
  *total = all;
  return before + incl - x;
}

// Per-chunk selection flags for the emit pass.  Thread t owns keys
// begin + 16 t .. begin + 16 t + 15 (in index order); take[i] tells whether
// key i is selected and pos[i] its rank among the segment's selected keys.
struct TakeChunk {
  bool take[kSegPer];
  int32_t pos[kSegPer];
};

__device__ inline void take_chunk(const SegSel& s, int unit, const ChunkRef& cr, int32_t* scratch, TakeChunk& out) {
  const SegState st = s.state[size_t(unit) * s.n_seqs + cr.seq];
  const SegOffset off = s.offsets[size_t(unit) * s.chunks_per_unit + s.info[cr.seq].chunk_begin + cr.c];
  const uint32_t T = st.prefix;
  const int32_t need = st.k_rem;
  const uint32_t* keys = seg_keys(s, unit, cr.seq);
  const int32_t i0 = cr.begin + threadIdx.x * kSegPer;
  uint32_t key[kSegPer];
  int32_t n_eq = 0;
#pragma unroll
  for (int i = 0; i < kSegPer; ++i) {
    const bool in = i0 + i < cr.end;
    key[i] = in ? keys[i0 + i] : 0xffffffffu;
    n_eq += (in && st.k > 0 && key[i] == T) ? 1 : 0;
  }
  int32_t eq_tot;
  int32_t eq_rank = off.eq_before + seg_block_exscan(n_eq, scratch, &eq_tot);
  int32_t n_take = 0;
#pragma unroll
  for (int i = 0; i < kSegPer; ++i) {
    const bool in = i0 + i < cr.end;
    bool t = false;
    if (in && st.k > 0) {
      if (key[i] < T) t = true;
      else if (key[i] == T) t = eq_rank++ < need;
    }
    out.take[i] = t;
    n_take += t ? 1 : 0;
  }
  int32_t take_tot;
  int32_t p = off.out + seg_block_exscan(n_take, scratch, &take_tot);
#pragma unroll
  for (int i = 0; i < kSegPer; ++i) {
    out.pos[i] = p;
    p += out.take[i] ? 1 : 0;
  }
}

// Zero the segments' histograms (before the producer pass).
hipError_t launch_segsel_zero(const SegSel& s, int32_t n_units, hipStream_t stream);
// Launch the generic middle passes (pivots, refines, count, offsets).
hipError_t launch_segsel_middle(const SegSel& s, int32_t n_units, hipStream_t stream);

}  // namespace stlite
