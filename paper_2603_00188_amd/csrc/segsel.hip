// Generic middle passes of the segmented k-smallest selection (segsel.h):
// pivots, refining histograms, per-chunk counts and per-segment offsets.
#include <algorithm>

#include "segsel.h"

namespace stlite {
namespace {

constexpr int kShift[3] = {21, 10, 0};
constexpr int kBins[3] = {2048, 2048, 1024};

// Find the bin of level LEVEL that holds the k_rem-th key of the current
// prefix and narrow the prefix to it.  One work-group per segment.
template <int LEVEL>
__global__ __launch_bounds__(kSegThreads) void seg_pivot_kernel(SegSel s) {
  __shared__ int32_t scratch[kSegThreads / 64];
  const int32_t seq = blockIdx.x;
  const int unit = blockIdx.y;
  SegState* stp = &s.state[size_t(unit) * s.n_seqs + seq];
  SegState st;
  if (LEVEL == 0) {
    const int32_t k = s.info[seq].k;
    st = SegState{0u, 0u, k, k};
  } else {
    st = *stp;
  }
  __syncthreads();  // every thread has read the state before it is rewritten
  if (st.k <= 0) {
    if (LEVEL == 0 && threadIdx.x == 0) *stp = st;
    return;
  }
  constexpr int per = kBins[LEVEL] / kSegThreads;
  const uint32_t* h = seg_hist(s, unit, seq, LEVEL) + threadIdx.x * per;
  int32_t c[per];
  int32_t local = 0;
#pragma unroll
  for (int j = 0; j < per; ++j) {
    c[j] = int32_t(h[j]);
    local += c[j];
  }
  int32_t total;
  int32_t before = seg_block_exscan(local, scratch, &total);
#pragma unroll
  for (int j = 0; j < per; ++j) {
    if (before < st.k_rem && st.k_rem <= before + c[j]) {
      const uint32_t bin = uint32_t(threadIdx.x * per + j);
      SegState out;
      out.prefix = st.prefix | (bin << kShift[LEVEL]);
      out.mask = st.mask | (uint32_t(kBins[LEVEL] - 1) << kShift[LEVEL]);
      out.k_rem = st.k_rem - before;
      out.k = st.k;
      *stp = out;
    }
    before += c[j];
  }
}

// Histogram of the level-LEVEL digit over the keys that match the prefix.
template <int LEVEL>
__global__ __launch_bounds__(kSegThreads) void seg_refine_kernel(SegSel s) {
  __shared__ uint32_t lh[kSegBins];
  const int unit = blockIdx.y;
  const ChunkRef cr = seg_chunk(s, blockIdx.x);
  const SegState st = s.state[size_t(unit) * s.n_seqs + cr.seq];
  if (st.k <= 0 || cr.begin >= cr.end) return;
  seg_hist_zero(lh);
  __syncthreads();
  const uint32_t* keys = seg_keys(s, unit, cr.seq);
#pragma unroll 4
  for (int j = 0; j < kSegPer; ++j) {
    const int32_t i = cr.begin + j * kSegThreads + threadIdx.x;
    uint32_t key = 0;
    bool pred = false;
    if (i < cr.end) {
      key = keys[i];
      pred = (key & st.mask) == st.prefix;
    }
    seg_hist_add(lh, pred, (key >> kShift[LEVEL]) & uint32_t(kBins[LEVEL] - 1));
  }
  __syncthreads();
  seg_hist_flush(lh, seg_hist(s, unit, cr.seq, LEVEL));
}

// Keys below and equal to the exact pivot T, per chunk.
__global__ __launch_bounds__(kSegThreads) void seg_count_kernel(SegSel s) {
  __shared__ int32_t scratch[kSegThreads / 64];
  const int unit = blockIdx.y;
  const ChunkRef cr = seg_chunk(s, blockIdx.x);
  const SegState st = s.state[size_t(unit) * s.n_seqs + cr.seq];
  int32_t less = 0, eq = 0;
  if (st.k > 0) {
    const uint32_t* keys = seg_keys(s, unit, cr.seq);
    for (int j = 0; j < kSegPer; ++j) {
      const int32_t i = cr.begin + j * kSegThreads + threadIdx.x;
      if (i < cr.end) {
        const uint32_t key = keys[i];
        less += key < st.prefix ? 1 : 0;
        eq += key == st.prefix ? 1 : 0;
      }
    }
  }
  int32_t tl, te;
  seg_block_exscan(less, scratch, &tl);
  seg_block_exscan(eq, scratch, &te);
  if (threadIdx.x == 0) s.counts[size_t(unit) * s.chunks_per_unit + blockIdx.x] = SegCount{tl, te};
}

// Per segment: where each chunk's selected keys start in the output, and how
// many keys equal to T precede the chunk (lowest index first among ties).
__global__ __launch_bounds__(64) void seg_offsets_kernel(SegSel s) {
  const int32_t seq = blockIdx.x;
  const int unit = blockIdx.y;
  if (threadIdx.x != 0) return;
  const SegState st = s.state[size_t(unit) * s.n_seqs + seq];
  if (s.pivot_value)
    s.pivot_value[size_t(unit) * s.n_seqs + seq] = st.k > 0 ? order_key_value(st.prefix) : __builtin_nanf("");
  const int32_t c0 = s.info[seq].chunk_begin, c1 = s.info[seq + 1].chunk_begin;
  const SegCount* cnt = s.counts + size_t(unit) * s.chunks_per_unit;
  SegOffset* off = s.offsets + size_t(unit) * s.chunks_per_unit;
  int32_t out = 0, eq_before = 0;
  for (int32_t c = c0; c < c1; ++c) {
    off[c] = SegOffset{out, eq_before};
    const SegCount k = cnt[c];
    const int32_t eq_taken = min(max(st.k_rem - eq_before, 0), k.eq);
    out += k.less + eq_taken;
    eq_before += k.eq;
  }
}

__global__ __launch_bounds__(256) void seg_zero_kernel(SegSel s, size_t words) {
  for (size_t i = size_t(blockIdx.x) * blockDim.x + threadIdx.x; i < words; i += size_t(gridDim.x) * blockDim.x)
    s.hist[i] = 0u;
}

}  // namespace

hipError_t launch_segsel_zero(const SegSel& s, int32_t n_units, hipStream_t stream) {
  const size_t words = size_t(n_units) * s.n_seqs * 3 * kSegBins;
  const unsigned blocks = unsigned(std::min<size_t>((words + 255) / 256, 4096));
  hipLaunchKernelGGL(seg_zero_kernel, dim3(blocks), dim3(256), 0, stream, s, words);
  return hipGetLastError();
}

hipError_t launch_segsel_middle(const SegSel& s, int32_t n_units, hipStream_t stream) {
  const dim3 seg_grid(s.n_seqs, n_units), chunk_grid(s.chunks_per_unit, n_units);
#define STLITE_LAUNCH(kernel, grid, block)                                   \
  do {                                                                       \
    hipLaunchKernelGGL(kernel, grid, dim3(block), 0, stream, s);             \
    const hipError_t e = hipGetLastError();                                  \
    if (e != hipSuccess) return e;                                           \
  } while (0)
  // With no keys at all (no segment has a chunk) only the per-segment passes
  // run, so that every segment still gets its state and pivot value.
  const bool keys = s.chunks_per_unit > 0;
  STLITE_LAUNCH(seg_pivot_kernel<0>, seg_grid, kSegThreads);
  if (keys) STLITE_LAUNCH(seg_refine_kernel<1>, chunk_grid, kSegThreads);
  STLITE_LAUNCH(seg_pivot_kernel<1>, seg_grid, kSegThreads);
  if (keys) STLITE_LAUNCH(seg_refine_kernel<2>, chunk_grid, kSegThreads);
  STLITE_LAUNCH(seg_pivot_kernel<2>, seg_grid, kSegThreads);
  if (keys) STLITE_LAUNCH(seg_count_kernel, chunk_grid, kSegThreads);
  STLITE_LAUNCH(seg_offsets_kernel, seg_grid, 64);
#undef STLITE_LAUNCH
  return hipSuccess;
}

}  // namespace stlite
