// Integrated score and flat top-B (Eq. modal_scoring and Sec. integrated
// scoring of the paper), for every (unit, sequence) segment at once:
//   S = A on text tokens, S = M * (A + alpha * Phi) on visual tokens,
//   I_keep = the B tokens first in (S descending, index ascending) order,
//   written in ascending token order.
// The selection is the segmented radix select of segsel.h on the keys
// ~order_key(S) (ascending key = descending S).
#include "segsel.h"
#include "stlite_internal.h"

namespace stlite {
namespace {

constexpr int kMaxChunkFrames = 64;

// Sequence table of the selection: n = L_s, k = B_s.
__global__ __launch_bounds__(64) void select_plan_kernel(SelectArgs a) {
  if (threadIdx.x != 0) return;
  SeqInfo* info = a.info;
  const Layout& lay = a.lay;
  int32_t cb = 0;
  for (int32_t q = 0; q < lay.n_seqs; ++q) {
    const int32_t n = lay.cu_seqlens[q + 1] - lay.cu_seqlens[q];
    info[q] = SeqInfo{n, lay.cu_budget[q + 1] - lay.cu_budget[q], cb, 0};
    cb += (n + kSegChunk - 1) / kSegChunk;
  }
  info[lay.n_seqs] = SeqInfo{0, 0, cb, 0};
}

// Does token `tok` (absolute) lie in one of the sequence's frames f0 .. f1-1?
__device__ inline bool is_visual_search(const Layout& lay, int32_t f0, int32_t f1, int32_t tok) {
  int32_t lo = f0, hi = f1 - 1, hit = -1;
  while (lo <= hi) {  // last frame with offset <= tok
    const int32_t mid = (lo + hi) >> 1;
    if (lay.frame_meta[3 * mid] <= tok) { hit = mid; lo = mid + 1; } else { hi = mid - 1; }
  }
  return hit >= 0 && tok < lay.frame_meta[3 * hit] + lay.frame_meta[3 * hit + 1] * lay.frame_meta[3 * hit + 2];
}

// Scores, order keys and the level-0 histogram of one 4096-token chunk.
__global__ __launch_bounds__(kSegThreads) void select_keys_kernel(SelectArgs a) {
  const SegSel& s = a.sel;
  __shared__ uint32_t lh[kSegBins];
  __shared__ int32_t fr_lo[kMaxChunkFrames], fr_hi[kMaxChunkFrames];
  __shared__ int32_t nfr;
  const Layout& lay = a.lay;
  const int unit = blockIdx.y;
  const ChunkRef cr = seg_chunk(s, blockIdx.x);
  const int32_t seq_start = lay.cu_seqlens[cr.seq];
  const int32_t t_begin = seq_start + cr.begin, t_end = seq_start + cr.end;
  const int32_t f0 = lay.cu_frames[cr.seq], f1 = lay.cu_frames[cr.seq + 1];
  seg_hist_zero(lh);
  if (threadIdx.x == 0) {
    // frames overlapping [t_begin, t_end), in order; -1 if there are too many
    int32_t lo = f0, hi = f1 - 1, first = f1;
    while (lo <= hi) {  // first frame that ends after t_begin
      const int32_t mid = (lo + hi) >> 1;
      const int32_t end = lay.frame_meta[3 * mid] + lay.frame_meta[3 * mid + 1] * lay.frame_meta[3 * mid + 2];
      if (end > t_begin) { first = mid; hi = mid - 1; } else { lo = mid + 1; }
    }
    int32_t n = 0;
    for (int32_t f = first; f < f1 && lay.frame_meta[3 * f] < t_end; ++f) {
      if (n == kMaxChunkFrames) { n = -1; break; }
      fr_lo[n] = lay.frame_meta[3 * f];
      fr_hi[n] = lay.frame_meta[3 * f] + lay.frame_meta[3 * f + 1] * lay.frame_meta[3 * f + 2];
      ++n;
    }
    nfr = n;
  }
  __syncthreads();
  const int32_t n_fr = nfr;
  const size_t ubase = size_t(unit) * lay.total_tokens;
  uint32_t* keys = seg_keys(s, unit, cr.seq);
#pragma unroll 4
  for (int j = 0; j < kSegPer; ++j) {
    const int32_t i = cr.begin + j * kSegThreads + threadIdx.x;
    const bool in = i < cr.end;
    uint32_t key = 0;
    if (in) {
      const int32_t tok = seq_start + i;
      bool visual = false;
      if (n_fr >= 0) {
        for (int32_t f = 0; f < n_fr; ++f) visual |= (tok >= fr_lo[f]) & (tok < fr_hi[f]);
      } else {
        visual = is_visual_search(lay, f0, f1, tok);
      }
      const float A = a.a_base[ubase + tok];
      float S = A;
      if (visual) {
        const float x = a.phi ? fmaf(a.alpha, a.phi[ubase + tok], A) : A;
        S = (a.gate && a.gate[ubase + tok] == 0) ? 0.0f : x;
      }
      if (a.score) a.score[ubase + tok] = S;
      key = ~order_key(S);
      keys[i] = key;
    }
    seg_hist_add(lh, in, key >> 21);
  }
  __syncthreads();
  seg_hist_flush(lh, seg_hist(s, unit, cr.seq, 0));
}

// Kept token indices, ascending, at cu_budget[seq] + rank.
__global__ __launch_bounds__(kSegThreads) void select_emit_kernel(SelectArgs a) {
  const SegSel& s = a.sel;
  __shared__ int32_t scratch[kSegThreads / 64];
  const Layout& lay = a.lay;
  const int unit = blockIdx.y;
  const ChunkRef cr = seg_chunk(s, blockIdx.x);
  TakeChunk tc;
  take_chunk(s, unit, cr, scratch, tc);
  const int32_t seq_start = lay.cu_seqlens[cr.seq];
  const int32_t kb = lay.cu_budget[cr.seq], B = lay.cu_budget[cr.seq + 1] - kb;
  int32_t* kept = a.kept + size_t(unit) * lay.total_budget + kb;
  const int32_t i0 = cr.begin + threadIdx.x * kSegPer;
#pragma unroll
  for (int i = 0; i < kSegPer; ++i)
    if (tc.take[i] && tc.pos[i] < B) kept[tc.pos[i]] = seq_start + i0 + i;
}

}  // namespace

hipError_t launch_select(const SelectArgs& a, hipStream_t stream) {
  const SegSel& s = a.sel;
  const int32_t U = a.lay.n_units;
  hipLaunchKernelGGL(select_plan_kernel, dim3(1), dim3(64), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_segsel_zero(s, U, stream);
  if (e != hipSuccess) return e;
  const dim3 chunk_grid(s.chunks_per_unit, U);
  if (s.chunks_per_unit > 0) {
    hipLaunchKernelGGL(select_keys_kernel, chunk_grid, dim3(kSegThreads), 0, stream, a);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  e = launch_segsel_middle(s, U, stream);
  if (e != hipSuccess || s.chunks_per_unit == 0) return e;
  hipLaunchKernelGGL(select_emit_kernel, chunk_grid, dim3(kSegThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace stlite
