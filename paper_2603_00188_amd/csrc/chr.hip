// Numerator of the cache hit rate (Eq. chr of the paper): per (unit,
// sequence), the number of tokens two retained sets share, |I_keep cap I*|.
// Both sets arrive as the kept lists stlite_select_topk writes: strictly
// ascending absolute token indices, B_s per sequence.
//
// A work-group takes one 65,536-token span of one sequence for one unit: it
// finds each list's entries inside the span by binary search, marks the
// second list's tokens in an 8 KB LDS bitmap and counts the first list's
// tokens found there; span counts are added into hits, which a fill kernel
// zeroes first.  Entries outside their span are skipped, so lists that break
// the ordering contract give a wrong count, never an out-of-range access.
#include "stlite_internal.h"

namespace stlite {
namespace {

constexpr int32_t kSpan = 1 << 16;
constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void overlap_zero_kernel(int32_t* hits, int32_t n) {
  const int32_t i = int32_t(blockIdx.x) * kThreads + threadIdx.x;
  if (i < n) hits[i] = 0;
}

// First index in list[0, n) whose token is >= x.
__device__ inline int32_t lower_bound(const int32_t* list, int32_t n, int32_t x) {
  int32_t lo = 0, hi = n;
  while (lo < hi) {
    const int32_t mid = (lo + hi) >> 1;
    if (list[mid] < x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// Grid: x = sequence * spans_per_seq + span (spans_per_seq: of the longest
// sequence), y = unit.
__global__ __launch_bounds__(kThreads) void kept_overlap_kernel(OverlapArgs a) {
  __shared__ uint32_t bits[kSpan / 32];
  __shared__ int32_t range[4];
  __shared__ int32_t partial[kThreads / 64];
  const Layout& lay = a.lay;
  const int32_t s = int32_t(blockIdx.x) / a.spans_per_seq, c = int32_t(blockIdx.x) - s * a.spans_per_seq;
  const int unit = blockIdx.y;
  const int32_t seq0 = lay.cu_seqlens[s], L = lay.cu_seqlens[s + 1] - seq0;
  if (int64_t(c) * kSpan >= L) return;
  const int32_t t0 = seq0 + c * kSpan, t1 = seq0 + int32_t(min(int64_t(L), int64_t(c + 1) * kSpan));
  const int32_t k0 = lay.cu_budget[s], n = lay.cu_budget[s + 1] - k0;
  const int32_t* A = a.kept_a + size_t(unit) * lay.total_budget + k0;
  const int32_t* B = a.kept_b + size_t(unit) * lay.total_budget + k0;
  for (int i = threadIdx.x; i < kSpan / 32; i += kThreads) bits[i] = 0;
  if (threadIdx.x < 4) range[threadIdx.x] = lower_bound(threadIdx.x < 2 ? A : B, n, (threadIdx.x & 1) ? t1 : t0);
  __syncthreads();
  for (int32_t i = range[2] + threadIdx.x; i < range[3]; i += kThreads) {
    const int32_t t = B[i] - t0;
    if (t >= 0 && t < kSpan) atomicOr(&bits[t >> 5], 1u << (t & 31));
  }
  __syncthreads();
  int32_t cnt = 0;
  for (int32_t i = range[0] + threadIdx.x; i < range[1]; i += kThreads) {
    const int32_t t = A[i] - t0;
    if (t >= 0 && t < kSpan) cnt += (bits[t >> 5] >> (t & 31)) & 1u;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o);
  if ((threadIdx.x & 63) == 0) partial[threadIdx.x >> 6] = cnt;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t total = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) total += partial[w];
    if (total) atomicAdd(&a.hits[size_t(unit) * lay.n_seqs + s], total);
  }
}

}  // namespace

hipError_t launch_kept_overlap(const OverlapArgs& a, hipStream_t stream) {
  const int32_t n = a.lay.n_units * a.lay.n_seqs;
  hipLaunchKernelGGL(overlap_zero_kernel, dim3((n + kThreads - 1) / kThreads), dim3(kThreads), 0, stream, a.hits, n);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kept_overlap_kernel, dim3(unsigned(a.lay.n_seqs * a.spans_per_seq), a.lay.n_units),
                     dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace stlite
