// Mean-Attention base prior (the paper's appendix on the base scoring
// function): the window-aggregated A_base of Eq. base_attention averaged along
// each sequence's token axis over a centred window of `width` positions,
// positions outside the sequence counting as 0, divided by width:
//   A_mean[i] = (1/width) * sum_{j = i - r .. i + r, j in the sequence} A_base[j],
//   r = (width - 1) / 2.
//
// Bandwidth-bound: a work-group takes kMeanTile outputs of one unit, stages
// them plus r halo values on each side in LDS with coalesced loads, and each
// thread sums its outputs' windows from LDS in ascending order (lanes read
// consecutive LDS words, no bank conflicts); a thread tracks its outputs'
// sequence with one binary search over cu_seqlens, then forward steps.
#include "stlite_internal.h"

namespace stlite {
namespace {

constexpr int kMeanThreads = 256;
constexpr int kMeanTile = 2048;       // outputs per work-group
constexpr int kMeanPer = kMeanTile / kMeanThreads;

// Grid: x = 2048-token tile of the packed token axis, y = unit.
__global__ __launch_bounds__(kMeanThreads) void mean_attention_kernel(const float* __restrict__ a_base,
                                                                      float* __restrict__ a_mean, Layout lay,
                                                                      int32_t radius) {
  __shared__ float sh[kMeanTile + 2 * kMeanMaxRadius];
  const int32_t L = int32_t(lay.total_tokens);
  const int32_t t0 = int32_t(blockIdx.x) * kMeanTile;
  const float* src = a_base + size_t(blockIdx.y) * size_t(L);
  float* dst = a_mean + size_t(blockIdx.y) * size_t(L);
  const int32_t first = t0 - radius;  // token held by sh[0]
  const int32_t span = kMeanTile + 2 * radius;
  for (int32_t j = threadIdx.x; j < span; j += kMeanThreads) {
    const int32_t t = first + j;
    sh[j] = (t >= 0 && t < L) ? src[t] : 0.0f;
  }
  __syncthreads();
  const float w = float(2 * radius + 1);
  int32_t s = -1, s0 = 0, s1 = 0;
#pragma unroll 1
  for (int e = 0; e < kMeanPer; ++e) {
    const int32_t i = t0 + int32_t(threadIdx.x) + e * kMeanThreads;
    if (i >= L) break;
    if (s < 0) {  // last sequence starting at or before i (empty ones are skipped)
      int32_t lo = 0, hi = lay.n_seqs - 1;
      while (lo < hi) {
        const int32_t mid = (lo + hi + 1) >> 1;
        if (lay.cu_seqlens[mid] <= i) lo = mid; else hi = mid - 1;
      }
      s = lo;
      s0 = lay.cu_seqlens[s];
      s1 = lay.cu_seqlens[s + 1];
    }
    while (i >= s1) {
      ++s;
      s0 = lay.cu_seqlens[s];
      s1 = lay.cu_seqlens[s + 1];
    }
    const int32_t lo = max(i - radius, s0), hi = min(i + radius, s1 - 1);
    float acc = 0.0f;
    for (int32_t t = lo; t <= hi; ++t) acc += sh[t - first];
    dst[i] = acc / w;
  }
}

}  // namespace

hipError_t launch_mean_attention(const float* a_base, float* a_mean, const Layout& lay, int32_t width,
                                 hipStream_t stream) {
  if (lay.total_tokens == 0 || lay.n_units == 0) return hipSuccess;
  const unsigned tiles = unsigned((lay.total_tokens + kMeanTile - 1) / kMeanTile);
  hipLaunchKernelGGL(mean_attention_kernel, dim3(tiles, unsigned(lay.n_units)), dim3(kMeanThreads), 0, stream,
                     a_base, a_mean, lay, (width - 1) / 2);
  return hipGetLastError();
}

}  // namespace stlite
