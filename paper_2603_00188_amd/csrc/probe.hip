// Matrix-core and HBM read throughput probes (measurement only; see stlite_probe.h).
#include <type_traits>

#include "stlite_probe.h"
#include "stlite_internal.h"

namespace stlite {
namespace {

constexpr int kProbeThreads = 256;
constexpr int kProbeElems = 128;  // bf16 operand elements per lane: 8 A + 8 B fragments of 8

template <int SHAPE>
__global__ __launch_bounds__(kProbeThreads, 2) void probe_mfma_kernel(const uint16_t* ops, float* sink,
                                                                      int32_t iters) {
  const size_t lane_id = size_t(blockIdx.x) * kProbeThreads + threadIdx.x;
  const uint16_t* src = ops + lane_id * kProbeElems;
  bf16x8_t a[8], b[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(src + 8 * i));
    b[i] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4*>(src + 64 + 8 * i));
  }
  float s = 0.0f;
  if constexpr (SHAPE == 0) {
    f32x4_t acc[4] = {};
    for (int32_t it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[j & 3] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[j], b[7 - j], acc[j & 3], 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) s += acc[j][i];
  } else if constexpr (SHAPE == 2) {
    // The window score's instruction mix: two 32-key blocks in turn, each
    // MFMA followed by fma + exp2 + add on two finished logits of the other
    // block, in a fixed order (as in the score passes).
    f32x16_t acc[2] = {};
    float sum[16] = {};
    auto body = [&](auto kb_c) {
      constexpr int kb = decltype(kb_c)::value;
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        acc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[kk], b[(kk + 4 * kb) & 7], kk == 0 ? f32x16_t{} : acc[kb],
                                                          0, 0, 0);
        float sc = 0.125f;
        asm volatile("" : "+s"(sc));
        sum[2 * kk] += __builtin_amdgcn_exp2f(fmaf(acc[kb ^ 1][2 * kk], sc, -1.0f));
        sum[2 * kk + 1] += __builtin_amdgcn_exp2f(fmaf(acc[kb ^ 1][2 * kk + 1], sc, -1.0f));
        asm volatile("" ::"v"(sum[2 * kk]), "v"(sum[2 * kk + 1]));
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    for (int32_t it = 0; it < iters; it += 2) {
      body(std::integral_constant<int, 0>{});
      if (it + 1 < iters) body(std::integral_constant<int, 1>{});
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) s += sum[i] + acc[0][i] + acc[1][i];
  } else if constexpr (SHAPE == 3) {
    // The same vector work per matrix-core cycle on 16x16x32 MFMAs: two
    // accumulator sets of four 16x16 blocks, each MFMA pair followed by
    // fma + exp2 + add on two finished results of the other set.
    f32x4_t acc[2][4] = {};
    float sum[8] = {};
    auto body = [&](auto h_c) {
      constexpr int h = decltype(h_c)::value;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
#pragma unroll
        for (int p = 0; p < 2; ++p) {
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const int blk = 2 * p + t;
            acc[h][blk] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[(2 * kk + p) & 7], b[(kk + 2 * t + 4 * h) & 7],
                                                                  kk == 0 ? f32x4_t{} : acc[h][blk], 0, 0, 0);
          }
          float sc = 0.125f;
          asm volatile("" : "+s"(sc));
          const int e = 2 * kk + p;  // 0 .. 7: two results of block e / 2 of the other set
          sum[e] += __builtin_amdgcn_exp2f(fmaf(acc[h ^ 1][e >> 1][2 * (e & 1)], sc, -1.0f)) +
                    __builtin_amdgcn_exp2f(fmaf(acc[h ^ 1][e >> 1][2 * (e & 1) + 1], sc, -1.0f));
          asm volatile("" ::"v"(sum[e]));
          __builtin_amdgcn_sched_barrier(0);
        }
    };
    for (int32_t it = 0; it < iters; it += 2) {
      body(std::integral_constant<int, 0>{});
      if (it + 1 < iters) body(std::integral_constant<int, 1>{});
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) s += sum[i];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i) s += acc[0][j][i] + acc[1][j][i];
  } else {
    f32x16_t acc[2] = {};
    for (int32_t it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 8; ++j)
        acc[j & 1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[j], b[7 - j], acc[j & 1], 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int i = 0; i < 16; ++i) s += acc[j][i];
  }
  sink[lane_id] = s;
}

typedef uint32_t probe_u32x4_t __attribute__((ext_vector_type(4)));

// Streams n16 16-byte words once: each lane reads words i, i + stride, ...
// four at a time (all four loads issued before they are combined), with the
// default cache policy or non-temporal loads.  The XOR of what a lane read
// goes to the sink, so no load can be dropped.
template <bool NT>
__global__ __launch_bounds__(kProbeThreads) void probe_read_kernel(const probe_u32x4_t* src, size_t n16, float* sink) {
  const size_t stride = size_t(gridDim.x) * kProbeThreads;
  size_t i = size_t(blockIdx.x) * kProbeThreads + threadIdx.x;
  probe_u32x4_t acc = {0u, 0u, 0u, 0u};
  for (; i + 3 * stride < n16; i += 4 * stride) {
    probe_u32x4_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = NT ? __builtin_nontemporal_load(src + i + u * stride) : src[i + u * stride];
#pragma unroll
    for (int u = 0; u < 4; ++u) acc ^= v[u];
  }
  for (; i < n16; i += stride) acc ^= NT ? __builtin_nontemporal_load(src + i) : src[i];
  sink[size_t(blockIdx.x) * kProbeThreads + threadIdx.x] = __uint_as_float(acc.x ^ acc.y ^ acc.z ^ acc.w);
}

}  // namespace
}  // namespace stlite

extern "C" stlite_status stlite_probe_read(const void* src, size_t bytes, float* sink, int32_t n_groups,
                                           int32_t nontemporal, void* stream) {
  using namespace stlite;
  if (!src || !sink || n_groups < 1 || bytes == 0 || bytes % 16 != 0 ||
      reinterpret_cast<uintptr_t>(src) % 16 != 0)
    return STLITE_ERR_INVALID_ARG;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const probe_u32x4_t* words = static_cast<const probe_u32x4_t*>(src);
  if (nontemporal)
    hipLaunchKernelGGL(probe_read_kernel<true>, dim3(n_groups), dim3(kProbeThreads), 0, st, words, bytes / 16, sink);
  else
    hipLaunchKernelGGL(probe_read_kernel<false>, dim3(n_groups), dim3(kProbeThreads), 0, st, words, bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? STLITE_OK : STLITE_ERR_HIP;
}

extern "C" stlite_status stlite_probe_mfma(stlite_probe_shape shape, const uint16_t* operands, float* sink,
                                           int32_t n_groups, int32_t iters, void* stream) {
  using namespace stlite;
  if ((shape != STLITE_PROBE_MFMA_16X16X32_BF16 && shape != STLITE_PROBE_MFMA_32X32X16_BF16 &&
       shape != STLITE_PROBE_MFMA_32X32X16_BF16_EXP2 && shape != STLITE_PROBE_MFMA_16X16X32_BF16_EXP2) ||
      !operands || !sink || n_groups < 1 || iters < 1)
    return STLITE_ERR_INVALID_ARG;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (shape == STLITE_PROBE_MFMA_16X16X32_BF16)
    hipLaunchKernelGGL(probe_mfma_kernel<0>, dim3(n_groups), dim3(kProbeThreads), 0, st, operands, sink, iters);
  else if (shape == STLITE_PROBE_MFMA_32X32X16_BF16)
    hipLaunchKernelGGL(probe_mfma_kernel<1>, dim3(n_groups), dim3(kProbeThreads), 0, st, operands, sink, iters);
  else if (shape == STLITE_PROBE_MFMA_32X32X16_BF16_EXP2)
    hipLaunchKernelGGL(probe_mfma_kernel<2>, dim3(n_groups), dim3(kProbeThreads), 0, st, operands, sink, iters);
  else
    hipLaunchKernelGGL(probe_mfma_kernel<3>, dim3(n_groups), dim3(kProbeThreads), 0, st, operands, sink, iters);
  return hipGetLastError() == hipSuccess ? STLITE_OK : STLITE_ERR_HIP;
}
