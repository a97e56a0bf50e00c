// Component-centric Spatial Saliency (Eq. css_calc of the paper):
//   H_{u,v} = mean over the in-grid Moore neighbours n of cos(h_{u,v}, h_n),
//   Phi = 1 - H  (0 when a frame is 1x1; 0 on text tokens).
//
// A work-group stages an 8 x 16 tile of a frame's patch grid plus its one-cell
// halo (10 x 18 keys, 49 KB) in LDS, computes the 180 inverse norms once, and
// then gives each interior cell to 16 lanes: every lane keeps 8 dimensions of
// the centre key and, for each neighbour, adds rn_n * (its 8-dimension partial
// dot), so one 16-lane reduction per cell yields sum_n cos * ||centre||.
// Each key is read from HBM once per tile; halo re-reads hit L2.
#include "stlite_internal.h"

namespace stlite {
namespace {

constexpr int kTU = 8, kTV = 16;
constexpr int kHU = kTU + 2, kHV = kTV + 2;
constexpr int kCells = kHU * kHV;
constexpr int kCStride = kHeadDim + 8;

__device__ inline float dot8(uint4 a, uint4 b) {
  float s = 0.0f;
  s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.x), __builtin_bit_cast(bf16x2_t, b.x), s, false);
  s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.y), __builtin_bit_cast(bf16x2_t, b.y), s, false);
  s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.z), __builtin_bit_cast(bf16x2_t, b.z), s, false);
  s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a.w), __builtin_bit_cast(bf16x2_t, b.w), s, false);
  return s;
}

__global__ __launch_bounds__(256) void css_kernel(CssArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t cells[kCells * kCStride];
  __shared__ float rn[kCells];
  const Layout& lay = a.lay;
  const int f = blockIdx.x, split = blockIdx.y, unit = blockIdx.z;
  const int32_t off = lay.frame_meta[3 * f], R = lay.frame_meta[3 * f + 1], C = lay.frame_meta[3 * f + 2];
  const int32_t ntx = (C + kTV - 1) / kTV, nty = (R + kTU - 1) / kTU;
  const uint16_t* kframe = a.k + (size_t(unit) * lay.total_tokens + off) * kHeadDim;
  float* out = a.phi + size_t(unit) * lay.total_tokens + off;
  const int tid = threadIdx.x, group = tid >> 4, gl = tid & 15;

  for (int32_t t = split; t < nty * ntx; t += a.splits) {
    const int32_t u0 = (t / ntx) * kTU, v0 = (t % ntx) * kTV;
    __syncthreads();
    for (int i = tid; i < kCells * 16; i += blockDim.x) {
      const int cell = i >> 4, part = i & 15;
      const int32_t u = u0 - 1 + cell / kHV, v = v0 - 1 + cell % kHV;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (u >= 0 && u < R && v >= 0 && v < C)
        val = *reinterpret_cast<const uint4*>(kframe + size_t(u * C + v) * kHeadDim + part * 8);
      *reinterpret_cast<uint4*>(cells + cell * kCStride + part * 8) = val;
    }
    __syncthreads();
    for (int cell = group; cell < kCells; cell += 16) {
      const uint4 x = *reinterpret_cast<const uint4*>(cells + cell * kCStride + gl * 8);
      float ss = dot8(x, x);
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) ss += __shfl_xor(ss, o);
      if (gl == 0) rn[cell] = ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f;
    }
    __syncthreads();
    for (int ic = group; ic < kTU * kTV; ic += 16) {
      const int iu = ic / kTV, iv = ic % kTV;
      const int32_t u = u0 + iu, v = v0 + iv;
      const int centre = (iu + 1) * kHV + (iv + 1);
      const uint4 cx = *reinterpret_cast<const uint4*>(cells + centre * kCStride + gl * 8);
      float acc = 0.0f;
      int cnt = 0;
#pragma unroll
      for (int du = -1; du <= 1; ++du)
#pragma unroll
        for (int dv = -1; dv <= 1; ++dv) {
          if (du == 0 && dv == 0) continue;
          const int32_t uu = u + du, vv = v + dv;
          if (uu < 0 || uu >= R || vv < 0 || vv >= C) continue;
          const int nb = centre + du * kHV + dv;
          const uint4 nx = *reinterpret_cast<const uint4*>(cells + nb * kCStride + gl * 8);
          acc = fmaf(dot8(cx, nx), rn[nb], acc);
          ++cnt;
        }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) acc += __shfl_xor(acc, o);
      if (gl == 0 && u < R && v < C) out[u * C + v] = cnt > 0 ? 1.0f - acc * rn[centre] / float(cnt) : 0.0f;
    }
  }
}

// phi = 0 on every text token (the gaps between and after the frames).
__global__ __launch_bounds__(256) void css_text_kernel(CssArgs a) {
  const Layout& lay = a.lay;
  const int s = blockIdx.x, unit = blockIdx.y;
  float* out = a.phi + size_t(unit) * lay.total_tokens;
  const int32_t f0 = lay.cu_frames[s], f1 = lay.cu_frames[s + 1];
  int32_t prev = lay.cu_seqlens[s];
  for (int32_t f = f0; f <= f1; ++f) {
    const int32_t off = f < f1 ? lay.frame_meta[3 * f] : lay.cu_seqlens[s + 1];
    for (int32_t j = prev + threadIdx.x; j < off; j += blockDim.x) out[j] = 0.0f;
    if (f < f1) prev = off + lay.frame_meta[3 * f + 1] * lay.frame_meta[3 * f + 2];
  }
}

}  // namespace

hipError_t launch_css(const CssArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(css_text_kernel, dim3(a.lay.n_seqs, a.lay.n_units), dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.lay.n_frames == 0) return e;
  hipLaunchKernelGGL(css_kernel, dim3(a.lay.n_frames, a.splits, a.lay.n_units), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace stlite
