// The procedure over a layer's concatenated key space (the problem setup's
// K^(l) in R^{L x D}, D = H_kv * d): token t's keys of every kv head form one
// D-dimensional key h_t; CSS and TSG take their cosines over D, A is the mean
// over all the layer's query heads, and one kept set per layer serves every
// kv head.  Outputs of this file are per layer: [n_layers][total_tokens].
//
//   layer_mean_kernel  A_layer = mean over the kv heads of the per-head A
//                      (each already the mean over its query heads)
//   cat_norms_kernel   1/||h_j|| of the current frames' keys
//   rho_cat_kernel     rho = max over the current frame of cos(h_i, h_j): a
//                      dense N_hist x N_cur x D contraction on the matrix cores,
//                      historical rows resident as A operands (2 blocks of 16
//                      per wave, 4 H k-steps each), current keys streamed
//                      through a two-stage LDS ring in 32-key tiles of all heads
//   css_cat_kernel     Phi over the 3 x 3 Moore neighbourhood of h: a wave owns
//                      2 output rows (1 at four heads) x 16 columns and walks
//                      the neighbour rows head by head, accumulating each
//                      pair's dot product over the heads before scaling by the
//                      norms
#include <algorithm>

#include "stlite_internal.h"
#include "tile_lds.h"

namespace stlite {
namespace {

constexpr float kCatSnap = 1.0f - 1.0e-4f;
constexpr int kCatKeys = 32;   // current keys per rho tile
constexpr int kCatRows = 128;  // historical rows per rho work-group (half a 256-row block)

__device__ inline float sumsq8(uint4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j)
    s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, w[j]), __builtin_bit_cast(bf16x2_t, w[j]), s, false);
  return s;
}

__device__ inline float inv_norm(float ss) { return ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f; }

__device__ inline int32_t frame_size(const Layout& lay, int32_t f) {
  return lay.frame_meta[3 * f + 1] * lay.frame_meta[3 * f + 2];
}

__global__ __launch_bounds__(256) void layer_mean_kernel(const float* a_base, float* a_layer, int32_t n_layers,
                                                         int32_t H, int64_t L) {
  const int64_t n = int64_t(n_layers) * L;
  const float inv = 1.0f / float(H);
  for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) {
    const int64_t l = i / L, t = i - l * L;
    float s = 0.0f;
    for (int32_t h = 0; h < H; ++h) s += a_base[(l * H + h) * L + t];
    a_layer[i] = s * inv;
  }
}

// rn[layer][token] = 1/||h|| over the current frame of every sequence with a
// history.  Work-group (x, seq, layer): keys 64 x .. 64 x + 63, 16 lanes per key.
template <int H>
__global__ __launch_bounds__(256) void cat_norms_kernel(RhoArgs a) {
  const int s = blockIdx.y, layer = blockIdx.z;
  const Layout& lay = a.lay;
  const int32_t f0 = lay.cu_frames[s], f1 = lay.cu_frames[s + 1];
  if (f1 - f0 < 2) return;
  const int32_t off = lay.frame_meta[3 * (f1 - 1)];
  const int32_t n = min(frame_size(lay, f1 - 1), int32_t(blockIdx.x + 1) * 64);
  const size_t head_stride = size_t(lay.total_tokens) * kHeadDim;
  const uint16_t* klayer = a.k + size_t(layer) * H * head_stride;
  float* rn = a.rn_cur + size_t(layer) * lay.total_tokens;
  const int group = threadIdx.x >> 4, gl = threadIdx.x & 15;
  for (int32_t j = int32_t(blockIdx.x) * 64 + group; j < n; j += blockDim.x >> 4) {
    float ss = 0.0f;
#pragma unroll
    for (int h = 0; h < H; ++h)
      ss += sumsq8(*reinterpret_cast<const uint4*>(klayer + h * head_stride + size_t(off + j) * kHeadDim + gl * 8));
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) ss += __shfl_xor(ss, o);
    if (gl == 0) rn[off + j] = inv_norm(ss);
  }
}

// Grid: x = 2 * (256-row historical blocks), y = layer.  Tile layout in LDS:
// [head][32 keys][128 dims], the 16-byte chunk c of key k at slot c ^ (k & 15).
template <int H>
__global__ __launch_bounds__(256, 2) void rho_cat_kernel(RhoArgs a) {
  constexpr int kSteps = 4 * H;
  constexpr int kTile = H * kCatKeys * kHeadDim;
  __shared__ __attribute__((aligned(16))) uint16_t st0[kTile], st1[kTile];
  __shared__ int32_t tok_s[kCatRows];
  __shared__ float rnrow_s[kCatRows];
  const Layout& lay = a.lay;
  const int layer = blockIdx.y;
  const HistBlock hb = a.blocks[blockIdx.x >> 1];
  const int32_t row0 = hb.hb * kRhoRows + int32_t(blockIdx.x & 1) * kCatRows;
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 15, q = lane >> 4;
  const int32_t last = lay.cu_frames[hb.seq + 1] - 1;
  const int32_t cur_off = lay.frame_meta[3 * last];
  const int32_t n_cur = frame_size(lay, last);
  const int32_t ntiles = (n_cur + kCatKeys - 1) / kCatKeys;
  const size_t head_stride = size_t(lay.total_tokens) * kHeadDim;
  const uint16_t* klayer = a.k + size_t(layer) * H * head_stride;
  const float* rn_cur = a.rn_cur + size_t(layer) * lay.total_tokens + cur_off;

  // Historical rows row0 + 32 wave + 16 rb + n: A operands over all heads.
  int32_t tok[2];
  bf16x8_t ha[2][kSteps];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int32_t h = row0 + 32 * wave + 16 * rb + n;
    tok[rb] = h < hb.n_hist ? a.hist_tok[hb.hist_base + h] : -1;
    float ss = 0.0f;
#pragma unroll
    for (int g = 0; g < kSteps; ++g) {
      const uint4 v = tok[rb] >= 0 ? *reinterpret_cast<const uint4*>(klayer + (g >> 2) * head_stride +
                                                                      size_t(tok[rb]) * kHeadDim + (g & 3) * 32 + q * 8)
                                   : make_uint4(0, 0, 0, 0);
      ss += sumsq8(v);
      ha[rb][g] = __builtin_bit_cast(bf16x8_t, v);
    }
    ss += __shfl_xor(ss, 16);
    ss += __shfl_xor(ss, 32);
    if (q == 0) {
      tok_s[32 * wave + 16 * rb + n] = tok[rb];
      rnrow_s[32 * wave + 16 * rb + n] = inv_norm(ss);
    }
  }

  // Tile nt: keys nt * 32 .. nt * 32 + 31 of the current frame (clamped to its
  // last key, which leaves every max unchanged).  Wave-load m = wave + 4 i
  // (i < 2 H) moves keys 4 (m & 7) .. + 3 of head m >> 3.
  auto issue = [&](int32_t nt, uint16_t* dst) {
#pragma unroll
    for (int i = 0; i < 2 * H; ++i) {
      const int m = wave + 4 * i;
      const int hd = m >> 3, g = m & 7;
      const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint16_t*>(klayer + hd * head_stride + size_t(cur_off) * kHeadDim), 0, n_cur * (kHeadDim * 2),
          kBufferFlags);
      const int key = 4 * g + (lane >> 4);
      const int32_t kidx = min(nt * kCatKeys + key, n_cur - 1);
      const int ch = (lane & 15) ^ (key & 15);
      uint32_t lds = uint32_t(reinterpret_cast<uintptr_t>(dst + (hd * kCatKeys + 4 * g) * kHeadDim));
      asm volatile("" : "+s"(lds));
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (lds_void_t)(uintptr_t)lds, 16,
                                               uint32_t(kidx) * (kHeadDim * 2) + uint32_t(ch) * 16u, 0, 0, 0);
    }
  };
  // Inverse norms of tile nt's columns 16 kb + n.
  auto col_norms = [&](int32_t nt, float (&rn)[2]) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) rn[kb] = rn_cur[min(nt * kCatKeys + 16 * kb + n, n_cur - 1)];
  };

  float runmax[2][4];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) runmax[rb][i] = -INFINITY;
  float rn_c[2], rn_n[2];
  issue(0, st0);
  col_norms(0, rn_c);

  auto tile = [&](int32_t nt, const uint16_t* cur, uint16_t* nxt) {
    wait_vmcnt<0>();  // this tile's DMA and column norms have landed
    barrier_lds();    // every wave's share has landed; every wave is done with `nxt`
    if (nt + 1 < ntiles) {
      issue(nt + 1, nxt);
      col_norms(nt + 1, rn_n);
    }
    f32x4_t acc[2][2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) acc[rb][kb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int g = 0; g < kSteps; ++g) {
      bf16x8_t bf[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        bf[kb] = *reinterpret_cast<const bf16x8_t*>(cur + ((g >> 2) * kCatKeys + 16 * kb + n) * kHeadDim +
                                                    ((((g & 3) * 4 + q) ^ n) << 3));
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          acc[rb][kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ha[rb][g], bf[kb], acc[rb][kb], 0, 0, 0);
    }
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        runmax[rb][i] = __builtin_fmaxf(__builtin_fmaxf(runmax[rb][i], acc[rb][0][i] * rn_c[0]), acc[rb][1][i] * rn_c[1]);
    rn_c[0] = rn_n[0];
    rn_c[1] = rn_n[1];
  };
  for (int32_t nt = 0; nt < ntiles; nt += 2) {
    tile(nt, st0, st1);
    if (nt + 1 < ntiles) tile(nt + 1, st1, st0);
  }

  float* rho = a.rho + size_t(layer) * lay.total_tokens;
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = runmax[rb][i];
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      if (n == 0) {
        const int r = 32 * wave + 16 * rb + 4 * q + i;
        const int32_t t = tok_s[r];
        if (t >= 0) {
          float x = fminf(fmaxf(mx * rnrow_s[r], -1.0f), 1.0f);
          if (x >= kCatSnap) x = 1.0f;
          rho[t] = x + 0.0f;
        }
      }
    }
}

// Output rows of a CSS wave: 2, or 1 at four heads, where two rows of
// resident operands (128 VGPRs) leave too few registers for two waves per SIMD.
template <int H>
constexpr int css_cat_rows() { return H >= 4 ? 1 : 2; }
constexpr int kCssCols = 16;  // output columns of a CSS wave

// Loads key (row, col) of every head as MFMA operand fragments for output
// rows (lane (n, q): dims 32 kk + 8 q .. + 7 of head g >> 2, kk = g & 3) and
// returns 1/||h||.
template <int H>
__device__ inline float load_cat_operand(const uint16_t* kframe, size_t head_stride, int32_t row, int32_t col,
                                         int32_t C, int q, bf16x8_t (&frag)[4 * H]) {
  float ss = 0.0f;
#pragma unroll
  for (int g = 0; g < 4 * H; ++g) {
    const uint4 v = *reinterpret_cast<const uint4*>(kframe + (g >> 2) * head_stride + (size_t(row) * C + col) * kHeadDim +
                                                    (g & 3) * 32 + q * 8);
    ss += sumsq8(v);
    frag[g] = __builtin_bit_cast(bf16x8_t, v);
  }
  ss += __shfl_xor(ss, 16);
  ss += __shfl_xor(ss, 32);
  return inv_norm(ss);
}

// Grid: x = work-groups of four wave tiles (css_cat_rows x 16 outputs) in
// XCD-aware order, a.strips = the largest number of such tiles in a frame;
// y = layer.
template <int H>
__global__ __launch_bounds__(256) void css_cat_kernel(CssArgs a) {
  constexpr int KR = 1;
  constexpr int kCssRows = css_cat_rows<H>();
  const Layout& lay = a.lay;
  const int layer = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t per_xcd = int32_t(gridDim.x) >> 3;
  const int32_t logical = (int32_t(blockIdx.x & 7) * per_xcd + int32_t(blockIdx.x >> 3)) * 4 + wave;
  const int32_t f = logical / a.strips, t = logical - f * a.strips;
  if (f >= lay.n_frames) return;
  const int32_t off = lay.frame_meta[3 * f], R = lay.frame_meta[3 * f + 1], C = lay.frame_meta[3 * f + 2];
  const int32_t tiles_c = (C + kCssCols - 1) / kCssCols;
  const int32_t tr = t / tiles_c;
  const int32_t r0 = tr * kCssRows, c0 = (t - tr * tiles_c) * kCssCols;
  if (r0 >= R) return;
  const size_t head_stride = size_t(lay.total_tokens) * kHeadDim;
  const uint16_t* kframe = a.k + (size_t(layer) * H * lay.total_tokens + off) * kHeadDim;
  const int n = lane & 15, q = lane >> 4;

  bf16x8_t ha[kCssRows][4 * H];
  float rnA[kCssRows];
#pragma unroll
  for (int o = 0; o < kCssRows; ++o)
    rnA[o] = load_cat_operand<H>(kframe, head_stride, min(r0 + o, R - 1), min(c0 + n, C - 1), C, q, ha[o]);

  // Accumulator element (i, n) of block nb pairs output column c0 + 4 q + i
  // with strip key 16 nb + n, column c0 - 1 + 16 nb + n.
  uint32_t near = 0, self = 0;
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int32_t d = 16 * nb + n - 4 * q - i;
      const int32_t cc = c0 - KR + 16 * nb + n;
      if (d >= 0 && d <= 2 * KR && cc >= 0 && cc < C) near |= 1u << (4 * nb + i);
      if (d == KR) self |= 1u << (4 * nb + i);
    }
  float psum[kCssRows][4];
#pragma unroll
  for (int o = 0; o < kCssRows; ++o)
#pragma unroll
    for (int i = 0; i < 4; ++i) psum[o][i] = 0.0f;

  const int32_t rr0 = max(r0 - KR, 0), rr1 = min(r0 + kCssRows - 1 + KR, R - 1);
  auto fetch = [&](int32_t rr, int h, uint4 (&v)[2][4]) {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      const uint16_t* src = kframe + h * head_stride +
                            (size_t(rr) * C + min(max(c0 - KR + 16 * nb + n, 0), C - 1)) * kHeadDim + q * 8;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) v[nb][kk] = *reinterpret_cast<const uint4*>(src + kk * 32);
    }
  };
  // Head h of a row sits in buffer h & 1 (H is even); the next head's (or the
  // next row's first head's) loads are issued before this head's matrix work.
  uint4 buf[2][2][4];
  fetch(rr0, 0, buf[0]);
  for (int32_t rr = rr0; rr <= rr1; ++rr) {
    f32x4_t acc[kCssRows][2];
#pragma unroll
    for (int o = 0; o < kCssRows; ++o)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb) acc[o][nb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float ss[2] = {0.0f, 0.0f};
#pragma unroll
    for (int h = 0; h < H; ++h) {
      if (h + 1 < H) fetch(rr, h + 1, buf[(h + 1) & 1]);
      else if (rr < rr1) fetch(rr + 1, 0, buf[0]);
      const uint4 (&v)[2][4] = buf[h & 1];
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) ss[nb] += sumsq8(v[nb][kk]);
      // The sums are formed here, not after the last head: otherwise every
      // head's loaded keys stay live until then.
      asm volatile("" : "+v"(ss[0]), "+v"(ss[1]));
#pragma unroll
      for (int o = 0; o < kCssRows; ++o) {
        const int32_t ro = r0 + o;
        if (ro >= R || rr < ro - KR || rr > ro + KR) continue;  // uniform over the wave
#pragma unroll
        for (int nb = 0; nb < 2; ++nb)
#pragma unroll
          for (int kk = 0; kk < 4; ++kk)
            acc[o][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ha[o][4 * h + kk],
                                                                 __builtin_bit_cast(bf16x8_t, v[nb][kk]), acc[o][nb],
                                                                 0, 0, 0);
      }
      // Keep the scheduler from hoisting later heads' loads above this head:
      // one head in flight beside the one being multiplied.
      __builtin_amdgcn_sched_barrier(0);
    }
    float rn[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      float x = ss[nb] + __shfl_xor(ss[nb], 16);
      x += __shfl_xor(x, 32);
      rn[nb] = inv_norm(x);
    }
#pragma unroll
    for (int o = 0; o < kCssRows; ++o) {
      const int32_t ro = r0 + o;
      if (ro >= R || rr < ro - KR || rr > ro + KR) continue;
      const uint32_t keep = rr == ro ? near & ~self : near;
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          psum[o][i] = fmaf(acc[o][nb][i], (keep >> (4 * nb + i)) & 1u ? rn[nb] : 0.0f, psum[o][i]);
    }
  }

  float* phi = a.phi + size_t(layer) * lay.total_tokens + off;
#pragma unroll
  for (int o = 0; o < kCssRows; ++o)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float h = psum[o][i];
#pragma unroll
      for (int m = 1; m < 16; m <<= 1) h += __shfl_xor(h, m);
      const float rn_out = __shfl(rnA[o], 4 * q + i);
      const int32_t r = r0 + o, c = c0 + 4 * q + i;
      if (n == 0 && r < R && c < C) {
        const int32_t rows_in = min(r + KR, R - 1) - max(r - KR, 0) + 1;
        const int32_t cols_in = min(c + KR, C - 1) - max(c - KR, 0) + 1;
        const int32_t nn = rows_in * cols_in - 1;
        phi[size_t(r) * C + c] = nn > 0 ? 1.0f - h * rn_out / float(nn) : 0.0f;
      }
    }
}

// Phi = 0 on the text tokens of every layer (the frames are written by css_cat_kernel).
// Work-group (g, layer) writes text run g (token_run).
__global__ __launch_bounds__(256) void cat_text_kernel(CssArgs a) {
  const Layout& lay = a.lay;
  float* out = a.phi + size_t(blockIdx.y) * lay.total_tokens;
  int32_t b, e;
  token_run(lay, int32_t(blockIdx.x), false, &b, &e);
  for (int32_t j = b + int32_t(threadIdx.x); j < e; j += blockDim.x) out[j] = 0.0f;
}

}  // namespace

hipError_t launch_layer_mean(const float* a_base, float* a_layer, const Layout& lay, hipStream_t stream) {
  const int32_t n_layers = lay.n_units / lay.n_kv_heads;
  const int64_t n = int64_t(n_layers) * lay.total_tokens;
  const unsigned blocks = unsigned(std::max<int64_t>(1, std::min<int64_t>((n + 255) / 256, 8192)));
  hipLaunchKernelGGL(layer_mean_kernel, dim3(blocks), dim3(256), 0, stream, a_base, a_layer, n_layers,
                     lay.n_kv_heads, lay.total_tokens);
  return hipGetLastError();
}

hipError_t launch_tsg_rho_concat(const RhoArgs& r, const GateArgs& g, hipStream_t stream) {
  hipError_t e = launch_gate_prologue(g, stream);  // plan tables; rho_layer = 0 everywhere
  if (e != hipSuccess) return e;
  const int32_t H = r.lay.n_kv_heads, n_layers = r.lay.n_units / H;
  const dim3 norm_grid((std::max(r.max_cur, 1) + 63) / 64, r.lay.n_seqs, n_layers);
  const dim3 grid(2 * r.total_hist_blocks, n_layers);
  if (H == 2) {
    hipLaunchKernelGGL(cat_norms_kernel<2>, norm_grid, dim3(256), 0, stream, r);
    if (r.total_hist_blocks > 0) hipLaunchKernelGGL(rho_cat_kernel<2>, grid, dim3(256), 0, stream, r);
  } else if (H == 4) {
    hipLaunchKernelGGL(cat_norms_kernel<4>, norm_grid, dim3(256), 0, stream, r);
    if (r.total_hist_blocks > 0) hipLaunchKernelGGL(rho_cat_kernel<4>, grid, dim3(256), 0, stream, r);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_css_concat(const CssArgs& a, hipStream_t stream) {
  const int32_t H = a.lay.n_kv_heads, n_layers = a.lay.n_units / H;
  hipLaunchKernelGGL(cat_text_kernel, dim3(a.lay.n_frames + a.lay.n_seqs, n_layers), dim3(256), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.lay.n_frames == 0) return e;
  const int64_t logical = int64_t(a.lay.n_frames) * a.strips;
  const int64_t grid_x = ((logical + 3) / 4 + 7) / 8 * 8;
  const dim3 grid(unsigned(grid_x), n_layers);
  if (H == 2)
    hipLaunchKernelGGL(css_cat_kernel<2>, grid, dim3(256), 0, stream, a);
  else if (H == 4)
    hipLaunchKernelGGL(css_cat_kernel<4>, grid, dim3(256), 0, stream, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace stlite
