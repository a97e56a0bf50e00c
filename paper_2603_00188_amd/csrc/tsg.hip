// Trajectory-aware Semantic Gating (Sec. TSG of the paper).
//
//   rho_i = max_{j in current frame} cos(k_i, k_j)   for historical visual i
//   m = min(B, |pool|); the gate admits the m historical tokens first in
//   (rho ascending, index ascending) order (Eqs. budget_threshold and
//   temporal_mask in rank form); current frame and text get gate 1.
//
// rho is a dense N_hist x N_cur x 128 contraction: bf16 MFMA tiles with the
// historical rows resident in VGPRs (A operand, 256 rows per work-group) and
// the current frame streamed through LDS in 64-key tiles (B operand).  The
// epilogue never stores the logits: each lane scales its column by the key's
// inverse norm and keeps a running row max; 16-lane butterflies finish the max.
#include "block_select.h"
#include "stlite_internal.h"

namespace stlite {
namespace {

constexpr int kRhoRows = 256;
constexpr int kCurTile = 64;
constexpr int kKStride = kHeadDim + 8;
constexpr float kSnap = 1.0f - 1.0e-4f;

struct HistBlock {
  int32_t seq, hb, n_hist;
};

__device__ inline int32_t frame_size(const Layout& lay, int32_t f) {
  return lay.frame_meta[3 * f + 1] * lay.frame_meta[3 * f + 2];
}

__device__ inline int32_t hist_count(const Layout& lay, int32_t s) {
  const int32_t f0 = lay.cu_frames[s], f1 = lay.cu_frames[s + 1];
  int32_t n = 0;
  for (int32_t f = f0; f + 1 < f1; ++f) n += frame_size(lay, f);
  return n;
}

__device__ inline HistBlock locate_hist_block(const Layout& lay, int32_t x) {
  int32_t acc = 0;
  for (int32_t s = 0; s < lay.n_seqs; ++s) {
    const int32_t nh = hist_count(lay, s);
    const int32_t nb = (nh + kRhoRows - 1) / kRhoRows;
    if (x < acc + nb) return HistBlock{s, x - acc, nh};
    acc += nb;
  }
  return HistBlock{-1, 0, 0};
}

// Absolute token of the h-th historical visual token of sequence s.
__device__ inline int32_t hist_token(const Layout& lay, int32_t s, int32_t h) {
  const int32_t f0 = lay.cu_frames[s], f1 = lay.cu_frames[s + 1];
  for (int32_t f = f0; f + 1 < f1; ++f) {
    const int32_t n = frame_size(lay, f);
    if (h < n) return lay.frame_meta[3 * f] + h;
    h -= n;
  }
  return -1;
}

__device__ inline float sumsq8(uint4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  float s = 0.0f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const float lo = __uint_as_float(w[j] << 16), hi = __uint_as_float(w[j] & 0xffff0000u);
    s = fmaf(lo, lo, s);
    s = fmaf(hi, hi, s);
  }
  return s;
}

// Inverse norms of the current-frame keys: rn[unit][token] = 1/||k|| (0 for a zero key).
__global__ __launch_bounds__(256) void cur_norms_kernel(RhoArgs a) {
  const int s = blockIdx.x, unit = blockIdx.y;
  const Layout& lay = a.lay;
  const int32_t f0 = lay.cu_frames[s], f1 = lay.cu_frames[s + 1];
  if (f1 - f0 < 2) return;  // no history: nothing reads the current-frame norms
  const int32_t off = lay.frame_meta[3 * (f1 - 1)];
  const int32_t n = frame_size(lay, f1 - 1);
  const uint16_t* kunit = a.k + size_t(unit) * lay.total_tokens * kHeadDim;
  float* rn = a.rn_cur + size_t(unit) * lay.total_tokens;
  const int group = threadIdx.x >> 4, gl = threadIdx.x & 15;
  for (int32_t j = group; j < n; j += blockDim.x >> 4) {
    const uint4 v = *reinterpret_cast<const uint4*>(kunit + size_t(off + j) * kHeadDim + gl * 8);
    float ss = sumsq8(v);
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) ss += __shfl_xor(ss, o);
    if (gl == 0) rn[off + j] = ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f;
  }
}

__global__ __launch_bounds__(256) void rho_kernel(RhoArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ks[kCurTile * kKStride];
  __shared__ float rn_tile[kCurTile];
  __shared__ int32_t tok_s[kRhoRows];
  __shared__ float rnrow_s[kRhoRows];
  const Layout& lay = a.lay;
  const int unit = blockIdx.y;
  const HistBlock hb = locate_hist_block(lay, blockIdx.x);
  if (hb.seq < 0) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int32_t last = lay.cu_frames[hb.seq + 1] - 1;
  const int32_t cur_off = lay.frame_meta[3 * last];
  const int32_t n_cur = frame_size(lay, last);
  const uint16_t* kunit = a.k + size_t(unit) * lay.total_tokens * kHeadDim;

  // Historical rows: A operand (row = lane & 15 of each 16-row block).
  bf16x8_t ha[4][4];
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const int32_t h = hb.hb * kRhoRows + wave * 64 + b * 16 + (lane & 15);
    const int32_t tok = h < hb.n_hist ? hist_token(lay, hb.seq, h) : -1;
    float ss = 0.0f;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (tok >= 0) v = *reinterpret_cast<const uint4*>(kunit + size_t(tok) * kHeadDim + kk * 32 + (lane >> 4) * 8);
      ss += sumsq8(v);
      ha[b][kk] = __builtin_bit_cast(bf16x8_t, v);
    }
    ss += __shfl_xor(ss, 16);
    ss += __shfl_xor(ss, 32);
    if (lane < 16) {
      tok_s[wave * 64 + b * 16 + lane] = tok;
      rnrow_s[wave * 64 + b * 16 + lane] = ss > 0.0f ? 1.0f / sqrtf(ss) : 0.0f;
    }
  }

  float runmax[4][4];
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) runmax[b][i] = -INFINITY;

  const float* rn_cur = a.rn_cur + size_t(unit) * lay.total_tokens + cur_off;
  const uint16_t* kcur = kunit + size_t(cur_off) * kHeadDim;
  for (int32_t c0 = 0; c0 < n_cur; c0 += kCurTile) {
    __syncthreads();
    for (int i = threadIdx.x; i < kCurTile * 16; i += blockDim.x) {
      const int key = i >> 4, part = i & 15;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (c0 + key < n_cur) v = *reinterpret_cast<const uint4*>(kcur + size_t(c0 + key) * kHeadDim + part * 8);
      *reinterpret_cast<uint4*>(ks + key * kKStride + part * 8) = v;
    }
    if (threadIdx.x < kCurTile) rn_tile[threadIdx.x] = (c0 + threadIdx.x < n_cur) ? rn_cur[c0 + threadIdx.x] : 0.0f;
    __syncthreads();
    bf16x8_t kb[4][4];
    float rnl[4];
    bool valid[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      rnl[t] = rn_tile[t * 16 + (lane & 15)];
      valid[t] = c0 + t * 16 + (lane & 15) < n_cur;
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        kb[t][kk] = *reinterpret_cast<const bf16x8_t*>(ks + (t * 16 + (lane & 15)) * kKStride + kk * 32 +
                                                        (lane >> 4) * 8);
    }
#pragma unroll
    for (int b = 0; b < 4; ++b) {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ha[b][kk], kb[t][kk], acc, 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float v = valid[t] ? acc[i] * rnl[t] : -INFINITY;
          runmax[b][i] = fmaxf(runmax[b][i], v);
        }
      }
    }
  }
  __syncthreads();

  float* rho = a.rho + size_t(unit) * lay.total_tokens;
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = runmax[b][i];
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
      if ((lane & 15) == 0) {
        const int r = wave * 64 + b * 16 + (lane >> 4) * 4 + i;
        const int32_t tok = tok_s[r];
        if (tok >= 0) {
          float x = fminf(fmaxf(mx * rnrow_s[r], -1.0f), 1.0f);
          if (x >= kSnap) x = 1.0f;
          rho[tok] = x + 0.0f;
        }
      }
    }
}

// Rank-form gate for one (unit, sequence): admit the m = min(B, N_hist)
// smallest rho in (rho, index) order.
__global__ __launch_bounds__(kSelThreads) void gate_kernel(GateArgs a) {
  __shared__ SelectShared sh;
  const Layout& lay = a.lay;
  const int s = blockIdx.x, unit = blockIdx.y, tid = threadIdx.x;
  const int32_t seq_start = lay.cu_seqlens[s], seq_end = lay.cu_seqlens[s + 1];
  const int32_t f0 = lay.cu_frames[s], f1 = lay.cu_frames[s + 1];
  const int32_t B = lay.cu_budget[s + 1] - lay.cu_budget[s];
  const size_t ubase = size_t(unit) * lay.total_tokens;
  uint32_t* keys = a.keys + ubase + seq_start;  // compact historical keys, in token order
  const float* rho = a.rho + ubase;
  uint8_t* gate = a.gate + ubase;
  float* zf = a.rho_zero_fill ? a.rho_zero_fill + ubase : nullptr;

  int32_t nh = 0;
  for (int32_t f = f0; f + 1 < f1; ++f) {
    const int32_t off = lay.frame_meta[3 * f], n = frame_size(lay, f);
    for (int32_t j = tid; j < n; j += kSelThreads) keys[nh + j] = order_key(rho[off + j]);
    nh += n;
  }
  __syncthreads();
  const int32_t m = min(B, nh);
  uint32_t T = 0;
  int32_t need = 0;
  if (m > 0) T = block_radix_select(keys, nh, m, sh, &need);
  if (tid == 0 && a.tau) a.tau[size_t(unit) * lay.n_seqs + s] = m > 0 ? order_key_value(T) : __builtin_nanf("");

  int32_t running_eq = 0, h = 0, prev = seq_start;
  for (int32_t f = f0; f <= f1; ++f) {
    const bool is_frame = f < f1;
    const int32_t off = is_frame ? lay.frame_meta[3 * f] : seq_end;
    const int32_t n = is_frame ? frame_size(lay, f) : 0;
    for (int32_t j = prev + tid; j < off; j += kSelThreads) {  // text before this frame
      gate[j] = 1;
      if (zf) zf[j] = 0.0f;
    }
    if (is_frame && f == f1 - 1) {  // current frame: exempt from the gate
      for (int32_t j = tid; j < n; j += kSelThreads) {
        gate[off + j] = 1;
        if (zf) zf[off + j] = 0.0f;
      }
    } else if (is_frame) {
      for (int32_t base = 0; base < n; base += kSelThreads) {
        const int32_t j = base + tid;
        const bool in = j < n;
        const uint32_t key = in ? keys[h + j] : 0u;
        const bool eq = in && m > 0 && key == T;
        int32_t eq_tot;
        const int32_t eq_incl = block_inclusive_scan(eq ? 1 : 0, sh.wave_tot, &eq_tot);
        const bool take = (in && m > 0 && key < T) || (eq && running_eq + eq_incl - 1 < need);
        if (in) gate[off + j] = take ? 1 : 0;
        running_eq += eq_tot;
      }
      h += n;
    }
    prev = off + n;
  }
}

}  // namespace

hipError_t launch_tsg_threshold(const GateArgs& g, hipStream_t stream) {
  hipLaunchKernelGGL(gate_kernel, dim3(g.lay.n_seqs, g.lay.n_units), dim3(kSelThreads), 0, stream, g);
  return hipGetLastError();
}

hipError_t launch_tsg_gate(const RhoArgs& r, const GateArgs& g, hipStream_t stream) {
  hipLaunchKernelGGL(cur_norms_kernel, dim3(r.lay.n_seqs, r.lay.n_units), dim3(256), 0, stream, r);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (r.total_hist_blocks > 0) {
    hipLaunchKernelGGL(rho_kernel, dim3(r.total_hist_blocks, r.lay.n_units), dim3(256), 0, stream, r);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return launch_tsg_threshold(g, stream);
}

}  // namespace stlite
