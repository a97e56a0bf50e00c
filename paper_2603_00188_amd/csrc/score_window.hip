// Window base score A_base (Eq. base_attention) for every (layer, kv head,
// sequence): A_i = (1/G) sum_g sum_w softmax_{j <= p_w}(q_{g,w} . k_j / sqrt(d))_i.
//
// A column sum of softmax rows needs every row's normaliser first, so the
// logits Q K^T are formed twice on the matrix cores (bf16 MFMA, fp32
// accumulate):
//   pass 1  (rowstats) per key chunk: running (max, sum of 2^x) per window row,
//   combine            per row: log2 of the softmax denominator over all chunks,
//   pass 2  (colsum)   per key chunk: 2^(x - lse) summed over the G*window rows.
// Both passes keep the whole GQA group's window queries resident in VGPRs as
// the MFMA A operand (each wave owns row_blocks 16-row blocks) and stream
// 64-key tiles of K through LDS as the B operand, shared by all waves.
// Logits are kept in log2 units: x = (q . k) * log2(e) / sqrt(d).
#include "stlite_internal.h"

namespace stlite {
namespace {

constexpr int kTileKeys = 64;
constexpr int kKStride = kHeadDim + 8;  // staged key row: 272 bytes, keeps ds_read_b128 conflict-free
constexpr float kNegBig = -1.0e30f;

struct ChunkPos {
  int32_t seq, seq_start, seq_len, c0, c1, gchunk;
};

// Work-group x index -> (sequence, key range) for a fixed chunk length.
__device__ inline ChunkPos locate_chunk(const Layout& lay, int32_t chunk, int32_t gchunk) {
  ChunkPos r{-1, 0, 0, 0, 0, gchunk};
  int32_t acc = 0;
  for (int32_t s = 0; s < lay.n_seqs; ++s) {
    const int32_t a = lay.cu_seqlens[s], b = lay.cu_seqlens[s + 1];
    const int32_t n = (b - a + chunk - 1) / chunk;
    if (gchunk < acc + n) {
      const int32_t c = gchunk - acc;
      r.seq = s;
      r.seq_start = a;
      r.seq_len = b - a;
      r.c0 = c * chunk;
      r.c1 = min(r.c0 + chunk, b - a);
      return r;
    }
    acc += n;
  }
  return r;
}

// Stage keys [t0, t0+64) of one sequence (local indices, zero past `end`) into LDS.
__device__ inline void stage_keys(uint16_t* ks, const uint16_t* kseq, int32_t t0, int32_t end) {
  const int nthreads = blockDim.x;
  for (int i = threadIdx.x; i < kTileKeys * 16; i += nthreads) {
    const int key = i >> 4, part = i & 15;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (t0 + key < end)
      v = *reinterpret_cast<const uint4*>(kseq + size_t(t0 + key) * kHeadDim + part * 8);
    *reinterpret_cast<uint4*>(ks + key * kKStride + part * 8) = v;
  }
}

__device__ inline bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

template <int RB>
__device__ inline void load_queries(const ScoreArgs& a, const ChunkPos& cp, int unit, bf16x8_t (&qa)[RB][4]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int layer = unit / a.lay.n_kv_heads, kv = unit % a.lay.n_kv_heads;
  const uint16_t* qbase =
      a.q + ((size_t(layer) * a.lay.n_seqs + cp.seq) * a.n_q_heads + size_t(kv) * a.group) * a.window * kHeadDim;
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    const int row = (wave * RB + b) * 16 + (lane & 15);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row < a.rows)
        v = *reinterpret_cast<const uint4*>(qbase + size_t(row) * kHeadDim + kk * 32 + (lane >> 4) * 8);
      qa[b][kk] = as_bf16x8(v);
    }
  }
}

template <int RB>
__global__ __launch_bounds__(256) void score_rowstats_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ks[kTileKeys * kKStride];
  const int unit = blockIdx.y;
  const ChunkPos cp = locate_chunk(a.lay, a.chunk, blockIdx.x);
  if (cp.seq < 0) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float scale2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)

  bf16x8_t qa[RB][4];
  load_queries<RB>(a, cp, unit, qa);

  int32_t pos[RB][4];  // last visible key (local index) of each of the lane's output rows
  float m[RB][4], sum[RB][4];
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = (wave * RB + b) * 16 + (lane >> 4) * 4 + i;
      pos[b][i] = r < a.rows ? cp.seq_len - a.window + (r % a.window) : -1;
      m[b][i] = kNegBig;
      sum[b][i] = 0.0f;
    }

  const uint16_t* kseq = a.k + (size_t(unit) * a.lay.total_tokens + cp.seq_start) * kHeadDim;
  for (int32_t t0 = cp.c0; t0 < cp.c1; t0 += kTileKeys) {
    __syncthreads();
    stage_keys(ks, kseq, t0, cp.c1);
    __syncthreads();
    bf16x8_t kb[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        kb[t][kk] = *reinterpret_cast<const bf16x8_t*>(ks + (t * 16 + (lane & 15)) * kKStride + kk * 32 +
                                                        (lane >> 4) * 8);
    const bool clean = (t0 + kTileKeys <= cp.c1) && (t0 + kTileKeys - 1 <= cp.seq_len - a.window);
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      f32x4_t acc[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[b][kk], kb[t][kk], acc[t], 0, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          v[t] = acc[t][i] * scale2;
          if (!clean) {
            const int32_t j = t0 + t * 16 + (lane & 15);
            if (j >= cp.c1 || j > pos[b][i]) v[t] = -INFINITY;
          }
        }
        const float mx = fmaxf(fmaxf(fmaxf(m[b][i], v[0]), fmaxf(v[1], v[2])), v[3]);
        sum[b][i] = sum[b][i] * __builtin_amdgcn_exp2f(m[b][i] - mx) + __builtin_amdgcn_exp2f(v[0] - mx) +
                    __builtin_amdgcn_exp2f(v[1] - mx) + __builtin_amdgcn_exp2f(v[2] - mx) +
                    __builtin_amdgcn_exp2f(v[3] - mx);
        m[b][i] = mx;
      }
    }
  }

  // Merge the 16 lanes that hold the same rows (different key columns).
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mm = m[b][i], ss = sum[b][i];
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const float mo = __shfl_xor(mm, off);
        const float so = __shfl_xor(ss, off);
        const float mx = fmaxf(mm, mo);
        ss = ss * __builtin_amdgcn_exp2f(mm - mx) + so * __builtin_amdgcn_exp2f(mo - mx);
        mm = mx;
      }
      if ((lane & 15) == 0) {
        const int r = (wave * RB + b) * 16 + (lane >> 4) * 4 + i;
        a.partial[(size_t(unit) * a.total_chunks + cp.gchunk) * a.rows_pad + r] = make_float2(mm, ss);
      }
    }
}

__global__ __launch_bounds__(256) void score_combine_kernel(ScoreArgs a) {
  const int s = blockIdx.x, unit = blockIdx.y;
  int32_t first = 0;
  for (int32_t t = 0; t < s; ++t) {
    const int32_t L = a.lay.cu_seqlens[t + 1] - a.lay.cu_seqlens[t];
    first += (L + a.chunk - 1) / a.chunk;
  }
  const int32_t L = a.lay.cu_seqlens[s + 1] - a.lay.cu_seqlens[s];
  const int32_t nch = (L + a.chunk - 1) / a.chunk;
  for (int r = threadIdx.x; r < a.rows_pad; r += blockDim.x) {
    float out = INFINITY;  // padding rows contribute exp2(-inf) = 0 in pass 2
    if (r < a.rows) {
      const float2* pr = a.partial + (size_t(unit) * a.total_chunks + first) * a.rows_pad + r;
      float M = kNegBig;
      for (int32_t c = 0; c < nch; ++c) M = fmaxf(M, pr[size_t(c) * a.rows_pad].x);
      float Z = 0.0f;
      for (int32_t c = 0; c < nch; ++c) {
        const float2 v = pr[size_t(c) * a.rows_pad];
        Z += v.y * __builtin_amdgcn_exp2f(v.x - M);
      }
      out = M + __log2f(Z);
    }
    a.lse2[(size_t(unit) * a.lay.n_seqs + s) * a.rows_pad + r] = out;
  }
}

template <int RB>
__global__ __launch_bounds__(256) void score_colsum_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ks[kTileKeys * kKStride];
  __shared__ float red[4][kTileKeys];
  const int unit = blockIdx.y;
  const ChunkPos cp = locate_chunk(a.lay, a.chunk, blockIdx.x);
  if (cp.seq < 0) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nwaves = blockDim.x >> 6;
  const float scale2 = 1.4426950408889634f * 0.08838834764831845f;
  const float inv_g = 1.0f / float(a.group);

  bf16x8_t qa[RB][4];
  load_queries<RB>(a, cp, unit, qa);

  int32_t pos[RB][4];
  float lse[RB][4];
  const float* lrow = a.lse2 + (size_t(unit) * a.lay.n_seqs + cp.seq) * a.rows_pad;
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = (wave * RB + b) * 16 + (lane >> 4) * 4 + i;
      pos[b][i] = r < a.rows ? cp.seq_len - a.window + (r % a.window) : -1;
      lse[b][i] = lrow[r];
    }

  const uint16_t* kseq = a.k + (size_t(unit) * a.lay.total_tokens + cp.seq_start) * kHeadDim;
  float* aout = a.a_base + size_t(unit) * a.lay.total_tokens + cp.seq_start;
  for (int32_t t0 = cp.c0; t0 < cp.c1; t0 += kTileKeys) {
    __syncthreads();
    stage_keys(ks, kseq, t0, cp.c1);
    __syncthreads();
    bf16x8_t kb[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        kb[t][kk] = *reinterpret_cast<const bf16x8_t*>(ks + (t * 16 + (lane & 15)) * kKStride + kk * 32 +
                                                        (lane >> 4) * 8);
    const bool clean = (t0 + kTileKeys <= cp.c1) && (t0 + kTileKeys - 1 <= cp.seq_len - a.window);
    float col[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      f32x4_t acc[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[b][kk], kb[t][kk], acc[t], 0, 0, 0);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          float p = __builtin_amdgcn_exp2f(acc[t][i] * scale2 - lse[b][i]);
          if (!clean) {
            const int32_t j = t0 + t * 16 + (lane & 15);
            if (j >= cp.c1 || j > pos[b][i]) p = 0.0f;
          }
          col[t] += p;
        }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      col[t] += __shfl_xor(col[t], 16);
      col[t] += __shfl_xor(col[t], 32);
    }
    if (lane < 16) {
#pragma unroll
      for (int t = 0; t < 4; ++t) red[wave][t * 16 + lane] = col[t];
    }
    __syncthreads();
    if (threadIdx.x < kTileKeys) {
      float s = 0.0f;
      for (int w = 0; w < nwaves; ++w) s += red[w][threadIdx.x];
      const int32_t j = t0 + threadIdx.x;
      if (j < cp.c1) aout[j] = s * inv_g;
    }
  }
}

template <int RB>
hipError_t launch_rb(const ScoreArgs& a, hipStream_t stream) {
  const dim3 grid(a.total_chunks, a.lay.n_units);
  const dim3 block(64 * a.waves);
  hipLaunchKernelGGL(score_rowstats_kernel<RB>, grid, block, 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(score_combine_kernel, dim3(a.lay.n_seqs, a.lay.n_units), dim3(256), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(score_colsum_kernel<RB>, grid, block, 0, stream, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_score_window(const ScoreArgs& a, hipStream_t stream) {
  if (a.waves < 1 || a.waves > 4) return hipErrorInvalidValue;
  switch (a.row_blocks) {
    case 1: return launch_rb<1>(a, stream);
    case 2: return launch_rb<2>(a, stream);
    case 3: return launch_rb<3>(a, stream);
    case 4: return launch_rb<4>(a, stream);
    case 5: return launch_rb<5>(a, stream);
    case 6: return launch_rb<6>(a, stream);
    case 7: return launch_rb<7>(a, stream);
    case 8: return launch_rb<8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace stlite
