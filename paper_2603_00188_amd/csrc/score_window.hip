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
// the MFMA A operand (up to 8 waves, each owning up to four 16-row blocks) and
// stream 64-key tiles of K through LDS as the B operand, shared by all waves.
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

__device__ inline bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

// Register-prefetched staging of 64-key tiles into LDS: fetch() issues the
// global loads of the next tile before the current one is consumed, stage()
// writes them to the other LDS buffer afterwards.  Keys past `end` are zero.
template <int NW>
struct KeyStager {
  static constexpr int kThreads = NW * 64;
  static constexpr int kPer = kTileKeys * 16 / kThreads;
  uint4 pre[kPer];
  __device__ inline void fetch(const uint16_t* kseq, int32_t t0, int32_t end) {
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      const int i = threadIdx.x + r * kThreads;
      const int32_t j = t0 + (i >> 4);
      pre[r] = j < end ? *reinterpret_cast<const uint4*>(kseq + size_t(j) * kHeadDim + (i & 15) * 8)
                       : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ inline void stage(uint16_t* ks) const {
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      const int i = threadIdx.x + r * kThreads;
      *reinterpret_cast<uint4*>(ks + (i >> 4) * kKStride + (i & 15) * 8) = pre[r];
    }
  }
};

// Row blocks are dealt to waves round-robin (wave w owns blocks w, w + NW, ...),
// so that each SIMD of the CU gets the same number of real 16-row blocks.
template <int NW>
__device__ inline int block_of(int j) { return (threadIdx.x >> 6) + j * NW; }

template <int RB, int NW>
__device__ inline void load_queries(const ScoreArgs& a, const ChunkPos& cp, int unit, bf16x8_t (&qa)[RB][4]) {
  const int lane = threadIdx.x & 63;
  const int layer = unit / a.lay.n_kv_heads, kv = unit % a.lay.n_kv_heads;
  const uint16_t* qbase =
      a.q + ((size_t(layer) * a.lay.n_seqs + cp.seq) * a.n_q_heads + size_t(kv) * a.group) * a.window * kHeadDim;
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    const int row = block_of<NW>(b) * 16 + (lane & 15);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row < a.rows)
        v = *reinterpret_cast<const uint4*>(qbase + size_t(row) * kHeadDim + kk * 32 + (lane >> 4) * 8);
      qa[b][kk] = as_bf16x8(v);
    }
  }
}

__device__ inline void read_b_operand(const uint16_t* ks, bf16x8_t (&kb)[4][4]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int t = 0; t < 4; ++t)
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
      kb[t][kk] = *reinterpret_cast<const bf16x8_t*>(ks + (t * 16 + (lane & 15)) * kKStride + kk * 32 +
                                                      (lane >> 4) * 8);
}

// Q K^T of one 64-key tile for row block b: four 16x16 accumulators (one per
// 16-key sub-tile); the four MFMA chains are interleaved k-step by k-step.
template <int RB>
__device__ inline void tile_logits(const bf16x8_t (&qa)[RB][4], const bf16x8_t (&kb)[4][4], int b, f32x4_t (&acc)[4]) {
#pragma unroll
  for (int t = 0; t < 4; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
#pragma unroll
    for (int t = 0; t < 4; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[b][kk], kb[t][kk], acc[t], 0, 0, 0);
}

// Last key (local index) a lane's output row i of block b may see, -1 for padding rows.
template <int NW>
__device__ inline int32_t row_limit(const ScoreArgs& a, const ChunkPos& cp, int b, int i) {
  const int lane = threadIdx.x & 63;
  const int r = block_of<NW>(b) * 16 + (lane >> 4) * 4 + i;
  return r < a.rows ? cp.seq_len - a.window + (r % a.window) : -1;
}

// Pass 1 on one tile.  Per lane and window row: running max m of the raw
// logits (q.k units) and sum of 2^((x - m) s), s = log2(e)/sqrt(d), updated
// once per tile from the four values the lane holds for that row.
template <int RB, int NW, bool MASK>
__device__ inline void rowstats_tile(const ScoreArgs& a, const ChunkPos& cp, int32_t t0, const bf16x8_t (&qa)[RB][4],
                                     const bf16x8_t (&kb)[4][4], float (&m)[RB][4], float (&sum)[RB][4]) {
  const float scale2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    if (block_of<NW>(b) >= a.blocks) break;  // wave-uniform: padding blocks do no work
    f32x4_t acc[4];
    tile_logits<RB>(qa, kb, b, acc);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float v[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) v[t] = acc[t][i];
      if (MASK) {
        const int32_t lim = min(row_limit<NW>(a, cp, b, i), cp.c1 - 1);
#pragma unroll
        for (int t = 0; t < 4; ++t)
          if (t0 + t * 16 + (lane & 15) > lim) v[t] = -INFINITY;
      }
      const float mx = __builtin_fmaxf(__builtin_fmaxf(__builtin_fmaxf(m[b][i], v[0]), v[1]),
                                       __builtin_fmaxf(v[2], v[3]));
      const float ms = mx * scale2;
      float sacc = sum[b][i] * __builtin_amdgcn_exp2f(fmaf(m[b][i], scale2, -ms));
#pragma unroll
      for (int t = 0; t < 4; ++t) sacc += __builtin_amdgcn_exp2f(fmaf(v[t], scale2, -ms));
      sum[b][i] = sacc;
      m[b][i] = mx;
    }
  }
}

template <int RB, int NW>
__global__ __launch_bounds__(NW * 64) void score_rowstats_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ks[2][kTileKeys * kKStride];
  const int unit = blockIdx.y;
  const ChunkPos cp = locate_chunk(a.lay, a.chunk, blockIdx.x);
  if (cp.seq < 0) return;
  const int lane = threadIdx.x & 63;
  const float scale2 = 1.4426950408889634f * 0.08838834764831845f;

  bf16x8_t qa[RB][4];
  load_queries<RB, NW>(a, cp, unit, qa);
  float m[RB][4], sum[RB][4];
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      m[b][i] = kNegBig;
      sum[b][i] = 0.0f;
    }

  const uint16_t* kseq = a.k + (size_t(unit) * a.lay.total_tokens + cp.seq_start) * kHeadDim;
  // Tiles that end before the window starts are visible to every row: no mask.
  const int32_t clean_end = min(cp.c1, cp.seq_len - a.window + 1);
  KeyStager<NW> st;
  st.fetch(kseq, cp.c0, cp.c1);
  st.stage(ks[0]);
  __syncthreads();
  int buf = 0;
  for (int32_t t0 = cp.c0; t0 < cp.c1; t0 += kTileKeys) {
    const bool more = t0 + kTileKeys < cp.c1;
    if (more) st.fetch(kseq, t0 + kTileKeys, cp.c1);
    bf16x8_t kb[4][4];
    read_b_operand(ks[buf], kb);
    if (t0 + kTileKeys <= clean_end)
      rowstats_tile<RB, NW, false>(a, cp, t0, qa, kb, m, sum);
    else
      rowstats_tile<RB, NW, true>(a, cp, t0, qa, kb, m, sum);
    if (more) st.stage(ks[buf ^ 1]);
    __syncthreads();
    buf ^= 1;
  }

  // Merge the 16 lanes that hold the same rows (different key columns); log2 units.
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mm = m[b][i] * scale2, ss = sum[b][i];
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) {
        const float mo = __shfl_xor(mm, off);
        const float so = __shfl_xor(ss, off);
        const float mx = fmaxf(mm, mo);
        ss = ss * __builtin_amdgcn_exp2f(mm - mx) + so * __builtin_amdgcn_exp2f(mo - mx);
        mm = mx;
      }
      if ((lane & 15) == 0) {
        const int r = block_of<NW>(b) * 16 + (lane >> 4) * 4 + i;
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

// Pass 2 on one tile: col[t] += 2^(x s - lse) over the lane's rows, for the
// lane's key column of sub-tile t.
template <int RB, int NW, bool MASK>
__device__ inline void colsum_tile(const ScoreArgs& a, const ChunkPos& cp, int32_t t0, const bf16x8_t (&qa)[RB][4],
                                   const bf16x8_t (&kb)[4][4], const float (&lse)[RB][4], float (&col)[4]) {
  const float scale2 = 1.4426950408889634f * 0.08838834764831845f;
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    if (block_of<NW>(b) >= a.blocks) break;  // wave-uniform: padding blocks do no work
    f32x4_t acc[4];
    tile_logits<RB>(qa, kb, b, acc);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      int32_t lim = 0;
      if (MASK) lim = min(row_limit<NW>(a, cp, b, i), cp.c1 - 1);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        float p = __builtin_amdgcn_exp2f(fmaf(acc[t][i], scale2, -lse[b][i]));
        if (MASK && t0 + t * 16 + (lane & 15) > lim) p = 0.0f;
        col[t] += p;
      }
    }
  }
}

// Pass 2.  A_j = (1/G) sum over rows of 2^(x_rj - lse_r): the lane's four
// rows per block are summed in registers, then across the four lane groups
// that share a key column, then across waves in LDS.
template <int RB, int NW>
__global__ __launch_bounds__(NW * 64) void score_colsum_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ks[2][kTileKeys * kKStride];
  __shared__ float red[2][NW][kTileKeys];  // per LDS buffer: no barrier between read and next write
  const int unit = blockIdx.y;
  const ChunkPos cp = locate_chunk(a.lay, a.chunk, blockIdx.x);
  if (cp.seq < 0) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float inv_g = 1.0f / float(a.group);

  bf16x8_t qa[RB][4];
  load_queries<RB, NW>(a, cp, unit, qa);
  float lse[RB][4];
  const float* lrow = a.lse2 + (size_t(unit) * a.lay.n_seqs + cp.seq) * a.rows_pad;
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) lse[b][i] = lrow[block_of<NW>(b) * 16 + (lane >> 4) * 4 + i];

  const uint16_t* kseq = a.k + (size_t(unit) * a.lay.total_tokens + cp.seq_start) * kHeadDim;
  float* aout = a.a_base + size_t(unit) * a.lay.total_tokens + cp.seq_start;
  const int32_t clean_end = min(cp.c1, cp.seq_len - a.window + 1);
  KeyStager<NW> st;
  st.fetch(kseq, cp.c0, cp.c1);
  st.stage(ks[0]);
  __syncthreads();
  int buf = 0;
  for (int32_t t0 = cp.c0; t0 < cp.c1; t0 += kTileKeys) {
    const bool more = t0 + kTileKeys < cp.c1;
    if (more) st.fetch(kseq, t0 + kTileKeys, cp.c1);
    bf16x8_t kb[4][4];
    read_b_operand(ks[buf], kb);
    float col[4] = {0.f, 0.f, 0.f, 0.f};
    if (t0 + kTileKeys <= clean_end)
      colsum_tile<RB, NW, false>(a, cp, t0, qa, kb, lse, col);
    else
      colsum_tile<RB, NW, true>(a, cp, t0, qa, kb, lse, col);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      col[t] += __shfl_xor(col[t], 16);
      col[t] += __shfl_xor(col[t], 32);
    }
    if (lane < 16) {
#pragma unroll
      for (int t = 0; t < 4; ++t) red[buf][wave][t * 16 + lane] = col[t];
    }
    if (more) st.stage(ks[buf ^ 1]);
    __syncthreads();
    if (threadIdx.x < kTileKeys) {
      float s = 0.0f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += red[buf][w][threadIdx.x];
      const int32_t j = t0 + threadIdx.x;
      if (j < cp.c1) aout[j] = s * inv_g;
    }
    buf ^= 1;
  }
}

template <int RB, int NW>
hipError_t launch_rb(const ScoreArgs& a, hipStream_t stream) {
  const dim3 grid(a.total_chunks, a.lay.n_units);
  const dim3 block(64 * NW);
  hipLaunchKernelGGL((score_rowstats_kernel<RB, NW>), grid, block, 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(score_combine_kernel, dim3(a.lay.n_seqs, a.lay.n_units), dim3(256), 0, stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((score_colsum_kernel<RB, NW>), grid, block, 0, stream, a);
  return hipGetLastError();
}

template <int NW>
hipError_t launch_nw(const ScoreArgs& a, hipStream_t stream) {
  switch (a.row_blocks) {
    case 1: return launch_rb<1, NW>(a, stream);
    case 2: return launch_rb<2, NW>(a, stream);
    case 3: return launch_rb<3, NW>(a, stream);
    case 4: return launch_rb<4, NW>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_score_window(const ScoreArgs& a, hipStream_t stream) {
  switch (a.waves) {
    case 1: return launch_nw<1>(a, stream);
    case 2: return launch_nw<2>(a, stream);
    case 4: return launch_nw<4>(a, stream);
    case 8: return launch_nw<8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace stlite
