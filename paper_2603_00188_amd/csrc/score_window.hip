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
// the MFMA A operand (up to eight waves, each owning up to four 16-row blocks)
// and stream 64-key tiles of K, DMA'd into a three-stage LDS ring, as the B
// operand shared by all waves.  Inside a wave the MFMAs of one row block run
// under the softmax arithmetic of the previous one.
// Logits are kept in log2 units: x = (q . k) * log2(e) / sqrt(d).
#include "stlite_internal.h"
#include "tile_lds.h"

namespace stlite {
namespace {

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

// Q K^T of half a tile (32 keys: sub-tiles 2h and 2h+1) for row block b: two
// 16x16 accumulators, two interleaved MFMA chains over the k-steps.
template <int RB>
__device__ inline void half_logits(const bf16x8_t (&qa)[RB][4], const bf16x8_t (&kb)[2][4], int b, f32x4_t (&acc)[2]) {
#pragma unroll
  for (int t = 0; t < 2; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
#pragma unroll
    for (int t = 0; t < 2; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[b][kk], kb[t][kk], acc[t], 0, 0, 0);
}

__device__ inline void load_half_b(const uint16_t* tile, int h, bf16x8_t (&kb)[2][4]) {
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) kb[t][kk] = tile_b_operand(tile, 2 * h + t, kk);
}

// Ask the scheduler to alternate one MFMA with `valu` vector instructions, so
// that the softmax arithmetic of one group of blocks runs under the next
// group's MFMAs (8 MFMAs per block).
template <int valu, int GP>
__device__ inline void interleave_mfma_valu() {
#pragma unroll
  for (int i = 0; i < 8 * GP; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, valu, 0);
  }
}

// Masked tiles read each window row's last visible key (local index; -1 for
// padding rows) from a small LDS table instead of keeping it in VGPRs.
__device__ inline void fill_row_limits(const ScoreArgs& a, const ChunkPos& cp, int32_t* lim_s) {
  for (int r = threadIdx.x; r < a.rows_pad; r += blockDim.x)
    lim_s[r] = r < a.rows ? min(cp.seq_len - a.window + (r % a.window), cp.c1 - 1) : -1;
}

// Sets the two values of row i of block b (sub-tiles 2h, 2h+1) that the row
// may not see to -inf.
template <int NW, bool MASK>
__device__ inline void mask_pair(int32_t t0, int h, int b, int i, const int32_t* lim_s, float (&v)[2]) {
  if (MASK) {
    const int lane = threadIdx.x & 63;
    const int32_t lim = lim_s[block_of<NW>(b) * 16 + (lane >> 4) * 4 + i];
#pragma unroll
    for (int t = 0; t < 2; ++t)
      if (t0 + (2 * h + t) * 16 + (lane & 15) > lim) v[t] = -INFINITY;
  }
}

// Pass 1 keeps, per lane and window row, an offset o (log2 units) and
// sum = sum of 2^(x s - o) over the lane's keys, s = log2(e)/sqrt(d).  The
// offsets are the lane's row maxima over the chunk's first tile; every tile
// then only adds 2^(x s - o).  A logit more than ~128 above its offset
// overflows the sum to +inf, and score_rowstats_exact_kernel recomputes that
// chunk.
constexpr float kScale2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)
// Row blocks whose MFMAs are issued together (2 accumulators each).
constexpr int kRowGroup = 2;
constexpr int kColGroup = 2;

template <int RB, int NW, bool MASK>
__device__ inline void rowstats_half(int32_t t0, int h, int b, const f32x4_t (&acc)[2], const int32_t* lim_s,
                                     const float (&o)[RB][4], float (&sum)[RB][4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float v[2] = {acc[0][i], acc[1][i]};
    mask_pair<NW, MASK>(t0, h, b, i, lim_s, v);
    sum[b][i] += __builtin_amdgcn_exp2f(fmaf(v[0], kScale2, -o[b][i])) +
                 __builtin_amdgcn_exp2f(fmaf(v[1], kScale2, -o[b][i]));
  }
}

template <int RB, int NW, bool MASK>
__device__ inline void colsum_half(int32_t t0, int h, int b, const f32x4_t (&acc)[2], const int32_t* lim_s,
                                   const float (&lse)[RB][4], float (&col)[2]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float v[2] = {acc[0][i], acc[1][i]};
    mask_pair<NW, MASK>(t0, h, b, i, lim_s, v);
    col[0] += __builtin_amdgcn_exp2f(fmaf(v[0], kScale2, -lse[b][i]));
    col[1] += __builtin_amdgcn_exp2f(fmaf(v[1], kScale2, -lse[b][i]));
  }
}

// Q K^T of half a tile for the blocks of group g (GP blocks from block g*GP):
// 2*GP independent 16x16 accumulators, interleaved over the k-steps.
template <int RB, int GP>
__device__ inline void group_logits(const bf16x8_t (&qa)[RB][4], const bf16x8_t (&kb)[2][4], int g, bool last_real,
                                    f32x4_t (&acc)[GP][2]) {
#pragma unroll
  for (int j = 0; j < GP; ++j)
#pragma unroll
    for (int t = 0; t < 2; ++t) acc[j][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
#pragma unroll
    for (int j = 0; j < GP; ++j) {
      const int b = g * GP + j;
      if (b < RB - 1 || (b == RB - 1 && last_real))
#pragma unroll
        for (int t = 0; t < 2; ++t)
          acc[j][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qa[b][kk], kb[t][kk], acc[j][t], 0, 0, 0);
    }
}

// One tile of pass 1 (PASS == 1) or pass 2 (PASS == 2), as two 32-key halves;
// within a half the blocks go in groups of GP, and the MFMAs of group g+1 are
// issued among the vector instructions of group g.
template <int RB, int NW, int PASS, bool MASK, int GP>
__device__ inline void score_tile(const ScoreArgs& a, int32_t t0, const bf16x8_t (&qa)[RB][4], const uint16_t* tile,
                                  const int32_t* lim_s, const float (&o)[RB][4], float (&sum)[RB][4],
                                  float (&col)[4]) {
  constexpr int NG = (RB + GP - 1) / GP;
  const bool last_real = block_of<NW>(RB - 1) < a.blocks;  // wave-uniform
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    bf16x8_t kb[2][4];
    load_half_b(tile, h, kb);
    f32x4_t acc[2][GP][2];
    group_logits<RB, GP>(qa, kb, 0, last_real, acc[0]);
    float c2[2] = {0.f, 0.f};
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if (g + 1 < NG) group_logits<RB, GP>(qa, kb, g + 1, last_real, acc[(g + 1) & 1]);
#pragma unroll
      for (int j = 0; j < GP; ++j) {
        const int b = g * GP + j;
        if (b < RB - 1 || (b == RB - 1 && last_real)) {
          if (PASS == 1)
            rowstats_half<RB, NW, MASK>(t0, h, b, acc[g & 1][j], lim_s, o, sum);
          else
            colsum_half<RB, NW, MASK>(t0, h, b, acc[g & 1][j], lim_s, o, c2);
        }
      }
      interleave_mfma_valu<3, GP>();
      __builtin_amdgcn_sched_barrier(0);  // at most two groups' accumulators live
    }
    if (PASS == 2) {
      col[2 * h] += c2[0];
      col[2 * h + 1] += c2[1];
    }
  }
}

// Merge the 16 lanes that hold the same rows (different key columns) and
// write the chunk's (offset, sum) per window row; log2 units.
template <int RB, int NW>
__device__ inline void write_partials(const ScoreArgs& a, const ChunkPos& cp, int unit, const float (&o)[RB][4],
                                      const float (&sum)[RB][4]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mm = o[b][i], ss = sum[b][i];
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

// Pass 1 offsets: the lane's maximum of each row over the first tile (raw
// logits of masked-out keys excluded; a row that sees none of them sees none
// of the chunk's later keys either and gets kNegBig).
template <int RB, int NW>
__device__ inline void first_tile_offsets(const ScoreArgs& a, int32_t t0, const bf16x8_t (&qa)[RB][4],
                                          const uint16_t* tile, const int32_t* lim_s, float (&o)[RB][4]) {
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    float mx[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
    if (block_of<NW>(b) < a.blocks) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        bf16x8_t kb[2][4];
        load_half_b(tile, h, kb);
        f32x4_t acc[2];
        half_logits<RB>(qa, kb, b, acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v[2] = {acc[0][i], acc[1][i]};
          mask_pair<NW, true>(t0, h, b, i, lim_s, v);
          mx[i] = __builtin_fmaxf(__builtin_fmaxf(mx[i], v[0]), v[1]);
        }
      }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) o[b][i] = mx[i] == -INFINITY ? kNegBig : mx[i] * kScale2;
  }
}

template <int RB, int NW>
__global__ __launch_bounds__(NW * 64) void score_rowstats_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ks0[kTileElems], ks1[kTileElems], ks2[kTileElems];
  __shared__ int32_t lim_s[NW * RB * 16];
  __shared__ int32_t risky;
  const int unit = blockIdx.y;
  const ChunkPos cp = locate_chunk(a.lay, a.chunk, blockIdx.x);
  if (cp.seq < 0) return;
  if (threadIdx.x == 0) risky = 0;
  fill_row_limits(a, cp, lim_s);
  bf16x8_t qa[RB][4];
  load_queries<RB, NW>(a, cp, unit, qa);

  const uint16_t* kseq = a.k + (size_t(unit) * a.lay.total_tokens + cp.seq_start) * kHeadDim;
  const TileDma<NW> dma;
  // Tiles that end before the window starts are visible to every row: no mask.
  const int32_t clean_end = min(cp.c1, cp.seq_len - a.window + 1);
  const int32_t ntiles = (cp.c1 - cp.c0 + kTileKeys - 1) / kTileKeys;
  constexpr int kLoads = 16 / NW;  // tile DMA wave-loads per wave
  dma.issue(kseq, cp.c0, cp.c1 - 1, ks0);
  if (ntiles > 1) dma.issue(kseq, cp.c0 + kTileKeys, cp.c1 - 1, ks1);

  float o[RB][4], sum[RB][4], col_unused[4];
  {
    if (ntiles > 1) wait_vmcnt<kLoads>(); else wait_vmcnt<0>();
    barrier_lds();
    first_tile_offsets<RB, NW>(a, cp.c0, qa, ks0, lim_s, o);
  }
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) sum[b][i] = 0.0f;

  auto step = [&](int32_t n, const uint16_t* tile, uint16_t* nxt) {
    if (n > 0) {
      if (n + 1 < ntiles) wait_vmcnt<kLoads>(); else wait_vmcnt<0>();
      barrier_lds();
    }
    if (n + 2 < ntiles) dma.issue(kseq, cp.c0 + (n + 2) * kTileKeys, cp.c1 - 1, nxt);
    const int32_t t0 = cp.c0 + n * kTileKeys;
    if (t0 + kTileKeys <= clean_end)
      score_tile<RB, NW, 1, false, kRowGroup>(a, t0, qa, tile, lim_s, o, sum, col_unused);
    else
      score_tile<RB, NW, 1, true, kRowGroup>(a, t0, qa, tile, lim_s, o, sum, col_unused);
  };
  for (int32_t n = 0; n < ntiles; n += 3) {
    step(n, ks0, ks2);
    if (n + 1 < ntiles) step(n + 1, ks1, ks0);
    if (n + 2 < ntiles) step(n + 2, ks2, ks1);
  }

  write_partials<RB, NW>(a, cp, unit, o, sum);
  bool bad = false;
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) bad |= !(sum[b][i] < INFINITY);
  if (__ballot(bad) != 0 && (threadIdx.x & 63) == 0) atomicOr(&risky, 1);
  __syncthreads();
  if (threadIdx.x == 0) a.redo[size_t(unit) * a.total_chunks + cp.gchunk] = risky;
}

// Exact pass 1 for the chunks flagged by score_rowstats_kernel: a running row
// max per lane with the sums rescaled on every tile (plain staging; it only
// runs when a chunk's logits rise far enough above the first tile's to overflow the
// lean pass's sums).
template <int RB, int NW>
__global__ __launch_bounds__(NW * 64) void score_rowstats_exact_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ks0[kTileElems];
  __shared__ int32_t lim_s[NW * RB * 16];
  const int unit = blockIdx.y;
  if (a.redo[size_t(unit) * a.total_chunks + blockIdx.x] == 0) return;
  const ChunkPos cp = locate_chunk(a.lay, a.chunk, blockIdx.x);
  if (cp.seq < 0) return;
  fill_row_limits(a, cp, lim_s);
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
  const TileDma<NW> dma;
  for (int32_t t0 = cp.c0; t0 < cp.c1; t0 += kTileKeys) {
    __syncthreads();
    dma.issue(kseq, t0, cp.c1 - 1, ks0);
    wait_vmcnt<0>();
    __syncthreads();
#pragma unroll
    for (int b = 0; b < RB; ++b) {
      if (block_of<NW>(b) >= a.blocks) break;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        bf16x8_t kb[2][4];
        load_half_b(ks0, h, kb);
        f32x4_t acc[2];
        half_logits<RB>(qa, kb, b, acc);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v[2] = {acc[0][i], acc[1][i]};
          mask_pair<NW, true>(t0, h, b, i, lim_s, v);
          const float mx = __builtin_fmaxf(__builtin_fmaxf(m[b][i], v[0]), v[1]);
          const float ms = mx * kScale2;
          sum[b][i] = sum[b][i] * __builtin_amdgcn_exp2f(fmaf(m[b][i], kScale2, -ms)) +
                      __builtin_amdgcn_exp2f(fmaf(v[0], kScale2, -ms)) +
                      __builtin_amdgcn_exp2f(fmaf(v[1], kScale2, -ms));
          m[b][i] = mx;
        }
      }
    }
  }
  float o[RB][4];
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) o[b][i] = m[b][i] * kScale2;
  write_partials<RB, NW>(a, cp, unit, o, sum);
}

// Per (sequence, row): lse = log2 of the softmax denominator over the
// sequence's chunks.  Each chunk's (offset, sum) is first turned into its
// log2 total, so that the merge cannot overflow however large a chunk's sum.
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
      float M = -INFINITY;
      for (int32_t c = 0; c < nch; ++c) {
        const float2 v = pr[size_t(c) * a.rows_pad];
        M = fmaxf(M, v.x + __log2f(v.y));
      }
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
// Pass 2.  A_j = (1/G) sum over rows of 2^(x_rj - lse_r): the lane's four
// rows per block are summed in registers, then across the four lane groups
// that share a key column, then across waves in LDS.
template <int RB, int NW>
__global__ __launch_bounds__(NW * 64) void score_colsum_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ks0[kTileElems], ks1[kTileElems], ks2[kTileElems];
  __shared__ float red0[NW][kTileKeys], red1[NW][kTileKeys], red2[NW][kTileKeys];
  __shared__ int32_t lim_s[NW * RB * 16];
  const int unit = blockIdx.y;
  const ChunkPos cp = locate_chunk(a.lay, a.chunk, blockIdx.x);
  if (cp.seq < 0) return;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float inv_g = 1.0f / float(a.group);

  fill_row_limits(a, cp, lim_s);
  bf16x8_t qa[RB][4];
  load_queries<RB, NW>(a, cp, unit, qa);
  float lse[RB][4];
  const float* lrow = a.lse2 + (size_t(unit) * a.lay.n_seqs + cp.seq) * a.rows_pad;
#pragma unroll
  for (int b = 0; b < RB; ++b)
#pragma unroll
    for (int i = 0; i < 4; ++i) lse[b][i] = lrow[block_of<NW>(b) * 16 + (lane >> 4) * 4 + i];

  const uint16_t* kseq = a.k + (size_t(unit) * a.lay.total_tokens + cp.seq_start) * kHeadDim;
  const TileDma<NW> dma;
  float* aout = a.a_base + size_t(unit) * a.lay.total_tokens + cp.seq_start;
  const int32_t clean_end = min(cp.c1, cp.seq_len - a.window + 1);
  const int32_t ntiles = (cp.c1 - cp.c0 + kTileKeys - 1) / kTileKeys;
  constexpr int kLoads = 16 / NW;
  // Column sums of tile n are reduced across waves after the barrier of step n+1.
  auto reduce = [&](int32_t n, const float (&r)[NW][kTileKeys]) {
    if (threadIdx.x < kTileKeys) {
      float s = 0.0f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += r[w][threadIdx.x];
      const int32_t j = cp.c0 + n * kTileKeys + threadIdx.x;
      if (j < cp.c1) aout[j] = s * inv_g;
    }
  };
  dma.issue(kseq, cp.c0, cp.c1 - 1, ks0);
  if (ntiles > 1) dma.issue(kseq, cp.c0 + kTileKeys, cp.c1 - 1, ks1);
  float sum_unused[RB][4];
  auto step = [&](int32_t n, const uint16_t* tile, uint16_t* nxt, float (&r)[NW][kTileKeys],
                  const float (&rprev)[NW][kTileKeys]) {
    if (n + 1 < ntiles) wait_vmcnt<kLoads>(); else wait_vmcnt<0>();
    barrier_lds();
    if (n > 0) reduce(n - 1, rprev);
    if (n + 2 < ntiles) dma.issue(kseq, cp.c0 + (n + 2) * kTileKeys, cp.c1 - 1, nxt);
    const int32_t t0 = cp.c0 + n * kTileKeys;
    float col[4] = {0.f, 0.f, 0.f, 0.f};
    if (t0 + kTileKeys <= clean_end)
      score_tile<RB, NW, 2, false, kColGroup>(a, t0, qa, tile, lim_s, lse, sum_unused, col);
    else
      score_tile<RB, NW, 2, true, kColGroup>(a, t0, qa, tile, lim_s, lse, sum_unused, col);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      col[t] += __shfl_xor(col[t], 16);
      col[t] += __shfl_xor(col[t], 32);
    }
    if (lane < 16) {
#pragma unroll
      for (int t = 0; t < 4; ++t) r[wave][t * 16 + lane] = col[t];
    }
  };
  for (int32_t n = 0; n < ntiles; n += 3) {
    step(n, ks0, ks2, red0, red2);
    if (n + 1 < ntiles) step(n + 1, ks1, ks0, red1, red0);
    if (n + 2 < ntiles) step(n + 2, ks2, ks1, red2, red1);
  }
  barrier_lds();
  const int last = (ntiles - 1) % 3;
  reduce(ntiles - 1, last == 0 ? red0 : (last == 1 ? red1 : red2));
}

template <int RB, int NW>
hipError_t launch_rb(const ScoreArgs& a, hipStream_t stream) {
  const dim3 grid(a.total_chunks, a.lay.n_units);
  const dim3 block(64 * NW);
  hipLaunchKernelGGL((score_rowstats_kernel<RB, NW>), grid, block, 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((score_rowstats_exact_kernel<RB, NW>), grid, block, 0, stream, a);
  e = hipGetLastError();
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
