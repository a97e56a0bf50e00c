// Window base score A_base (Eq. base_attention) for every (layer, kv head,
// sequence): A_i = (1/G) sum_g sum_w softmax_{j <= p_w}(q_{g,w} . k_j / sqrt(d))_i.
//
// A column sum of softmax rows needs every row's normaliser first, so the
// logits Q K^T are formed twice on the matrix cores (bf16 MFMA, fp32
// accumulate):
//   pass 1  per key chunk: per window row, sum of 2^(x - o) for a fixed
//           offset o (the maximum over the chunk's first tile of the row's
//           group of eight rows),
//   combine per row: log2 of the softmax denominator over all chunks,
//   pass 2  per key chunk: 2^(x - lse) summed over the G*window rows.
// Logits are kept in log2 units: x = (q . k) * log2(e) / sqrt(d).
//
// Both passes use v_mfma_f32_32x32x16_bf16.  A work-group holds the whole
// GQA group's window queries resident in VGPRs as the A operand (ceil(blocks
// / 2) waves, each with up to two 32-row blocks) and streams 64-key tiles of K -- two 32-key blocks --
// through a three-stage LDS ring filled by DMA; the tiles are the B operand
// shared by all waves.  Every exponential and sum of one key block is issued
// between the MFMAs of the other, in an order fixed in the source: the long
// 32x32 MFMAs hide that vector work, which the short 16x16 forms cannot.
#include <algorithm>

#include "stlite_internal.h"
#include "tile_lds.h"

namespace stlite {
namespace {

constexpr float kNegBig = -1.0e30f;
constexpr float kScale2 = 1.4426950408889634f * 0.08838834764831845f;  // log2(e)/sqrt(128)

// Second launch-bound argument: the minimum number of waves per SIMD the
// register allocator budgets for (HIP's meaning of it).  Two (256 registers
// each) for groups of three or more waves: their resident queries fill the
// register file at two waves per SIMD, and an 8-wave group needs two waves on
// every SIMD at once.  One for the one- and two-wave groups of the smallest
// windows, whose resident queries need more registers than a higher target
// leaves.
template <int NW>
constexpr int kScoreMinGroups = NW <= 2 ? 1 : 2;

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

__device__ inline int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Row-block layouts of the score passes (a unit is one 32-row block against
// one 32-key block of a tile: eight MFMAs and 16 logits per lane).
//   kPlain:    wave w owns blocks w + j NW (j < RB), both key blocks.
//   kBalanced: 14 blocks on 8 waves.  Waves w and w + 4 of an 8-wave group
//              run on the same SIMD, and the passes are bound by each SIMD's
//              vector work, so a tile's 28 units are spread 7 per SIMD (the
//              plain layouts leave 8 on some SIMDs: 7 waves put 8, 8, 8 and 4
//              there): waves 0-3 own blocks 2w and 2w + 1 (4 units), waves 4-7
//              own block w + 4 (2 units) and one key block, w & 1, of block
//              10 + w / 2, i.e. 12 or 13 (1 unit).  The two waves sharing a
//              block add their row sums (pass 1) and each give the column
//              sums of their own key block (pass 2).
constexpr int kPlain = 0, kBalanced = 1;

template <int NW, int MODE = kPlain>
__device__ inline int block_of(int j) {
  const int w = wave_id();
  if constexpr (MODE == kBalanced) return w < 4 ? 2 * w + j : (j == 0 ? w + 4 : 10 + (w >> 1));
  else return w + j * NW;
}

// Units a wave of kind KIND owns: kind 0 every (row block, key block); kinds
// 1 and 2 (balanced waves 4-7 with w & 1 = KIND - 1) only key block KIND - 1
// of their second block.
template <int KIND>
constexpr bool owns(int rb, int kb) { return KIND == 0 || rb == 0 || kb == KIND - 1; }

// Window queries as the A operand: lane l holds row l & 31 of each block;
// k-step kk takes dims 16 kk + 8 (l >> 5) .. +7.
template <int RB, int NW, int MODE = kPlain>
__device__ inline void load_queries(const ScoreArgs& a, const ChunkPos& cp, int unit, bf16x8_t (&qa)[RB][8]) {
  const int lane = threadIdx.x & 63;
  const int layer = unit / a.lay.n_kv_heads, kv = unit % a.lay.n_kv_heads;
  const uint16_t* qbase =
      a.q + ((size_t(layer) * a.lay.n_seqs + cp.seq) * a.n_q_heads + size_t(kv) * a.group) * a.window * kHeadDim;
#pragma unroll
  for (int b = 0; b < RB; ++b) {
    const int row = block_of<NW, MODE>(b) * 32 + (lane & 31);
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (row < a.rows)
        v = *reinterpret_cast<const uint4*>(qbase + size_t(row) * kHeadDim + kk * 16 + (lane >> 5) * 8);
      qa[b][kk] = __builtin_bit_cast(bf16x8_t, v);
    }
  }
}

// Each window row's last visible key (local index; -1 for padding rows), in
// LDS for the masked tiles.
__device__ inline void fill_row_limits(const ScoreArgs& a, const ChunkPos& cp, int32_t* lim_s) {
  for (int r = threadIdx.x; r < a.rows_pad; r += blockDim.x)
    lim_s[r] = r < a.rows ? min(cp.seq_len - a.window + (r % a.window), cp.c1 - 1) : -1;
}

// Accumulator start of a masked tile: -inf where the row may not see the key
// (past its causal limit or past the chunk), 0 elsewhere.
template <int NW, int MODE = kPlain>
__device__ inline f32x16_t mask_init(int32_t t0, int kb, int rb, const int32_t* lim_s) {
  const int lane = threadIdx.x & 63;
  const int32_t key = t0 + kb * 32 + (lane & 31);
  const int base = block_of<NW, MODE>(rb) * 32;
  f32x16_t m;
#pragma unroll
  for (int i = 0; i < 16; ++i) m[i] = key > lim_s[base + acc32_row(i, lane)] ? -INFINITY : 0.0f;
  return m;
}

// Butterfly over the 32 lanes that hold the same rows (xor 1 .. 16).
__device__ inline float row_max32(float v) {
#pragma unroll
  for (int o = 1; o < 32; o <<= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// Sum of v over the 32 lanes holding the same rows, for all 16 registers at
// once: a reduce-scatter that halves the registers each level (xor 16 .. 1).
// On return v[0] of lane l holds the total of register reg_of(l) where
// reg_of(l) = 8 b4 + 4 b3 + 2 b2 + b1 + ... (the lane's bits 4..1 pick it).
__device__ inline float sum32_scatter(float (&v)[16]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int lvl = 0; lvl < 4; ++lvl) {
    const int half = 8 >> lvl;            // registers kept after this level
    const int bit = (lane >> (4 - lvl)) & 1;  // lane bit 4, 3, 2, 1
#pragma unroll
    for (int j = 0; j < half; ++j) {
      const float send = bit ? v[j] : v[j + half];
      const float keep = bit ? v[j + half] : v[j];
      v[j] = keep + __shfl_xor(send, 16 >> lvl);
    }
  }
  return v[0] + __shfl_xor(v[0], 1);
}

// Register that sum32_scatter leaves in lane l.
__device__ inline int scatter_reg(int lane) {
  return 8 * ((lane >> 4) & 1) + 4 * ((lane >> 3) & 1) + 2 * ((lane >> 2) & 1) + ((lane >> 1) & 1);
}

// Shared memory of a score-pass work-group.
template <int RB, int NW>
struct ScoreShared {
  uint16_t ks0[kTileElems] __attribute__((aligned(16)));
  uint16_t ks1[kTileElems] __attribute__((aligned(16)));
  uint16_t ks2[kTileElems] __attribute__((aligned(16)));
  int32_t lim_s[NW * RB * 32];
  float red_s[2][NW][kTileKeys];
  float xch[2][32];  // balanced pass 1: the second sharing wave's row sums of blocks 12 and 13
  int32_t risky;
};

// One pass over a chunk of keys.  PASS 1 writes per-row (offset, sum) for the
// chunk (and flags the chunk if a sum overflowed); PASS 2 writes A for the
// chunk's keys.  KIND: which units of its blocks the wave owns (owns<KIND>).
template <int PASS, int RB, int NW, int MODE, int KIND>
__device__ __forceinline__ void score_pass_body(const ScoreArgs& a, ScoreShared<RB, NW>& sh, const ChunkPos& cp,
                                                int unit) {
  uint16_t* const ks0 = sh.ks0;
  uint16_t* const ks1 = sh.ks1;
  uint16_t* const ks2 = sh.ks2;
  int32_t* const lim_s = sh.lim_s;
  const int lane = threadIdx.x & 63;
  const int wave = wave_id();
  // The wave's last block may lie past the real rows (uniform; plain layout).
  const bool last_real = block_of<NW, MODE>(RB - 1) < a.blocks;

  bf16x8_t qa[RB][8];
  load_queries<RB, NW, MODE>(a, cp, unit, qa);
  // Pass 1: offsets o of the row groups g = i >> 2 (rows 8 g .. 8 g + 7 of a
  // block); pass 2: row log-normalisers lse.  Both in log2 units.
  float ofs[RB][4];
  float lse[RB][16];
  if (PASS == 2) {
    const float* lrow = a.lse2 + (size_t(unit) * a.lay.n_seqs + cp.seq) * a.rows_pad;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < 16; ++i) lse[rb][i] = lrow[block_of<NW, MODE>(rb) * 32 + acc32_row(i, lane)];
  }

  const uint16_t* kseq = a.k + (size_t(unit) * a.lay.total_tokens + cp.seq_start) * kHeadDim;
  const TileDma<NW> dma;
  // Tiles that end before the window starts are visible to every row: no mask.
  const int32_t clean_end = min(cp.c1, cp.seq_len - a.window + 1);
  const int32_t ntiles = (cp.c1 - cp.c0 + kTileKeys - 1) / kTileKeys;
  dma.issue(kseq, cp.c0, cp.c1 - 1, ks0);
  if (ntiles > 1) dma.issue(kseq, cp.c0 + kTileKeys, cp.c1 - 1, ks1);

  f32x16_t acc[2][RB];  // [key block][row block]
  bf16x8_t kbuf[4];     // B fragments g = 8 kb + kk, read three MFMA groups ahead
  float sum[RB][16];    // pass 1
  float col[2];         // pass 2: two partial column sums of the block being summed
  const float inv_g = 1.0f / float(a.group);
  float* aout = a.a_base + size_t(unit) * a.lay.total_tokens + cp.seq_start;

  auto read_b = [&](const uint16_t* tile, int g) { kbuf[g % 4] = tile_b32_operand(tile, g / 8, g % 8); };
  // Rows of a padded block are zero queries: their MFMAs run (which keeps the
  // loop free of branches) but nothing of them is written.
  auto real = [&](int rb) { return rb < RB - 1 || last_real; };
  // Tiles before clean_end need no mask; only the chunk's last tiles can.
  const int32_t n_clean = max(0, min(ntiles, (clean_end - cp.c0) / kTileKeys));

  // Tile 0 (and tile 1) landed.
  wait_vmcnt<0>();
  barrier_lds();

  if (PASS == 1) {
    // Offsets: each row group's maximum over the first tile (masked keys
    // excluded; a group that sees none of them sees none of the chunk and
    // gets kNegBig).  A row far below its group's offset can underflow its
    // sum; the chunk is then flagged for the exact pass.  Every unit of the
    // wave's blocks is formed here, owned or not, so that the two waves
    // sharing a block take the same offsets.
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        read_b(ks0, 8 * kb + kk);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          acc[kb][rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
              qa[rb][kk], kbuf[(8 * kb + kk) % 4],
              kk == 0 ? mask_init<NW, MODE>(cp.c0, kb, rb, lim_s) : acc[kb][rb], 0, 0, 0);
      }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float m = -INFINITY;
#pragma unroll
        for (int i = 4 * g; i < 4 * g + 4; ++i) m = fmaxf(m, fmaxf(acc[0][rb][i], acc[1][rb][i]));
        m = row_max32(m);
        m = fmaxf(m, __shfl_xor(m, 32));
        ofs[rb][g] = m == -INFINITY ? kNegBig : m * kScale2;
      }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < 16; ++i) sum[rb][i] = 0.0f;
  }

  // Vector work on element i of row block rb of key block kb's accumulators.
  auto elem = [&](int kb, int rb, int i) {
    if (PASS == 1)
      sum[rb][i] += __builtin_amdgcn_exp2f(fmaf(acc[kb][rb][i], kScale2, -ofs[rb][i >> 2]));
    else
      col[i & 1] += __builtin_amdgcn_exp2f(fmaf(acc[kb][rb][i], kScale2, -lse[rb][i]));
  };
  // The same for two elements at a fixed place in the instruction stream:
  // the scale reaches them through an empty volatile asm on a scalar copy
  // and their results feed another, and such statements keep their order
  // relative to the scheduling barriers -- so the arithmetic can be neither
  // hoisted above the preceding MFMA nor sunk below the next one.
  auto elem_pinned = [&](int kb, int rb, int i) {
    float sc = kScale2;
    asm volatile("" : "+s"(sc));
    if (PASS == 1) {
      sum[rb][i] += __builtin_amdgcn_exp2f(fmaf(acc[kb][rb][i], sc, -ofs[rb][i >> 2]));
      sum[rb][i + 1] += __builtin_amdgcn_exp2f(fmaf(acc[kb][rb][i + 1], sc, -ofs[rb][i >> 2]));
      asm volatile("" ::"v"(sum[rb][i]), "v"(sum[rb][i + 1]));
    } else {
      col[0] += __builtin_amdgcn_exp2f(fmaf(acc[kb][rb][i], sc, -lse[rb][i]));
      col[1] += __builtin_amdgcn_exp2f(fmaf(acc[kb][rb][i + 1], sc, -lse[rb][i + 1]));
      asm volatile("" ::"v"(col[0]), "v"(col[1]));
    }
  };
  // Pass 2: the wave's column sums of key block kb of tile n go to LDS.
  auto put_cols = [&](int32_t n, int kb) {
    float c = col[0] + col[1];
    c += __shfl_xor(c, 32);
    if (lane < 32) sh.red_s[n & 1][wave][kb * 32 + lane] = c;
  };
  // Pass 2: A of tile n's keys, once every wave's column sums are in LDS.
  auto reduce = [&](int32_t n) {
    if (threadIdx.x < kTileKeys) {
      float s = 0.0f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += sh.red_s[n & 1][w][threadIdx.x];
      const int32_t j = cp.c0 + n * kTileKeys + threadIdx.x;
      if (j < cp.c1) aout[j] = s * inv_g;
    }
  };
  // Section kb of a clean tile: the MFMAs of key block kb, each MFMA followed
  // by the vector work on two elements of key block kb ^ 1 (i and i + 1 of
  // the same row group, i even), in that order; units the wave does not own
  // are left out.  B fragments past the tile's sixteen are the next tile's
  // first three.
  auto section = [&](int kb, const uint16_t* tile, const uint16_t* next) {
    col[0] = 0.0f;
    col[1] = 0.0f;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const int g = 8 * kb + kk;
      if (g + 3 < 16)
        read_b(tile, g + 3);
      else
        read_b(next, g + 3 - 16);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        if (owns<KIND>(rb, kb))
          acc[kb][rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[rb][kk], kbuf[g % 4],
                                                                kk == 0 ? f32x16_t{} : acc[kb][rb], 0, 0, 0);
        if (owns<KIND>(rb, kb ^ 1)) elem_pinned(kb ^ 1, rb, 2 * kk);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  if (n_clean > 0) {
    // The "previous key block 1" before the first tile contributes nothing.
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[1][rb][i] = -INFINITY;
    read_b(ks0, 0);
    read_b(ks0, 1);
    read_b(ks0, 2);
    // One clean tile.  Between its sections: wait for tile n+1's DMA, barrier
    // (every wave is past tile n-1, whose stage the DMA of tile n+2 then
    // overwrites), and in pass 2 the finished column sums of tile n-1.
    auto step = [&](int32_t n, const uint16_t* tile, const uint16_t* next, uint16_t* nxt2) {
      section(0, tile, next);
      if (PASS == 2) put_cols(n - 1, 1);
      wait_vmcnt<0>();
      barrier_lds();
      if (PASS == 2 && n > 0) reduce(n - 1);
      if (n + 2 < ntiles) dma.issue(kseq, cp.c0 + (n + 2) * kTileKeys, cp.c1 - 1, nxt2);
      __builtin_amdgcn_sched_barrier(0);
      section(1, tile, next);
      if (PASS == 2) put_cols(n, 0);
    };
    for (int32_t n = 0; n < n_clean; n += 3) {
      step(n, ks0, ks1, ks2);
      if (n + 1 < n_clean) step(n + 1, ks1, ks2, ks0);
      if (n + 2 < n_clean) step(n + 2, ks2, ks0, ks1);
    }
    // Key block 1 of the last clean tile.
    col[0] = 0.0f;
    col[1] = 0.0f;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
      if (owns<KIND>(rb, 1))
#pragma unroll
        for (int i = 0; i < 16; ++i) elem(1, rb, i);
    if (PASS == 2) {
      put_cols(n_clean - 1, 1);
      barrier_lds();
      reduce(n_clean - 1);
    }
  }

  // The masked tiles at the end of the chunk, one at a time.
  auto stage = [&](int32_t n) { return n % 3 == 0 ? ks0 : (n % 3 == 1 ? ks1 : ks2); };
  for (int32_t n = n_clean; n < ntiles; ++n) {
    const int32_t t0 = cp.c0 + n * kTileKeys;
    wait_vmcnt<0>();
    barrier_lds();
    if (n + 2 < ntiles) dma.issue(kseq, t0 + 2 * kTileKeys, cp.c1 - 1, stage(n + 2));
    const uint16_t* tile = stage(n);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int kk = 0; kk < 8; ++kk) {
        read_b(tile, 8 * kb + kk);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb)
          if (owns<KIND>(rb, kb))
            acc[kb][rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                qa[rb][kk], kbuf[(8 * kb + kk) % 4],
                kk == 0 ? mask_init<NW, MODE>(t0, kb, rb, lim_s) : acc[kb][rb], 0, 0, 0);
      }
      col[0] = 0.0f;
      col[1] = 0.0f;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb)
        if (owns<KIND>(rb, kb))
#pragma unroll
          for (int i = 0; i < 16; ++i) elem(kb, rb, i);
      if (PASS == 2) put_cols(n, kb);
    }
    if (PASS == 2) {
      barrier_lds();
      reduce(n);
    }
  }

  if (PASS == 1) {
    // (offset, sum) per row: the offset is common to the 32 lanes of a row, so
    // the chunk's sum is a plain sum over them.  A row that sees a key of the
    // chunk but whose sum overflowed, or underflowed below 2^-60 (its logits
    // far under its group's offset), sends the chunk to the exact pass.
    float srow[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) srow[rb] = sum32_scatter(sum[rb]);
    const int i = scatter_reg(lane);
    if constexpr (MODE == kBalanced) {
      // A shared block's second wave hands its half of the row sums over.
      if (KIND == 2 && (lane & 1) == 0) sh.xch[(wave - 4) >> 1][acc32_row(i, lane)] = srow[1];
      __syncthreads();
      if (KIND == 1) srow[1] += sh.xch[(wave - 4) >> 1][acc32_row(i, lane)];
    }
    bool bad = false;
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      if (MODE == kBalanced && KIND == 2 && rb == 1) continue;  // written by the first sharing wave
      const float s = srow[rb];
      const int r = block_of<NW, MODE>(rb) * 32 + acc32_row(i, lane);
      float o = ofs[rb][0];
#pragma unroll
      for (int g = 1; g < 4; ++g) o = (i >> 2) == g ? ofs[rb][g] : o;
      if ((lane & 1) == 0 && real(rb)) {
        a.partial[(size_t(unit) * a.total_chunks + cp.gchunk) * a.rows_pad + r] = make_float2(o, s);
        bad |= r < a.rows && lim_s[r] >= cp.c0 && !(s >= 0x1.0p-60f && s < INFINITY);
      }
    }
    if (__ballot(bad) != 0 && lane == 0) atomicOr(&sh.risky, 1);
    __syncthreads();
    if (threadIdx.x == 0) a.redo[size_t(unit) * a.total_chunks + cp.gchunk] = sh.risky;
  }
}

template <int PASS, int RB, int NW, int MODE>
__global__ __launch_bounds__(NW * 64, kScoreMinGroups<NW>) void score_pass_kernel(ScoreArgs a) {
  __shared__ ScoreShared<RB, NW> sh;
  const int unit = blockIdx.y;
  const ChunkPos cp = locate_chunk(a.lay, a.chunk, blockIdx.x);
  if (cp.seq < 0) return;
  if (PASS == 1 && threadIdx.x == 0) sh.risky = 0;
  fill_row_limits(a, cp, sh.lim_s);
  if constexpr (MODE == kBalanced) {
    static_assert(NW == 8 && RB == 2, "the balanced layout is 14 blocks on 8 waves");
    const int w = wave_id();
    if (w < 4)
      score_pass_body<PASS, RB, NW, MODE, 0>(a, sh, cp, unit);
    else if (w & 1)
      score_pass_body<PASS, RB, NW, MODE, 2>(a, sh, cp, unit);
    else
      score_pass_body<PASS, RB, NW, MODE, 1>(a, sh, cp, unit);
  } else {
    score_pass_body<PASS, RB, NW, MODE, 0>(a, sh, cp, unit);
  }
}

// Exact pass 1 for the chunks flagged by the lean pass: a running row max per
// lane with the sums rescaled on every tile (plain staging; it only runs when
// a chunk's logits rise far enough above the first tile's to overflow the lean
// pass's sums).
template <int RB, int NW>
__global__ __launch_bounds__(NW * 64, kScoreMinGroups<NW>) void score_rowstats_exact_kernel(ScoreArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t ks0[kTileElems];
  __shared__ int32_t lim_s[NW * RB * 32];
  const int unit = blockIdx.y;
  // A few work-groups per unit walk the unit's chunks: most launches find no
  // flagged chunk, and the flag reads then cost little.
  for (int32_t x = blockIdx.x; x < a.total_chunks; x += gridDim.x) {
  if (a.redo[size_t(unit) * a.total_chunks + x] == 0) continue;
  const ChunkPos cp = locate_chunk(a.lay, a.chunk, x);
  if (cp.seq < 0) continue;
  __syncthreads();  // the previous chunk's readers of lim_s are done
  const int lane = threadIdx.x & 63;
  fill_row_limits(a, cp, lim_s);
  bf16x8_t qa[RB][8];
  load_queries<RB, NW>(a, cp, unit, qa);
  float m[RB][16], sum[RB][16];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      m[rb][i] = kNegBig;
      sum[rb][i] = 0.0f;
    }
  const uint16_t* kseq = a.k + (size_t(unit) * a.lay.total_tokens + cp.seq_start) * kHeadDim;
  const TileDma<NW> dma;
  for (int32_t t0 = cp.c0; t0 < cp.c1; t0 += kTileKeys) {
    __syncthreads();
    dma.issue(kseq, t0, cp.c1 - 1, ks0);
    wait_vmcnt<0>();
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      if (block_of<NW>(rb) >= a.blocks) break;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        f32x16_t acc = mask_init<NW>(t0, kb, rb, lim_s);
#pragma unroll
        for (int kk = 0; kk < 8; ++kk)
          acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qa[rb][kk], tile_b32_operand(ks0, kb, kk), acc, 0, 0, 0);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float mx = __builtin_fmaxf(m[rb][i], acc[i]);
          sum[rb][i] = sum[rb][i] * __builtin_amdgcn_exp2f((m[rb][i] - mx) * kScale2) +
                       __builtin_amdgcn_exp2f((acc[i] - mx) * kScale2);
          m[rb][i] = mx;
        }
      }
    }
  }
  // Merge the 32 lanes of each row: (max, sum) pairs in log2 units.
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float mm = m[rb][i] * kScale2, ss = sum[rb][i];
#pragma unroll
      for (int off = 1; off < 32; off <<= 1) {
        const float mo = __shfl_xor(mm, off);
        const float so = __shfl_xor(ss, off);
        const float mx = fmaxf(mm, mo);
        ss = ss * __builtin_amdgcn_exp2f(mm - mx) + so * __builtin_amdgcn_exp2f(mo - mx);
        mm = mx;
      }
      if ((lane & 31) == 0 && block_of<NW>(rb) < a.blocks) {
        const int r = block_of<NW>(rb) * 32 + acc32_row(i, lane);
        a.partial[(size_t(unit) * a.total_chunks + cp.gchunk) * a.rows_pad + r] = make_float2(mm, ss);
      }
    }
  }
}

// Per (sequence, row): lse = log2 of the softmax denominator over the
// sequence's chunks.  Each chunk's (offset, sum) is first turned into its
// log2 total t_c, and the totals are merged in one pass as a running maximum M
// with Z = sum 2^(t_c - M), so that the merge cannot overflow however large a
// chunk's sum.  One row per thread; work-group (row block of 64, sequence, unit).
__global__ __launch_bounds__(64) void score_combine_kernel(ScoreArgs a) {
  const int s = blockIdx.y, unit = blockIdx.z;
  const int r = blockIdx.x * 64 + threadIdx.x;
  if (r >= a.rows_pad) return;
  int32_t first = 0;
  for (int32_t t = 0; t < s; ++t) {
    const int32_t L = a.lay.cu_seqlens[t + 1] - a.lay.cu_seqlens[t];
    first += (L + a.chunk - 1) / a.chunk;
  }
  const int32_t L = a.lay.cu_seqlens[s + 1] - a.lay.cu_seqlens[s];
  const int32_t nch = (L + a.chunk - 1) / a.chunk;
  float out = INFINITY;  // padding rows contribute exp2(-inf) = 0 in pass 2
  if (r < a.rows) {
    const float2* pr = a.partial + (size_t(unit) * a.total_chunks + first) * a.rows_pad + r;
    float M = -INFINITY, Z = 0.0f;
#pragma unroll 8
    for (int32_t c = 0; c < nch; ++c) {
      const float2 v = pr[size_t(c) * a.rows_pad];
      const float t = v.x + __log2f(v.y);  // -inf for an empty sum
      if (t > M) {
        Z = Z * __builtin_amdgcn_exp2f(M - t) + 1.0f;
        M = t;
      } else if (t > -INFINITY) {
        Z += __builtin_amdgcn_exp2f(t - M);
      }
    }
    out = M + __log2f(Z);
  }
  a.lse2[(size_t(unit) * a.lay.n_seqs + s) * a.rows_pad + r] = out;
}

template <int RB, int NW, int MODE = kPlain>
hipError_t launch_rb(const ScoreArgs& a, hipStream_t stream) {
  const dim3 grid(a.total_chunks, a.lay.n_units);
  const dim3 block(64 * NW);
  hipLaunchKernelGGL((score_pass_kernel<1, RB, NW, MODE>), grid, block, 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((score_rowstats_exact_kernel<RB, NW>), dim3(std::min(a.total_chunks, 4), a.lay.n_units), block, 0,
                     stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(score_combine_kernel, dim3((a.rows_pad + 63) / 64, a.lay.n_seqs, a.lay.n_units), dim3(64), 0,
                     stream, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((score_pass_kernel<2, RB, NW, MODE>), grid, block, 0, stream, a);
  return hipGetLastError();
}

template <int NW>
hipError_t launch_nw(const ScoreArgs& a, hipStream_t stream) {
  switch (a.row_blocks) {
    case 1: return launch_rb<1, NW>(a, stream);
    case 2: return launch_rb<2, NW>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_score_window(const ScoreArgs& a, hipStream_t stream) {
  // The exact pass 1 keeps the plain 8-wave layout (blocks w and w + 8): it
  // writes whole rows, whichever waves hold them.
  if (a.balanced) return a.waves == 8 && a.row_blocks == 2 && a.blocks == 14 ? launch_rb<2, 8, kBalanced>(a, stream)
                                                                            : hipErrorInvalidValue;
  switch (a.waves) {
    case 1: return launch_nw<1>(a, stream);
    case 2: return launch_nw<2>(a, stream);
    case 3: return launch_nw<3>(a, stream);
    case 4: return launch_nw<4>(a, stream);
    case 5: return launch_nw<5>(a, stream);
    case 6: return launch_nw<6>(a, stream);
    case 7: return launch_nw<7>(a, stream);
    case 8: return launch_nw<8>(a, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace stlite
