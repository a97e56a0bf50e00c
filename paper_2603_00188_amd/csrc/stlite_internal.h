// Internal declarations shared by the host layer and the gfx950 kernels of
// libstlite.  Nothing here is part of the public ABI (include/stlite.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace stlite {

constexpr int kHeadDim = 128;
constexpr int kMaxWindowRows = 512;  // G * window limit (window queries stay in registers)

// ---------------------------------------------------------------------------
// Per-call launch descriptions (filled by the host layer, passed by value).
// ---------------------------------------------------------------------------

struct Layout {
  const int32_t* cu_seqlens;
  const int32_t* cu_frames;
  const int32_t* frame_meta;
  const int32_t* cu_budget;
  int32_t n_seqs;
  int32_t n_frames;
  int32_t n_units;       // n_layers * n_kv_heads
  int32_t n_kv_heads;
  int64_t total_tokens;
  int64_t total_budget;
};

// Token run g of a layout's non-frame tokens, [*b, *e): for g < n_frames the
// text after frame g, up to the next frame of its sequence or the sequence's
// end, preceded by frame g itself when with_current and frame g is its
// sequence's last (current) frame; for n_frames <= g < n_frames + n_seqs the
// text before sequence g - n_frames's first frame (all of it when it has no
// frame).  Runs of all g cover exactly the text (and current) tokens.
__device__ inline void token_run(const Layout& lay, int32_t g, bool with_current, int32_t* b, int32_t* e) {
  if (g < lay.n_frames) {
    int32_t lo = 0, hi = lay.n_seqs - 1;  // the sequence of frame g: last s with cu_frames[s] <= g
    while (lo < hi) {
      const int32_t mid = (lo + hi + 1) >> 1;
      if (lay.cu_frames[mid] <= g) lo = mid;
      else hi = mid - 1;
    }
    const bool last = g + 1 == lay.cu_frames[lo + 1];
    const int32_t start = lay.frame_meta[3 * g];
    *b = with_current && last ? start : start + lay.frame_meta[3 * g + 1] * lay.frame_meta[3 * g + 2];
    *e = last ? lay.cu_seqlens[lo + 1] : lay.frame_meta[3 * (g + 1)];
  } else {
    const int32_t s = g - lay.n_frames;
    *b = lay.cu_seqlens[s];
    *e = lay.cu_frames[s] < lay.cu_frames[s + 1] ? lay.frame_meta[3 * lay.cu_frames[s]] : lay.cu_seqlens[s + 1];
  }
}

struct ScoreArgs {
  Layout lay;
  const uint16_t* q;     // [layers][seqs][Hq][window][d]
  const uint16_t* k;     // [units][L][d]
  float* a_base;         // [units][L]
  float2* partial;       // workspace [units][total_chunks][rows_pad] (max, sum) in log2 units
  float* lse2;           // workspace [units][seqs][rows_pad]
  int32_t* redo;         // workspace [units][total_chunks]: chunk needs the exact pass 1
  int32_t n_q_heads;
  int32_t group;         // G
  int32_t window;
  int32_t rows;          // G * window
  int32_t rows_pad;      // waves * row_blocks * 32
  int32_t blocks;        // ceil(rows / 32) real 32-row blocks
  int32_t waves;         // 1 .. 8
  int32_t row_blocks;    // 32-row MFMA blocks per wave (1 or 2)
  int32_t balanced;      // 1: 14 blocks on 8 waves, 7 units per SIMD (score_window.hip)
  int32_t chunk;         // keys per work-group (multiple of 64)
  int32_t total_chunks;  // sum over sequences of ceil(L_s / chunk)
};

// Historical rows per work-group of the rho contraction.
constexpr int kRhoRows = 256;

// One kRhoRows-row block of historical tokens: sequence, block index within the
// sequence, the sequence's historical token count, and where its historical
// tokens start in the flattened hist_tok table.
struct HistBlock {
  int32_t seq, hb, n_hist, hist_base;
};

// Similarity of the frame-similarity maximum (values of stlite_similarity).
enum Sim : int32_t { kSimCosine = 0, kSimDot = 1, kSimNegL2 = 2 };

struct RhoArgs {
  Layout lay;
  int32_t sim;           // Sim
  const uint16_t* k;
  float* rn_cur;         // workspace [units][L], per current-frame key: 1/||k|| (cosine, dot) or -||k||^2 (-L2)
  float* rho;            // [units][L]; written on historical tokens
  int32_t* hist_tok;     // workspace [sum N_hist]: absolute token of every historical row
  HistBlock* blocks;     // workspace [total_hist_blocks]
  int32_t total_hist_blocks;  // sum over sequences of ceil(N_hist_s / kRhoRows)
  int32_t max_cur;       // largest current frame (tokens)
};

// Frames of one sequence that the selection kernels keep in LDS.
constexpr int kSelFrames = 1024;

// How a call's selections run.
enum SelPath : int32_t {
  kSelPathResident = 0,  // one work-group per segment, keys in registers (segsel_resident.h); no workspace
  kSelPathSplit = 1,     // splitters from a sample, then one classifying pass (segsel_split.h)
  kSelPathFourPass = 2,  // four radix passes over stored keys (segsel.h)
};

// Workspace and launch shape of one exact k-selection over (unit, sequence)
// segments.
struct SelPlan {
  // four passes (segsel.h), each segment cut into `parts` parts
  uint32_t* keys;        // [units][sel_key_stride]: one key per token
  uint32_t* hist0;       // [units][seqs][parts][2048 + 64]: level-0 part histograms (bins, 32-bin sums)
  uint32_t* hist1;       // [units][seqs][parts][2048 + 64]: level 1
  uint32_t* hist2;       // [units][seqs][parts][1024 + 32]: level 2
  int32_t* below;        // [units][seqs][parts]: keys below the level-1 prefix
  int32_t* state;        // [units][seqs][8]: k, then prefix and rank after levels 0 and 1
  int32_t parts;         // 1 .. 16
  // splitters (segsel_split.h); the same workspace bytes as the four passes' arrays
  uint8_t* codes;        // [units][256 * sp_tile_stride]: each token's class against the splitters, per tile
  int32_t* tiles;        // [units][sp_tile_stride][8]: per 256-token tile counts and output offset
  uint2* cands;          // [units][sp_cand_stride]: (key, token) of the tokens between the splitters
  int32_t* sstate;       // [units][seqs][kSpWords]: splitters, counts, mode, T, tie cut
  int32_t split_parts;   // work-groups per segment of the classify and emit passes (launch_split refines it)
  int32_t split_tiles;   // 256-token tiles of the longest segment
  int32_t split_exact;   // 1: resolve every segment by the exact streaming selection (diagnostic)
  int32_t lds_frames;    // 1: no sequence has more than kSelFrames frames
  int32_t path;          // SelPath
};

// Splitter selection layout: per unit, one tile record per 256 tokens of each
// sequence (sequence seq's first record at sp_tile_base) and a candidate list
// per sequence sized 40/256 (~15.6 %) of its tokens + 256 (from
// sp_cand_base(s0, seq) to sp_cand_base(s0 + n, seq + 1)).  Both bases are
// monotone in (s0, seq), and a sequence's range ends at or before the next
// sequence's base.
constexpr int kSpWords = 16;
__host__ __device__ inline int64_t sp_tile_stride(int64_t total_tokens, int32_t n_seqs) {
  return total_tokens / 256 + int64_t(n_seqs) + 1;
}
__host__ __device__ inline int64_t sp_tile_base(int64_t s0, int32_t seq) { return s0 / 256 + int64_t(seq); }
__host__ __device__ inline int64_t sp_cand_base(int64_t s0, int32_t seq) { return (s0 * 40) / 256 + 256 * int64_t(seq); }
__host__ __device__ inline int64_t sp_cand_stride(int64_t total_tokens, int32_t n_seqs) {
  return sp_cand_base(total_tokens, n_seqs) + 256;
}

// Longest sequence whose selections run segment-resident (one work-group per
// segment, keys kept in registers).
constexpr int32_t kSelResidentCapacity = 32768;

// Key rows of a selection: a row of sel_key_stride keys per unit; the keys of
// sequence seq (first token s0) start at sel_key_base, a multiple of 4, and the
// 16-byte group holding a sequence's last key stays inside the row and clear of
// the next sequence.
__host__ __device__ inline int64_t sel_key_stride(int64_t total_tokens, int32_t n_seqs) {
  return ((total_tokens + 3) / 4) * 4 + 4 * int64_t(n_seqs);
}
__host__ __device__ inline int64_t sel_key_base(int32_t s0, int32_t seq) { return int64_t(s0 / 4) * 4 + 4 * int64_t(seq); }

struct GateArgs {
  Layout lay;
  const float* rho;      // [units][L] (historical entries read)
  float* rho_zero_fill;  // nullable: its entries of non-historical tokens are zeroed (the rho pass writes the rest)
  uint8_t* gate;         // nullable for the rho-only call; [units][L]
  int32_t* hist_tok;     // workspace [sum N_hist]: absolute token of every historical row
  HistBlock* blocks;     // workspace [total_hist_blocks]
  SelPlan sel;           // workspace of the rank gate's selection
  float* tau;            // nullable [units][seqs]: rho of the last admitted token, NaN when none is
};

struct CssArgs {
  Layout lay;
  const uint16_t* k;
  const uint8_t* gate;   // nullable (3 x 3 only): Phi = 0 where gate == 0
  float* phi;
  int32_t strips;        // largest number of 14-column strips in a frame (3 x 3), or of 4 x 16 tiles (k x k)
};

struct OverlapArgs {
  Layout lay;
  const int32_t* kept_a;  // [units][total_budget], ascending per sequence
  const int32_t* kept_b;
  int32_t* hits;          // [units][n_seqs]
  int32_t spans_per_seq;  // 65,536-token spans of the longest sequence
};

struct SelectArgs {
  Layout lay;
  const float* a_base;
  const float* phi;      // nullable
  const uint8_t* gate;   // nullable
  float alpha;
  int32_t* kept;         // [units][total_budget]
  float* score;          // nullable [units][L]
  SelPlan sel;           // workspace of the top-B selection
};

struct CompactArgs {
  Layout lay;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* kept;   // [units][total_budget], or [n_layers][total_budget] with kept_per_layer
  int32_t kept_per_layer;
  uint16_t* k_out;
  uint16_t* v_out;
};

struct DecodeArgs {
  Layout lay;
  const uint16_t* q;       // [layers][seqs][Hq][d]: one decode query per head
  const uint16_t* k;       // [units][total_rows][d]
  const uint16_t* v;
  const int32_t* cu_rows;  // [n_seqs + 1]: the sequences' rows in this cache
  int64_t total_rows;
  float* out;              // [layers][seqs][Hq][d]
  float* pm;               // workspace [units][total_chunks][16]: chunk max (log2 units)
  float* pl;               // workspace [units][total_chunks][16]: chunk sum
  float* po;               // workspace [units][total_chunks][16][d]: chunk O, unnormalised
  int32_t n_q_heads;
  int32_t group;           // G <= 16
  int32_t chunk;           // rows per work-group
  int32_t total_chunks;
};

hipError_t launch_score_window(const ScoreArgs& a, hipStream_t stream);
hipError_t launch_decode(const DecodeArgs& a, hipStream_t stream);
hipError_t launch_tsg_gate(const RhoArgs& r, const GateArgs& g, hipStream_t stream);
hipError_t launch_tsg_threshold(const GateArgs& g, hipStream_t stream);
hipError_t launch_tsg_rho(const RhoArgs& r, const GateArgs& g, hipStream_t stream);
// gate = 1[float32(rho) <= tau] on historical tokens, 1 elsewhere (g.gate, g.rho, g.lay).
hipError_t launch_tsg_fixed_gate(const GateArgs& g, float tau, hipStream_t stream);
// Rank gate and tau_red from g.rho (the exact selection of segsel.h).
hipError_t launch_gate_select(const GateArgs& g, hipStream_t stream);
// TSG plan tables (historical-token table, rho blocks) and the
// fill of g.gate with 1 (every token) and of g.rho_zero_fill with 0 (the
// tokens that are not historical) over g.lay.n_units units.
hipError_t launch_gate_prologue(const GateArgs& g, hipStream_t stream);
// Concatenated key space (D = n_kv_heads * 128; outputs [n_layers][total_tokens]).
hipError_t launch_layer_mean(const float* a_base, float* a_layer, const Layout& lay, hipStream_t stream);
hipError_t launch_tsg_rho_concat(const RhoArgs& r, const GateArgs& g, hipStream_t stream);
hipError_t launch_css_concat(const CssArgs& a, hipStream_t stream);
// hits[u][s] = |kept_a cap kept_b| of sequence s in unit u.
hipError_t launch_kept_overlap(const OverlapArgs& a, hipStream_t stream);
hipError_t launch_css(const CssArgs& a, hipStream_t stream);
// Phi under a k x k neighbourhood, nbhd = k in {5, 7, 9}.
hipError_t launch_css_wide(const CssArgs& a, int32_t nbhd, hipStream_t stream);
hipError_t launch_select(const SelectArgs& a, hipStream_t stream);
// Mean-Attention prior: a_mean = a_base averaged over `width` (odd) positions
// along each sequence, zero outside it ([units][total_tokens] each).
constexpr int32_t kMeanMaxRadius = 127;  // width <= 255
hipError_t launch_mean_attention(const float* a_base, float* a_mean, const Layout& lay, int32_t width,
                                 hipStream_t stream);
hipError_t launch_compact(const CompactArgs& a, hipStream_t stream);

// ---------------------------------------------------------------------------
// Device helpers
// ---------------------------------------------------------------------------

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Total order of fp32 values as unsigned integers (ascending key = ascending
// value); -0 is folded onto +0 so that the two zeros tie.
__device__ __forceinline__ uint32_t order_key(float x) {
  const uint32_t u = __float_as_uint(x + 0.0f);
  // negative: all bits flipped; non-negative: the sign bit set
  return u ^ (uint32_t(int32_t(u) >> 31) | 0x80000000u);
}

__device__ __forceinline__ float order_key_value(uint32_t key) {
  uint32_t u = (key & 0x80000000u) ? (key & 0x7fffffffu) : ~key;
  return __uint_as_float(u);
}

}  // namespace stlite
