/*
 * stlite.h -- C ABI of the MI355X (gfx950) ST-Lite KV-cache compression pass.
 *
 * ST-Lite compresses the prefill KV cache of a GUI-agent trajectory, per layer
 * and kv head, to a flat budget B = floor(beta * L) tokens (problem setup and
 * the algorithm "ST-Lite Compression Procedure" of the paper).  The pass is
 * five asynchronous calls, each one batched over all layers, kv heads and
 * packed sequences:
 *
 *   stlite_score_window  A_base, window voting of softmax rows  (Eq. base_attention)
 *   stlite_tsg_gate      rho, tau_red and the hard gate M_time    (Sec. TSG; Eqs.
 *                        budget_threshold, temporal_mask)
 *   stlite_css_saliency  Phi_space = 1 - mean Moore cosine        (Eq. css_calc)
 *   stlite_select_topk   S and the retained set I_keep = Top_B(S) (Eq. modal_scoring)
 *   stlite_compact_kv    K' = K[I_keep], V' = V[I_keep]           (the algorithm's result)
 *
 * and, for the decoding phase that consumes the cache,
 *
 *   stlite_decode_attention  softmax(q K^T / sqrt(d)) V over the full or the
 *                            compacted cache                  (problem setup)
 *
 * the variants of the paper's ablations,
 *
 *   stlite_mean_attention    the Mean-Attention base prior: A_base pooled along
 *                            the sequence (base scoring function ablation)
 *   stlite_tsg_similarity    rho under the dot product or -L2 (similarity ablation)
 *   stlite_tsg_fixed_gate    gate = 1[rho <= tau] for a fixed tau (necessity controls)
 *   stlite_css_saliency_nbhd CSS over 5x5, 7x7, 9x9 windows (neighbourhood ablation)
 *   stlite_layer_mean, stlite_tsg_rho_concat, stlite_css_saliency_concat,
 *   stlite_compact_kv_layer  the concatenated (per-layer) key space
 *
 * and, for the cache hit rate evaluation,
 *
 *   stlite_kept_overlap      |I_keep cap I*| per unit and sequence (Eq. chr)
 *
 * Conventions shared by every call
 * --------------------------------
 * Pointers are DEVICE pointers unless their name starts with h_ (host).  bf16
 * tensors are passed as their 16-bit patterns (uint16_t).  `stream` is a
 * hipStream_t passed as void* (NULL = the default stream); every call only
 * enqueues work on it and never synchronises the host.
 *
 * Units and layouts (innermost dimension contiguous, head_dim d = 128):
 *   unit u = layer * n_kv_heads + kv_head; query head g belongs to kv head g / G,
 *   G = n_q_heads / n_kv_heads.
 *   q_win    bf16  [n_layers][n_seqs][n_q_heads][window][d]  queries of the last
 *                  `window` tokens of every sequence (window position w is token
 *                  L_s - window + w of sequence s)
 *   k, v     bf16  [n_layers][n_kv_heads][total_tokens][d]
 *   a_base, phi, rho, score   fp32  [n_layers][n_kv_heads][total_tokens]
 *   gate     uint8 [n_layers][n_kv_heads][total_tokens]   1 = eligible
 *   tau      fp32  [n_layers][n_kv_heads][n_seqs]
 *   kept     int32 [n_layers][n_kv_heads][total_budget]   absolute token indices;
 *                  sequence s owns entries cu_budget[s] .. cu_budget[s+1]-1, in
 *                  ascending token order
 *   k_out, v_out bf16 [n_layers][n_kv_heads][total_budget][d]
 *
 * Sequences are packed back to back (cu_seqlens).  Each sequence lists its
 * frames (screenshots) in temporal order; a frame is a row-major rows x cols
 * patch grid of consecutive visual tokens.  The LAST frame of a sequence is its
 * current frame; the visual tokens of its other frames are historical; every
 * token in no frame is text.
 *
 * Ownership and errors: the caller allocates every buffer, including the
 * workspace sized by stlite_workspace_size; the library allocates nothing and
 * keeps no state between calls (calls are re-entrant; calls that share a
 * workspace must be ordered on one stream).  Inputs are never written; outputs
 * must not alias inputs; every element of every output is written.  Host-side
 * arguments (the h_ mirrors, sizes, pointers) are validated before anything is
 * enqueued: a failing call returns STLITE_ERR_INVALID_ARG / _UNSUPPORTED /
 * _WORKSPACE with nothing enqueued and a message for stlite_last_error().  A
 * failed kernel launch returns STLITE_ERR_HIP.  The device metadata arrays must
 * hold the same values as their host mirrors; kernels read them without
 * re-validating.
 */
#ifndef STLITE_H
#define STLITE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define STLITE_ABI_VERSION 2

typedef enum stlite_status {
  STLITE_OK = 0,
  STLITE_ERR_INVALID_ARG = 1, /* malformed argument or layout */
  STLITE_ERR_UNSUPPORTED = 2, /* well formed, but outside what the kernels implement */
  STLITE_ERR_WORKSPACE = 3,   /* workspace missing or too small */
  STLITE_ERR_HIP = 4          /* a HIP runtime call or kernel launch failed */
} stlite_status;

/* Which call a workspace size is asked for. */
typedef enum stlite_call {
  STLITE_CALL_SCORE_WINDOW = 0,
  STLITE_CALL_TSG_GATE = 1,
  STLITE_CALL_CSS_SALIENCY = 2,
  STLITE_CALL_SELECT_TOPK = 3,
  STLITE_CALL_COMPACT_KV = 4,
  STLITE_CALL_TSG_THRESHOLD = 5,
  STLITE_CALL_TSG_RHO = 6,
  STLITE_CALL_DECODE_FULL = 7,    /* stlite_decode_attention on STLITE_CACHE_FULL */
  STLITE_CALL_DECODE_COMPACT = 8, /* stlite_decode_attention on STLITE_CACHE_COMPACT */
  STLITE_CALL_TSG_RHO_CONCAT = 9  /* stlite_tsg_rho_concat */
} stlite_call;

/* Which cache a decode call reads. */
typedef enum stlite_cache {
  STLITE_CACHE_FULL = 0,    /* k, v [n_layers][n_kv_heads][total_tokens][d]: sequence s owns
                               rows cu_seqlens[s] .. cu_seqlens[s+1]-1 */
  STLITE_CACHE_COMPACT = 1  /* k_out, v_out [n_layers][n_kv_heads][total_budget][d]: sequence s
                               owns rows cu_budget[s] .. cu_budget[s+1]-1 */
} stlite_cache;

/* Similarity of the TSG frame-similarity maximum (stlite_tsg_similarity). */
typedef enum stlite_similarity {
  STLITE_SIM_COSINE = 0,  /* cos(k_i, k_j): the method's choice (Sec. TSG) */
  STLITE_SIM_DOT = 1,     /* k_i . k_j                  (similarity-metric ablation) */
  STLITE_SIM_NEG_L2 = 2   /* -||k_i - k_j||             (similarity-metric ablation) */
} stlite_similarity;

/*
 * The packed problem: model shape, window and the varlen layout.
 *
 * Limits: head_dim == 128; n_q_heads % n_kv_heads == 0; 1 <= window <= L_s for
 * every sequence; G * window <= 512 (the window queries of one kv head stay
 * resident in registers); total_tokens < 2^31; L_s <= 2^28; rows * cols <= 2^22
 * for every frame; n_seqs <= 65535;
 * n_layers * n_kv_heads <= 65535 (outside these, STLITE_ERR_UNSUPPORTED).
 * Budgets are per sequence
 * (the same for every layer and head: the paper's flat budget) and must satisfy
 * 0 <= B_s <= L_s; stlite_budget computes floor(beta * L_s).
 */
typedef struct stlite_problem {
  int32_t n_layers;
  int32_t n_q_heads;
  int32_t n_kv_heads;
  int32_t head_dim;
  int32_t n_seqs;
  int32_t n_frames;      /* frames over all sequences */
  int32_t window;        /* delta: observation window length */
  int32_t reserved;      /* must be 0 */
  int64_t total_tokens;  /* = cu_seqlens[n_seqs] */
  int64_t total_budget;  /* = cu_budget[n_seqs] */
  /* device arrays */
  const int32_t* cu_seqlens;  /* [n_seqs+1] token prefix sums, cu_seqlens[0] = 0 */
  const int32_t* cu_frames;   /* [n_seqs+1] frame prefix sums, cu_frames[0] = 0 */
  const int32_t* frame_meta;  /* [n_frames][3] = {absolute token offset, rows, cols} */
  const int32_t* cu_budget;   /* [n_seqs+1] budget prefix sums, cu_budget[0] = 0 */
  /* host mirrors of the same four arrays (validation and launch sizing) */
  const int32_t* h_cu_seqlens;
  const int32_t* h_cu_frames;
  const int32_t* h_frame_meta;
  const int32_t* h_cu_budget;
} stlite_problem;

/* ABI version of the loaded library (STLITE_ABI_VERSION it was built with). */
int32_t stlite_abi_version(void);

/* Human-readable name of a status code (static string). */
const char* stlite_status_string(stlite_status status);

/* Detail of the last error returned on the calling thread ("" if none). */
const char* stlite_last_error(void);

/*
 * Flat per-layer budget B = floor(L * beta_num / beta_den) in exact integer
 * arithmetic (problem setup; beta = beta_num / beta_den in (0, 1]).  Returns -1
 * when L < 0, beta_num <= 0, beta_den <= 0 or beta_num > beta_den.
 */
int64_t stlite_budget(int64_t L, int64_t beta_num, int64_t beta_den);

/* Checks every host-visible field of `p` (STLITE_OK or the reason it fails). */
stlite_status stlite_validate(const stlite_problem* p);

/* Bytes of device workspace `call` needs for problem `p` (0 is possible). */
stlite_status stlite_workspace_size(const stlite_problem* p, stlite_call call, size_t* bytes);

/*
 * Window base score (Eq. base_attention), per unit and sequence:
 *   A_i = (1/G) sum_{g in group} sum_{w < window} softmax_{j <= p_w}(q_{g,w} . k_j / sqrt(d))_i
 * with p_w = L_s - window + w (a window query sees the keys up to its own
 * position) and A_i = 0 for keys no window query sees.  bf16 operands, fp32
 * accumulation.  Writes a_base [units][total_tokens].
 */
stlite_status stlite_score_window(const stlite_problem* p, const uint16_t* q_win,
                                  const uint16_t* k, float* a_base, void* workspace,
                                  size_t workspace_bytes, void* stream);

/*
 * Component-centric Spatial Saliency (Eq. css_calc): for every visual token,
 * H = mean over its in-grid Moore neighbours (8, 5 or 3 of them) of the key
 * cosine, and phi = 1 - H; phi = 0 for a 1x1 frame and for text tokens.  A
 * cosine with a zero key is 0.  Writes phi [units][total_tokens].
 * gate (nullable) is the TSG gate [units][total_tokens] that stlite_tsg_gate
 * or stlite_tsg_threshold wrote: where gate == 0 the token's phi is written
 * as exactly 0 without being computed (Eq. modal_scoring multiplies it by
 * M = 0), and cosines that no admitted token needs are skipped; where
 * gate != 0, phi is bit for bit the value of the ungated call.
 */
stlite_status stlite_css_saliency(const stlite_problem* p, const uint16_t* k, const uint8_t* gate,
                                  float* phi, void* stream);

/*
 * CSS under a wider neighbourhood, for the paper's neighbourhood-size ablation
 * (appendix CSS Neighborhood Size Ablation): H = mean over the in-grid cells of
 * the nbhd x nbhd square centred on the token, other than the token itself, of
 * the key cosine; phi = 1 - H (0 when the square holds no other in-grid cell,
 * and on text).  nbhd = 3 is exactly stlite_css_saliency; 5, 7 and 9 run on the
 * matrix cores (bf16 products, fp32 sums).  Any other nbhd is
 * STLITE_ERR_INVALID_ARG.  Writes phi [units][total_tokens]; no workspace.
 */
stlite_status stlite_css_saliency_nbhd(const stlite_problem* p, int32_t nbhd, const uint16_t* k,
                                       float* phi, void* stream);

/*
 * Trajectory-aware Semantic Gating (Sec. TSG): for every historical visual
 * token i, rho_i = max over the current frame j of cos(k_i, k_j), clamped to
 * [-1, 1] and snapped to 1 when >= 1 - 1e-4.  Then, with m = min(B_s, |hist|),
 * the gate admits the m historical tokens first in (rho ascending, index
 * ascending) order -- the rank form of M_time = 1[rho <= tau_red] -- and
 * tau_red is the rho of the last admitted token (NaN if m = 0).  Text and
 * current-frame tokens get gate 1.
 * rho (nullable) receives rho on historical tokens and 0 elsewhere; tau
 * (nullable) receives tau_red per [unit][seq]; gate is required.
 */
stlite_status stlite_tsg_gate(const stlite_problem* p, const uint16_t* k, float* rho,
                              float* tau, uint8_t* gate, void* workspace,
                              size_t workspace_bytes, void* stream);

/*
 * The similarity half of stlite_tsg_gate (Sec. TSG, the frame-similarity
 * maximum): rho [units][total_tokens] receives rho on historical tokens, with
 * the same clamp and snap, and 0 elsewhere.  rho is required.  Together with
 * stlite_tsg_threshold it computes exactly what stlite_tsg_gate computes.
 */
stlite_status stlite_tsg_rho(const stlite_problem* p, const uint16_t* k, float* rho,
                             void* workspace, size_t workspace_bytes, void* stream);

/*
 * rho under another similarity, for the paper's similarity-metric ablation
 * (appendix Similarity Metric Ablation): rho_i = max over the current frame j of
 *   STLITE_SIM_COSINE  cos(k_i, k_j) with the clamp and snap above (the same
 *                      result as stlite_tsg_rho);
 *   STLITE_SIM_DOT     k_i . k_j, unclamped;
 *   STLITE_SIM_NEG_L2  -||k_i - k_j||, the squared distance snapped to 0 when it
 *                      is at most 1e-5 ||k_i||^2 (the duplicate class, as the
 *                      cosine snap is for the cosine).
 * bf16 operands, fp32 accumulation; -||k_i - k_j||^2 is formed as
 * 2 k_i.k_j - ||k_j||^2 - ||k_i||^2, so its absolute error scales with the
 * squared norms.  Writes rho [units][total_tokens] (0 off the history); needs
 * the workspace of STLITE_CALL_TSG_RHO.  An unknown `sim` is
 * STLITE_ERR_INVALID_ARG.  Feed the result to stlite_tsg_threshold for the
 * adaptive gate.
 */
stlite_status stlite_tsg_similarity(const stlite_problem* p, stlite_similarity sim,
                                    const uint16_t* k, float* rho, void* workspace,
                                    size_t workspace_bytes, void* stream);

/*
 * The fixed-threshold gate of the paper's component-necessity controls
 * (appendix Component Necessity Controls), in place of the adaptive percentile
 * threshold: gate_i = 1[float32 rho_i <= tau] on historical tokens (rho as
 * written by stlite_tsg_rho or stlite_tsg_similarity; a NaN rho gates 0),
 * gate = 1 on text and the current frame.  tau must not be NaN.  Writes gate
 * [units][total_tokens]; needs no workspace.
 */
stlite_status stlite_tsg_fixed_gate(const stlite_problem* p, const float* rho, float tau,
                                    uint8_t* gate, void* stream);

/*
 * The threshold-and-gate half of stlite_tsg_gate on a caller-supplied rho
 * [units][total_tokens] (only its historical entries are read).  Same gate and
 * tau semantics.  Lets a caller gate on another similarity signal.
 */
stlite_status stlite_tsg_threshold(const stlite_problem* p, const float* rho, float* tau,
                                   uint8_t* gate, void* workspace, size_t workspace_bytes,
                                   void* stream);

/*
 * Integrated score and flat top-B (Eq. modal_scoring; Sec. integrated scoring):
 *   S_i = A_i on text;  S_i = M_i * (A_i + alpha * phi_i) on visual tokens,
 * then the B_s tokens of each sequence first in (S descending, index
 * ascending) order are kept and written to `kept` in ascending order.
 * phi == NULL drops the CSS term; gate == NULL means M = 1 everywhere
 * (a_base alone with both NULL is SnapKV's voting with a flat budget).
 * alpha must be finite and >= 0.  score (nullable) receives S [units][total_tokens].
 */
stlite_status stlite_select_topk(const stlite_problem* p, const float* a_base,
                                 const float* phi, const uint8_t* gate, float alpha,
                                 int32_t* kept, float* score, void* workspace,
                                 size_t workspace_bytes, void* stream);

/*
 * Cache compaction: k_out[u][j] = k[u][kept[u][j]] and likewise for v, as exact
 * 256-byte row copies.  kept must hold valid token indices of the owning
 * sequence (as written by stlite_select_topk).
 */
stlite_status stlite_compact_kv(const stlite_problem* p, const uint16_t* k, const uint16_t* v,
                                const int32_t* kept, uint16_t* k_out, uint16_t* v_out,
                                void* stream);

/*
 * Decode attention over a cache: the decoding phase of the problem setup,
 * which attends each new query over the cached keys and values -- the full
 * prefill cache, or the compacted K', V' that stlite_compact_kv writes (the
 * compression procedure returns them for that phase).  For every layer,
 * sequence s and query head g (kv head g / G):
 *   out_g = sum_j softmax_j(q_g . k_j / sqrt(d)) v_j
 * over all of sequence s's rows of the chosen cache (the decode query follows
 * every cached token: no mask); a sequence with no rows gets out = 0.
 *   q_dec  bf16 [n_layers][n_seqs][n_q_heads][d]   one decode query per head
 *   k, v   bf16, the layout of `cache` (see stlite_cache)
 *   out    fp32 [n_layers][n_seqs][n_q_heads][d]
 * bf16 operands, fp32 logits, softmax and accumulation.  Needs G <= 16 and the
 * workspace of STLITE_CALL_DECODE_FULL / _COMPACT.
 */
stlite_status stlite_decode_attention(const stlite_problem* p, stlite_cache cache,
                                      const uint16_t* q_dec, const uint16_t* k,
                                      const uint16_t* v, float* out, void* workspace,
                                      size_t workspace_bytes, void* stream);

/*
 * The concatenated key space (problem setup: the cache of a layer is
 * K^(l) in R^{L x D}; here D = n_kv_heads * 128): token t's keys of every kv
 * head, one after the other, form h_t; the cosines of CSS and TSG run over D;
 * A is the mean over all of the layer's query heads; one kept set per layer
 * serves every kv head.  Outputs are per layer, [n_layers][total_tokens] (fp32)
 * or [n_layers][total_budget] (kept).  The threshold, gate and top-B steps are
 * stlite_tsg_threshold and stlite_select_topk on a layer-level problem: the same
 * layout and budgets with n_kv_heads = n_q_heads = 1.  Implemented for
 * n_kv_heads = 2 or 4 (else STLITE_ERR_UNSUPPORTED).
 */

/* a_layer[l][t] = (1/n_kv_heads) sum_h a_base[l * n_kv_heads + h][t]: the mean over
 * the layer's query heads, since each a_base row is its kv head's group mean. */
stlite_status stlite_layer_mean(const stlite_problem* p, const float* a_base, float* a_layer,
                                void* stream);

/* rho over the concatenated keys (Sec. TSG with h in R^D): rho_layer [n_layers][L]
 * gets the clamped, snapped maximum cosine on historical tokens and 0 elsewhere.
 * Needs the workspace of STLITE_CALL_TSG_RHO_CONCAT. */
stlite_status stlite_tsg_rho_concat(const stlite_problem* p, const uint16_t* k, float* rho_layer,
                                    void* workspace, size_t workspace_bytes, void* stream);

/* Phi over the concatenated keys (Eq. css_calc with h in R^D, 3 x 3 window):
 * phi_layer [n_layers][L], 0 on text.  No workspace. */
stlite_status stlite_css_saliency_concat(const stlite_problem* p, const uint16_t* k, float* phi_layer,
                                         void* stream);

/* Compaction with one kept set per layer: k_out[l * n_kv_heads + h][j] =
 * k[l * n_kv_heads + h][kept_layer[l][j]], likewise v; exact row copies. */
stlite_status stlite_compact_kv_layer(const stlite_problem* p, const uint16_t* k, const uint16_t* v,
                                      const int32_t* kept_layer, uint16_t* k_out, uint16_t* v_out,
                                      void* stream);

/*
 * The Mean-Attention base prior of the paper's base-scoring ablation (appendix
 * "Sensitivity to the Base Attention Scoring Function": one-dimensional
 * average pooling of the attention over the prompt sequence).  Reading: the
 * window-aggregated A_base that stlite_score_window writes (Eq. base_attention,
 * so the prior keeps its dependence on the observation window) is averaged
 * along each sequence's token axis over a centred window of `width` positions;
 * positions outside the sequence count as 0 and the divisor is always width:
 *
 *   a_mean[i] = (1/width) * sum_{j = i-r .. i+r, j inside i's sequence} a_base[j],
 *   r = (width - 1) / 2.
 *
 * The pooling runs over every token (text and visual alike) and never crosses
 * from one packed sequence into the next.  a_mean then takes A_base's place in
 * stlite_select_topk.
 *
 * a_base, a_mean  fp32 [n_layers][n_kv_heads][total_tokens]; a_mean must not
 *                 alias a_base; every element of a_mean is written.
 * width           odd, 1 <= width <= 255 (width 1 copies a_base).
 * Errors: STLITE_ERR_INVALID_ARG for a NULL or aliased pointer or a width
 * outside the range, nothing enqueued; STLITE_ERR_HIP for a failed launch.
 * No workspace.
 */
stlite_status stlite_mean_attention(const stlite_problem* p, const float* a_base, int32_t width,
                                    float* a_mean, void* stream);

/*
 * Cache hit rate numerator (Sec. cache hit rate evaluation, Eq. chr):
 *   hits[u][s] = |kept_a[u] cap kept_b[u]| over sequence s's entries
 * for two retained sets in the layout stlite_select_topk writes (B_s strictly
 * ascending absolute token indices of sequence s per unit).  With kept_b the
 * oracle set I* -- the top-B_s of the first decode query's attention over the
 * full cache, which stlite_score_window with window 1 and that query followed
 * by stlite_select_topk with no phi and no gate computes -- hits / B_s is the
 * CHR of kept_a for that unit and step.  hits int32 [units][n_seqs]; no
 * workspace.  Lists that break the ordering contract give a wrong count but
 * no out-of-range access.
 */
stlite_status stlite_kept_overlap(const stlite_problem* p, const int32_t* kept_a,
                                  const int32_t* kept_b, int32_t* hits, void* stream);

/*
 * stlite_select_topk without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the selection's workspace is a static
 * device array of STLITE_NOALLOC_SCRATCH_BYTES inside the library, one per
 * GPU, held from module load until the process ends.  Same arguments, results
 * and errors as stlite_select_topk; a problem whose selection needs more than
 * STLITE_NOALLOC_SCRATCH_BYTES (stlite_workspace_size with
 * STLITE_CALL_SELECT_TOPK) fails with STLITE_ERR_WORKSPACE, nothing enqueued.
 * The call allocates nothing: on the first call on a device it looks up that
 * device's copy of the array (hipGetSymbolAddress on the current device, which
 * must be the device of `stream`).  Every call on one GPU shares that GPU's
 * array: calls that may overlap on one GPU (other streams, other threads)
 * race and must be ordered by the caller.
 */
#define STLITE_NOALLOC_SCRATCH_BYTES (32u << 20)

stlite_status stlite_select_topk_noalloc(const stlite_problem* p, const float* a_base,
                                         const float* phi, const uint8_t* gate, float alpha,
                                         int32_t* kept, float* score, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* STLITE_H */
