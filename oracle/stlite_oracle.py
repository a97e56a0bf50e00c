"""fp64 CPU oracle of the ST-Lite prefill-time KV-cache compression pass.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and the
benchmark's CPU-baseline leg may import or call this module; the compression
library never does, and this module imports nothing from it.

The oracle is plain and slow on purpose: each function writes out one
definition of the paper in float64 (NumPy; fp64 matmul is used as a library
primitive for dot products), in the order the paper's compression procedure
(the algorithm "ST-Lite Compression Procedure", appendix "Algorithm Details")
takes them:

  budget           B = floor(beta * L)                      (problem setup)
  base_score       A_base, window voting of softmax rows      (Eq. base_attention)
  mean_attention   the Mean-Attention base prior: 1D average
                   pooling of A_base along the sequence       (appendix on the base
                                                               scoring function; R-mean)
  css_saliency     H = mean Moore-neighbour cosine, Phi = 1-H (Eq. css_calc, Sec. CSS);
                   k x k neighbourhoods for the neighbourhood-size ablation
  tsg_rho          rho_i = max cosine to the current frame    (Sec. TSG)
  tsg_similarity   the same maximum for dot product or -L2    (similarity ablation)
  tsg_gate         tau_red = min(B,|pool|)-th smallest rho,
                   M_time = 1[rho <= tau_red]                 (Eqs. budget_threshold, temporal_mask)
  tsg_fixed_gate   M_time = 1[rho <= tau] for a fixed tau     (component-necessity control)
  integrate        S = A (text), M (A + alpha Phi) (visual)   (Eq. modal_scoring)
  select_topk      I_keep = Top_B(S)                          (Sec. integrated scoring)
  compact          K' = K[I_keep], V' = V[I_keep]             (algorithm's return value)
  decode_attention softmax(q K^T / sqrt(d)) V over a cache    (problem setup: the decoding
                   phase that consumes K', V')
  cache_hit_rate   |I_keep cap I*| / |I*|, I* = Top_B of the first decode
                   query's attention over the full cache      (Eq. chr)
  compress_layer_concat  the procedure over the layer's concatenated
                   key space, one kept set per layer          (problem setup; R3b)
  recompress_steps the procedure at every step t of one trajectory, on step
                   t's own context (frames 0..t and their text), with the
                   per-step cache hit rates                   (Eq. history_context, Eq. chr)
  trajectory_cache_hit_rate  (1/T) sum_t of the per-step rates      (Eq. chr)

Readings where the paper is silent (each is also listed in the design notes):

  R1  causal window: window query at position p only sees keys 0..p;
  R2  GQA: A_base of a kv head is the mean over its G query heads of the
      single-head window sum;
  R3  CSS and TSG use the key vectors of each kv head separately (d = 128);
  R5  grid borders: only in-grid Moore neighbours count (8/5/3); no neighbour
      (1x1 grid) gives Phi = 0;
  R6  cosine with a zero-norm vector is 0;
  R7  ties at tau_red: the gate admits exactly m = min(B, |pool|) historical
      tokens, taken in (rho ascending, index ascending) order;
  R8  rho >= 1 - 1e-4 is snapped to exactly 1 (duplicate class);
  R5b a k x k neighbourhood (k = 5, 7, 9) keeps R5's rule: its in-grid cells
      other than the centre, equally weighted;
  R-chr the attention of the first decode query that defines the oracle set
      is averaged over the kv head's query heads (as R2 does for A_base), so
      that I* and I_keep are sets of the same (layer, kv head) unit;
  R3b the concatenated-head alternative to R3: h_t is token t's keys of all
      kv heads concatenated (D = H_kv * d), A the mean over all the layer's
      query heads, and one kept set per layer serves every kv head;
  R8b under the negative-L2 similarity, a squared distance <= 1e-5 ||k_i||^2
      is snapped to 0 (the same duplicate class);
  R9  beta is a rational num/den and B = floor(L*num/den) in integers;
  R11 no forced keep of the window; R13 gated-out visual tokens score 0;
  R16 I_keep is emitted in ascending token order;
  R-mean the Mean-Attention base prior is the window-aggregated A_base of
      Eq. base_attention averaged over a centred window of `width` (odd)
      positions along the sequence's token axis, zero outside the sequence,
      divided by width (pooling with zero padding and a fixed divisor);
  R-step recompression along a trajectory: step t compresses its own full
      prefill cache (frames 0..t and the text after each, B_t = floor(beta L_t)),
      with no reuse of an earlier step's compacted cache;
  R-dec ranking decisions (gate admission, top-B) are taken on the scores
      rounded to float32, the precision the GPU kernels compute them in; ties
      go to the lowest token index.

Parity unpinned (by the paper): readings R1, R2, R3, R8 and R11 are choices the
paper does not arbitrate -- it prints no numeric A_base, Phi, rho or S for any
input -- so the tests pin the oracle under these readings (closed forms,
invariants, the literal twin), not against printed values.

Arrays: keys/values/queries arrive as bf16 bit patterns (uint16) exactly as
stored; ``bf16_to_f64`` widens them exactly.  Token indices inside one
sequence are local (0..L-1); ``compress_sequence`` adds the sequence offset.
"""
from __future__ import annotations

import math
from typing import Dict, List, Sequence, Tuple

import numpy as np

SNAP_EPS = 1e-4          # reading R8
L2_SNAP = 1e-5           # reading R8b
DECIDE_DTYPE = np.float32  # reading R-dec


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns (uint16) to float64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


# ---------------------------------------------------------------------------
# Budget (problem setup: B = floor(beta * L); Alg. initialisation)
# ---------------------------------------------------------------------------

def budget(L: int, beta_num: int, beta_den: int) -> int:
    """B = floor(beta * L) with beta = beta_num / beta_den, in exact integers."""
    if L < 0 or beta_num <= 0 or beta_den <= 0 or beta_num > beta_den:
        raise ValueError("need L >= 0 and 0 < beta <= 1")
    return (int(L) * int(beta_num)) // int(beta_den)


# ---------------------------------------------------------------------------
# Window base score (Eq. base_attention)
# ---------------------------------------------------------------------------

def base_score(Q: np.ndarray, K: np.ndarray, row_chunk: int = 64) -> np.ndarray:
    """A_base for one kv head of one sequence.

    Q: [G, delta, d] float64 -- the group's window queries; window position w
       sits at token p = L - delta + w.
    K: [L, d] float64.
    Returns A [L]: (1/G) * sum_g sum_w softmax_{i <= p}(q_{g,w} . k_i / sqrt(d)).
    """
    G, delta, d = Q.shape
    L = K.shape[0]
    if delta > L:
        raise ValueError("window longer than the sequence")
    rows = Q.reshape(G * delta, d)
    pos = np.tile(np.arange(L - delta, L), G)           # token position of every row
    A = np.zeros(L, dtype=np.float64)
    scale = 1.0 / math.sqrt(d)
    keys = np.arange(L)
    for r0 in range(0, rows.shape[0], row_chunk):
        z = (rows[r0:r0 + row_chunk] @ K.T) * scale      # [r, L] logits
        visible = keys[None, :] <= pos[r0:r0 + row_chunk, None]   # R1 causal
        z = np.where(visible, z, -np.inf)
        zmax = z.max(axis=1, keepdims=True)
        e = np.exp(z - zmax)
        P = e / e.sum(axis=1, keepdims=True)              # softmax over visible keys
        A += P.sum(axis=0)
    return A / G                                          # R2


# ---------------------------------------------------------------------------
# Cosine helper (R6)
# ---------------------------------------------------------------------------

def mean_attention(A: np.ndarray, width: int) -> np.ndarray:
    """Mean-Attention base prior (appendix on the base scoring function,
    reading R-mean): A_mean_i = (1/width) sum_{j=i-r}^{i+r} A_j with r = (width-1)/2
    and A_j = 0 for j outside the sequence (0..L-1).  width odd, >= 1."""
    if width < 1 or width % 2 == 0:
        raise ValueError("width must be odd and >= 1")
    A = np.asarray(A, dtype=np.float64)
    L = len(A)
    r = (width - 1) // 2
    out = np.zeros(L)
    for i in range(L):
        out[i] = A[max(i - r, 0):min(i + r, L - 1) + 1].sum() / width
    return out


def _cos_matrix(X: np.ndarray, Y: np.ndarray) -> np.ndarray:
    nx = np.sqrt((X * X).sum(axis=1))
    ny = np.sqrt((Y * Y).sum(axis=1))
    dots = X @ Y.T
    den = nx[:, None] * ny[None, :]
    return np.where(den > 0, dots / np.where(den > 0, den, 1.0), 0.0)


def _cos_rows(X: np.ndarray, Y: np.ndarray) -> np.ndarray:
    """Row-wise cosine of equally shaped [n, d] arrays."""
    nx = np.sqrt((X * X).sum(axis=1))
    ny = np.sqrt((Y * Y).sum(axis=1))
    den = nx * ny
    dots = (X * Y).sum(axis=1)
    return np.where(den > 0, dots / np.where(den > 0, den, 1.0), 0.0)


# ---------------------------------------------------------------------------
# Component-centric Spatial Saliency (Eq. css_calc and Phi_space = 1 - H)
# ---------------------------------------------------------------------------

MOORE = [(-1, -1), (-1, 0), (-1, 1), (0, -1), (0, 1), (1, -1), (1, 0), (1, 1)]
CSS_SIZES = (3, 5, 7, 9)   # the neighbourhood sizes of the CSS neighbourhood-size ablation


def neighbourhood(k: int):
    """Offsets (du, dv) of a k x k neighbourhood without its centre; k = 3 is the
    Moore neighbourhood of Eq. css_calc, k = 5, 7, 9 the ablation's wider ones
    (reading R5b: the same in-grid rule at every size)."""
    if k not in CSS_SIZES:
        raise ValueError(f"neighbourhood size {k} not in {CSS_SIZES}")
    r = k // 2
    return [(du, dv) for du in range(-r, r + 1) for dv in range(-r, r + 1) if (du, dv) != (0, 0)]


def css_frame(X: np.ndarray, rows: int, cols: int, k: int = 3) -> np.ndarray:
    """Phi for one frame.  X: [rows*cols, d] keys in row-major grid order."""
    d = X.shape[1]
    grid = X.reshape(rows, cols, d)
    acc = np.zeros((rows, cols))
    cnt = np.zeros((rows, cols))
    for du, dv in neighbourhood(k):
        # centre cells whose neighbour (u+du, v+dv) is inside the grid (R5)
        u0, u1 = max(0, -du), min(rows, rows - du)
        v0, v1 = max(0, -dv), min(cols, cols - dv)
        if u1 <= u0 or v1 <= v0:
            continue
        c = grid[u0:u1, v0:v1].reshape(-1, d)
        n = grid[u0 + du:u1 + du, v0 + dv:v1 + dv].reshape(-1, d)
        acc[u0:u1, v0:v1] += _cos_rows(c, n).reshape(u1 - u0, v1 - v0)
        cnt[u0:u1, v0:v1] += 1
    H = np.where(cnt > 0, acc / np.where(cnt > 0, cnt, 1), 1.0)   # no neighbour -> Phi = 0
    return (1.0 - H).reshape(-1)


def css_saliency(K: np.ndarray, frames: Sequence[Tuple[int, int, int]], k: int = 3) -> np.ndarray:
    """Phi_space over one sequence (0 on text tokens).  frames: local (offset, rows, cols);
    k: neighbourhood size (3 = Eq. css_calc; 5, 7, 9 = the neighbourhood-size ablation)."""
    phi = np.zeros(K.shape[0])
    for off, r, c in frames:
        phi[off:off + r * c] = css_frame(K[off:off + r * c], r, c, k)
    return phi


# ---------------------------------------------------------------------------
# Trajectory-aware Semantic Gating (Sec. TSG; Eqs. budget_threshold, temporal_mask)
# ---------------------------------------------------------------------------

def split_tokens(L: int, frames: Sequence[Tuple[int, int, int]]):
    """(historical visual, current-frame visual, text) local token indices."""
    hist: List[np.ndarray] = []
    cur = np.zeros(0, dtype=np.int64)
    visual = np.zeros(L, dtype=bool)
    for f, (off, r, c) in enumerate(frames):
        idx = np.arange(off, off + r * c)
        visual[idx] = True
        if f == len(frames) - 1:
            cur = idx
        else:
            hist.append(idx)
    h = np.concatenate(hist) if hist else np.zeros(0, dtype=np.int64)
    return h, cur, np.flatnonzero(~visual)


def tsg_rho(K: np.ndarray, hist: np.ndarray, cur: np.ndarray, chunk: int = 4096) -> np.ndarray:
    """rho_i = max over current-frame j of cos(k_i, k_j), clamped to [-1, 1], snapped (R8)."""
    rho = np.zeros(len(hist))
    if len(hist) == 0:
        return rho
    if len(cur) == 0:
        raise ValueError("historical tokens need a current frame")
    Kc = K[cur]
    for a in range(0, len(hist), chunk):
        rho[a:a + chunk] = _cos_matrix(K[hist[a:a + chunk]], Kc).max(axis=1)
    rho = np.clip(rho, -1.0, 1.0)
    return np.where(rho >= 1.0 - SNAP_EPS, 1.0, rho)


def tsg_similarity(K: np.ndarray, hist: np.ndarray, cur: np.ndarray, sim: str = "cosine",
                   chunk: int = 4096) -> np.ndarray:
    """rho_i = max over current-frame j of sim(k_i, k_j), for the similarity
    functions of the paper's similarity-metric ablation (appendix Similarity
    Metric Ablation; Sec. TSG for the cosine):

      cosine   cos(k_i, k_j) with the clamp and snap of tsg_rho (R8);
      dot      k_i . k_j;
      neg_l2   -||k_i - k_j||, the squared distance snapped to 0 when it is
               at most L2_SNAP ||k_i||^2 (reading R8b: the duplicate class of
               the distance, as R8 is for the cosine).
    """
    if sim == "cosine":
        return tsg_rho(K, hist, cur, chunk)
    rho = np.zeros(len(hist))
    if len(hist) == 0:
        return rho
    if len(cur) == 0:
        raise ValueError("historical tokens need a current frame")
    Kc = K[cur]
    for a in range(0, len(hist), chunk):
        Kh = K[hist[a:a + chunk]]
        if sim == "dot":
            rho[a:a + chunk] = (Kh @ Kc.T).max(axis=1)
        elif sim == "neg_l2":
            # ||a - b||^2 = ||a||^2 + ||b||^2 - 2 a.b in float64 (cancellation ~1e-16 of
            # the norms, far below the snap); the literal twin sums (a - b)^2 directly.
            n2 = (Kh * Kh).sum(axis=1)
            d2 = n2[:, None] + (Kc * Kc).sum(axis=1)[None, :] - 2.0 * (Kh @ Kc.T)
            d2 = np.maximum(d2.min(axis=1), 0.0)
            d2 = np.where(d2 <= L2_SNAP * n2, 0.0, d2)
            rho[a:a + chunk] = -np.sqrt(d2)
        else:
            raise ValueError(f"unknown similarity {sim!r}")
    return rho


def tsg_fixed_gate(rho: np.ndarray, hist: np.ndarray, L: int, tau: float) -> np.ndarray:
    """The fixed-threshold control of the paper's Component Necessity Controls:
    a historical token is gated out when its rho exceeds tau, whatever the
    distribution (decided on float32 rho, R-dec); text and the current frame
    get 1."""
    gate = np.ones(L, dtype=np.uint8)
    gate[hist] = (rho.astype(DECIDE_DTYPE) <= DECIDE_DTYPE(tau)).astype(np.uint8)
    return gate


def tsg_gate(rho: np.ndarray, hist: np.ndarray, L: int, B: int):
    """M_time over all L tokens (1 for text and the current frame) and tau_red.

    m = min(B, |pool|) historical tokens are admitted, those first in
    (rho ascending, index ascending) order, decided on float32 rho (R7, R-dec).
    tau_red is the rho of the m-th admitted token (NaN when m = 0).
    """
    gate = np.ones(L, dtype=np.uint8)
    m = min(B, len(hist))
    if len(hist) == 0:
        return gate, float("nan")
    r32 = rho.astype(DECIDE_DTYPE)
    order = np.lexsort((hist, r32))          # primary rho asc, secondary index asc
    gate[hist] = 0
    gate[hist[order[:m]]] = 1
    tau = float(r32[order[m - 1]]) if m > 0 else float("nan")
    return gate, tau


# ---------------------------------------------------------------------------
# Integrated score and flat top-B (Eq. modal_scoring; Sec. integrated scoring)
# ---------------------------------------------------------------------------

def integrate(A: np.ndarray, phi: np.ndarray, gate: np.ndarray, visual: np.ndarray,
              alpha: float) -> np.ndarray:
    """S = A on text; S = M (A + alpha Phi) on visual tokens."""
    return np.where(visual, gate * (A + alpha * phi), A)


def select_topk(S: np.ndarray, B: int) -> np.ndarray:
    """The B tokens first in (S descending, index ascending) order, emitted ascending.

    The ranking is decided on float32 S (R-dec)."""
    s32 = S.astype(DECIDE_DTYPE)
    order = np.lexsort((np.arange(len(S)), -s32.astype(np.float64)))
    return np.sort(order[:B])


def compact(K_bits: np.ndarray, V_bits: np.ndarray, kept: np.ndarray):
    """K' = K[I_keep], V' = V[I_keep]: exact copies of the stored rows."""
    return K_bits[kept].copy(), V_bits[kept].copy()


# ---------------------------------------------------------------------------
# One (sequence, layer, kv head) unit, and whole packed batches
# ---------------------------------------------------------------------------

def compress_unit(Q_bits: np.ndarray, K_bits: np.ndarray, V_bits: np.ndarray,
                  frames: Sequence[Tuple[int, int, int]], beta: Tuple[int, int],
                  alpha: float = 1.0, use_css: bool = True, use_tsg: bool = True,
                  mean_width: int = 0) -> Dict:
    """Run the whole procedure for one unit; local indices.

    Q_bits [G, delta, d], K_bits/V_bits [L, d] (bf16 bits); frames local.
    use_css=False drops the Phi term (alpha = 0); use_tsg=False sets M = 1.
    mean_width > 0 scores with the Mean-Attention prior of that pooling width
    (returned as A_mean) in place of A_base (returned as A).
    """
    K = bf16_to_f64(K_bits)
    Q = bf16_to_f64(Q_bits)
    L = K.shape[0]
    B = budget(L, *beta)
    A = base_score(Q, K)
    prior = mean_attention(A, mean_width) if mean_width else A
    hist, cur, text = split_tokens(L, frames)
    visual = np.zeros(L, dtype=bool)
    visual[hist] = True
    visual[cur] = True
    phi = css_saliency(K, frames) if use_css else np.zeros(L)
    rho = tsg_rho(K, hist, cur)
    if use_tsg:
        gate, tau = tsg_gate(rho, hist, L, B)
    else:
        gate, tau = np.ones(L, dtype=np.uint8), float("nan")
    S = integrate(prior, phi, gate, visual, alpha if use_css else 0.0)
    kept = select_topk(S, B)
    k_out, v_out = compact(K_bits, V_bits, kept)
    out = dict(B=B, A=A, phi=phi, hist=hist, cur=cur, rho=rho, gate=gate, tau=tau,
               S=S, kept=kept, k_out=k_out, v_out=v_out, visual=visual)
    if mean_width:
        out["A_mean"] = prior
    return out


# ---------------------------------------------------------------------------
# Decode attention over a cache (problem setup: after prefill, the decoding
# phase attends each new query over the cached keys and values; the
# compression procedure hands K', V' to that phase)
# ---------------------------------------------------------------------------

def decode_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray) -> np.ndarray:
    """out_g = sum_j softmax_j(q_g . k_j / sqrt(d)) v_j for every query row g.

    Q [G, d], K and V [n, d] as float64; the decode query follows every cached
    row, so no row is masked.  A cache with no rows gives zeros."""
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    V = np.asarray(V, dtype=np.float64)
    if K.shape[0] == 0:
        return np.zeros((Q.shape[0], V.shape[1]))
    z = (Q @ K.T) / math.sqrt(K.shape[1])
    z = z - z.max(axis=1, keepdims=True)
    p = np.exp(z)
    p = p / p.sum(axis=1, keepdims=True)
    return p @ V


# ---------------------------------------------------------------------------
# Cache hit rate (Sec. cache hit rate evaluation, Eq. chr)
# ---------------------------------------------------------------------------

def decode_attention_scores(Q: np.ndarray, K: np.ndarray) -> np.ndarray:
    """a_i = (1/G) sum_g softmax_j(q_g . k_j / sqrt(d))_i over all L cached positions:
    the attention distribution of the first decode query over the full cache,
    averaged over the kv head's G query heads (reading R-chr, as R2 for A_base).
    Q [G, d], K [L, d] float64."""
    Q = np.asarray(Q, dtype=np.float64)
    K = np.asarray(K, dtype=np.float64)
    z = (Q @ K.T) / math.sqrt(K.shape[1])
    z = z - z.max(axis=1, keepdims=True)
    p = np.exp(z)
    p = p / p.sum(axis=1, keepdims=True)
    return p.mean(axis=0)


def chr_oracle_set(a_dec: np.ndarray, B: int) -> np.ndarray:
    """I* = Top_B of the decode attention (same order and tie-break as select_topk)."""
    return select_topk(a_dec, B)


def cache_hit_rate(kept: np.ndarray, oracle: np.ndarray) -> float:
    """|I_keep cap I*| / |I*| for one step and unit (Eq. chr before the average
    over steps); NaN when I* is empty (B = 0)."""
    if len(oracle) == 0:
        return float("nan")
    return len(np.intersect1d(kept, oracle)) / len(oracle)


def trajectory_cache_hit_rate(rates: Sequence[float]) -> float:
    """Eq. chr: the mean over the T evaluation steps of the per-step hit rates
    |I_keep^(t) cap I*^(t)| / |I*^(t)|.  Steps whose oracle set is empty (B_t = 0,
    rate NaN) are not evaluation steps and are left out; NaN if none is left."""
    r = [float(x) for x in rates if not math.isnan(float(x))]
    if not r:
        return float("nan")
    return sum(r) / len(r)


def recompress_steps(q_steps, q_dec_steps, k_bits, v_bits, frames: Sequence[Tuple[int, int, int]],
                     frame_ends: Sequence[int], steps: Sequence[int], beta, alpha=1.0) -> Dict:
    """The procedure at each listed step of one trajectory, for one unit (reading R-step).

    The trajectory's context at step t (Eq. history_context) is every token
    before frame t + 1: frames 0..t with the text after each, L_t = frame_ends[t]
    tokens, and its cache is the first L_t rows of the trajectory's keys and
    values.  Frame t is that step's current frame.  Each step is compressed on
    its own (compress_unit) at budget B_t = floor(beta * L_t); its oracle set
    I*^(t) is the top-B_t of its decode query's attention over those L_t rows.

    q_steps [T, G, delta, d] and q_dec_steps [T, G, d] (bf16 bits) are the
    window queries and decode queries of the listed steps; k_bits, v_bits
    [L, d] are the whole trajectory's rows; frames are (offset, rows, cols)
    local to it.  Returns the per-step outputs and cache hit rates and their
    Eq. chr mean.
    """
    outs, rates = [], []
    for i, t in enumerate(steps):
        L_t = int(frame_ends[t])
        out = compress_unit(q_steps[i], k_bits[:L_t], v_bits[:L_t], list(frames[:t + 1]), beta, alpha)
        a_dec = decode_attention_scores(bf16_to_f64(q_dec_steps[i]), bf16_to_f64(k_bits[:L_t]))
        star = chr_oracle_set(a_dec, out["B"])
        out["a_dec"] = a_dec
        out["star"] = star
        out["chr"] = cache_hit_rate(out["kept"], star)
        outs.append(out)
        rates.append(out["chr"])
    return dict(steps=outs, rates=rates, chr=trajectory_cache_hit_rate(rates))


def seq_frames_local(cu_seqlens, cu_frames, frame_meta, s: int):
    """Frames of sequence s with offsets made local to the sequence."""
    base = int(cu_seqlens[s])
    return [(int(o) - base, int(r), int(c))
            for o, r, c in frame_meta[cu_frames[s]:cu_frames[s + 1]]]


def compress_sequence(q_bits, k_bits, v_bits, cu_seqlens, cu_frames, frame_meta, s: int,
                      layer: int, kv: int, group: int, beta, alpha=1.0,
                      use_css=True, use_tsg=True, mean_width=0) -> Dict:
    """One unit of a packed batch.

    q_bits [layers, seqs, Hq, delta, d]; k_bits, v_bits [layers, Hkv, L_total, d].
    Kept indices are returned both local and absolute.
    """
    a, b = int(cu_seqlens[s]), int(cu_seqlens[s + 1])
    frames = seq_frames_local(cu_seqlens, cu_frames, frame_meta, s)
    Qg = q_bits[layer, s, kv * group:(kv + 1) * group]
    out = compress_unit(Qg, k_bits[layer, kv, a:b], v_bits[layer, kv, a:b], frames, beta,
                        alpha, use_css, use_tsg, mean_width)
    out["kept_abs"] = out["kept"] + a
    out["offset"] = a
    return out


# ---------------------------------------------------------------------------
# Concatenated-head key space (reading R3b): one kept set per layer
# ---------------------------------------------------------------------------

def compress_layer_concat(q_bits: np.ndarray, k_bits: np.ndarray, v_bits: np.ndarray,
                          frames: Sequence[Tuple[int, int, int]], beta: Tuple[int, int],
                          alpha: float = 1.0) -> Dict:
    """The procedure with the layer's key space D = H_kv * d (problem setup:
    K^(l) in R^{L x D} per layer) instead of one kv head's d; local indices.

    q_bits [H_q, delta, d], k_bits / v_bits [H_kv, L, d] (bf16 bits) of one layer
    and sequence.  h_t is the concatenation of token t's keys over the kv heads
    (CSS and TSG cosines over D), A is the mean over all H_q query heads of the
    single-head window sum (R2 over the whole layer), and the one kept set is
    applied to every kv head's K and V.
    """
    H_kv, L, d = k_bits.shape
    G = q_bits.shape[0] // H_kv
    Q = bf16_to_f64(q_bits)
    Kh = bf16_to_f64(k_bits)
    K = np.concatenate([Kh[h] for h in range(H_kv)], axis=1)      # [L, H_kv * d]
    B = budget(L, *beta)
    A = np.mean([base_score(Q[h * G:(h + 1) * G], Kh[h]) for h in range(H_kv)], axis=0)
    hist, cur, text = split_tokens(L, frames)
    visual = np.zeros(L, dtype=bool)
    visual[hist] = True
    visual[cur] = True
    phi = css_saliency(K, frames)
    rho = tsg_rho(K, hist, cur)
    gate, tau = tsg_gate(rho, hist, L, B)
    S = integrate(A, phi, gate, visual, alpha)
    kept = select_topk(S, B)
    return dict(B=B, A=A, phi=phi, hist=hist, cur=cur, rho=rho, gate=gate, tau=tau, S=S, kept=kept,
                k_out=k_bits[:, kept].copy(), v_out=v_bits[:, kept].copy(), visual=visual)

