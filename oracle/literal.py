"""Literal-loop twin of the fp64 oracle, for inputs of at most a few dozen tokens.

TEST INFRASTRUCTURE ONLY (same rule as ``stlite_oracle``: the compression library
never imports it).  Every quantity is written with explicit Python loops over
tokens, neighbours, rows and dimensions, straight from the paper's definitions,
so that a vectorisation slip in the NumPy oracle shows up as a disagreement:

  A_base^(i) = (1/G) sum_g sum_{p in window} exp(z_{g,p,i}) / sum_{j<=p} exp(z_{g,p,j}),
      z = q . k / sqrt(d)                               (Eq. base_attention; readings R1, R2)
  H_{u,v}   = (1/|N|) sum_{n in N(u,v)} cos(h_{u,v}, h_n), Phi = 1 - H   (Eq. css_calc;
              N the in-grid cells of the k x k square around (u, v), k = 3 by default)
  rho_i     = max_{j in current frame} cos(h_i, h_j)  (Sec. TSG); with k_i . k_j or
              -||k_i - k_j|| in place of the cosine (similarity-metric ablation; R8b)
  gate      = the m = min(B, |pool|) smallest rho by (rho, index)       (Eqs. budget_threshold,
                                                                        temporal_mask; R7)
  A_mean_i  = (1/w) sum_{|j - i| <= (w-1)/2, 0 <= j < L} A_j  (Mean-Attention prior; R-mean)
  S         = A (text) | M (A + alpha Phi) (visual)  (Eq. modal_scoring)
  I_keep    = first B by (S descending, index ascending), ascending  (Top_B; R16)
  out_g     = sum_j exp(z_gj) v_j / sum_j exp(z_gj), z = q_g . k_j / sqrt(d)
                                                    (decode attention over a cache)

It reuses nothing from the NumPy oracle except the bf16 widening rule, which it
restates with ``struct``.
"""
from __future__ import annotations

import math
import struct


def bf16(bits: int) -> float:
    return struct.unpack("<f", struct.pack("<I", (int(bits) & 0xFFFF) << 16))[0]


def f32(x: float) -> float:
    """Round a Python float to the nearest float32 (ranking precision, R-dec)."""
    return struct.unpack("<f", struct.pack("<f", x))[0]


def dot(a, b):
    s = 0.0
    for x, y in zip(a, b):
        s += x * y
    return s


def cos(a, b):
    na = math.sqrt(dot(a, a))
    nb = math.sqrt(dot(b, b))
    if na == 0.0 or nb == 0.0:
        return 0.0
    return dot(a, b) / (na * nb)


def base_score(Q, K):
    """Q: list[G][delta][d] floats, K: list[L][d]."""
    G = len(Q)
    delta = len(Q[0])
    L = len(K)
    d = len(K[0])
    A = [0.0] * L
    for g in range(G):
        for w in range(delta):
            p = L - delta + w
            z = [dot(Q[g][w], K[i]) / math.sqrt(d) for i in range(p + 1)]
            zm = max(z)
            den = 0.0
            for i in range(p + 1):
                den += math.exp(z[i] - zm)
            for i in range(p + 1):
                A[i] += math.exp(z[i] - zm) / den
    return [a / G for a in A]


def css(K, frames, k=3):
    L = len(K)
    phi = [0.0] * L
    r = k // 2
    for off, rows, cols in frames:
        for u in range(rows):
            for v in range(cols):
                centre = K[off + u * cols + v]
                total = 0.0
                count = 0
                for du in range(-r, r + 1):
                    for dv in range(-r, r + 1):
                        if du == 0 and dv == 0:
                            continue
                        uu, vv = u + du, v + dv
                        if 0 <= uu < rows and 0 <= vv < cols:
                            total += cos(centre, K[off + uu * cols + vv])
                            count += 1
                phi[off + u * cols + v] = 0.0 if count == 0 else 1.0 - total / count
    return phi


def partition(L, frames):
    hist, cur = [], []
    visual = [False] * L
    for f, (off, rows, cols) in enumerate(frames):
        ids = list(range(off, off + rows * cols))
        for i in ids:
            visual[i] = True
        if f == len(frames) - 1:
            cur = ids
        else:
            hist.extend(ids)
    return hist, cur, visual


def rho(K, hist, cur, snap=1e-4):
    out = {}
    for i in hist:
        best = -2.0
        for j in cur:
            c = cos(K[i], K[j])
            if c > best:
                best = c
        best = min(1.0, max(-1.0, best))
        if best >= 1.0 - snap:
            best = 1.0
        out[i] = best
    return out


def gate(rho_of, hist, L, B):
    g = [1] * L
    m = min(B, len(hist))
    ranked = sorted(hist, key=lambda i: (f32(rho_of[i]), i))
    for i in hist:
        g[i] = 0
    for i in ranked[:m]:
        g[i] = 1
    return g


def scores(A, phi, g, visual, alpha):
    return [g[i] * (A[i] + alpha * phi[i]) if visual[i] else A[i] for i in range(len(A))]


def top_b(S, B):
    ranked = sorted(range(len(S)), key=lambda i: (-f32(S[i]), i))
    return sorted(ranked[:B])


def mean_pool(A, width):
    """(1/width) sum of A over the centred window of width positions, the
    positions outside 0..L-1 counting as 0."""
    r = (width - 1) // 2
    out = []
    for i in range(len(A)):
        acc = 0.0
        for j in range(i - r, i + r + 1):
            if 0 <= j < len(A):
                acc += A[j]
        out.append(acc / width)
    return out


def compress(Q, K, frames, B, alpha=1.0, use_css=True, use_tsg=True, mean_width=0):
    L = len(K)
    A = base_score(Q, K)
    if mean_width:
        A = mean_pool(A, mean_width)
    hist, cur, visual = partition(L, frames)
    phi = css(K, frames) if use_css else [0.0] * L
    r = rho(K, hist, cur)
    g = gate(r, hist, L, B) if use_tsg else [1] * L
    S = scores(A, phi, g, visual, alpha if use_css else 0.0)
    return dict(A=A, phi=phi, rho=r, gate=g, S=S, kept=top_b(S, B))


def decode_attention(Q, K, V):
    """Q: list[G][d], K, V: list[n][d] floats; out: list[G][d] (zeros if n = 0)."""
    G = len(Q)
    d = len(Q[0])
    n = len(K)
    out = [[0.0] * d for _ in range(G)]
    if n == 0:
        return out
    for g in range(G):
        z = [dot(Q[g], K[j]) / math.sqrt(d) for j in range(n)]
        m = max(z)
        e = [math.exp(x - m) for x in z]
        tot = sum(e)
        for j in range(n):
            w = e[j] / tot
            for c in range(d):
                out[g][c] += w * V[j][c]
    return out


def tsg_similarity(K, hist, cur, sim):
    """rho_i = max over current j of dot(k_i, k_j) or of -sqrt(sum_c (k_ic - k_jc)^2)
    (the squared distance snapped to 0 when <= 1e-5 ||k_i||^2); cosine as tsg_rho."""
    out = []
    for i in hist:
        best = None
        for j in cur:
            if sim == "dot":
                v = dot(K[i], K[j])
            else:
                d2 = 0.0
                for a, b in zip(K[i], K[j]):
                    d2 += (a - b) * (a - b)
                if d2 <= 1e-5 * dot(K[i], K[i]):
                    d2 = 0.0
                v = -math.sqrt(d2)
            best = v if best is None or v > best else best
        out.append(best)
    return out


def decode_scores(Q, K):
    """a_i = (1/G) sum_g exp(z_gi) / sum_j exp(z_gj), z = q_g . k / sqrt(d), over all rows."""
    G, L, d = len(Q), len(K), len(K[0])
    a = [0.0] * L
    for g in range(G):
        z = [dot(Q[g], K[i]) / math.sqrt(d) for i in range(L)]
        zm = max(z)
        den = 0.0
        for i in range(L):
            den += math.exp(z[i] - zm)
        for i in range(L):
            a[i] += math.exp(z[i] - zm) / den / G
    return a


def hit_rate(kept, oracle):
    """Fraction of the oracle set found in kept (both lists of token indices)."""
    if not oracle:
        return float("nan")
    hits = 0
    for t in oracle:
        if t in kept:
            hits += 1
    return hits / len(oracle)


def compress_concat(Qs, Ks, frames, B, alpha=1.0):
    """The procedure over a layer's concatenated key space.  Qs: per kv head
    [G][delta][d]; Ks: per kv head [L][d].  A is the mean of the heads' window
    sums; h_t is token t's keys of every head, one after the other."""
    H, L = len(Ks), len(Ks[0])
    A_h = [base_score(Qs[h], Ks[h]) for h in range(H)]
    A = [sum(A_h[h][i] for h in range(H)) / H for i in range(L)]
    K = []
    for i in range(L):
        row = []
        for h in range(H):
            row.extend(Ks[h][i])
        K.append(row)
    hist, cur, visual = partition(L, frames)
    phi = css(K, frames)
    r = rho(K, hist, cur)
    g = gate(r, hist, L, B)
    S = scores(A, phi, g, visual, alpha)
    return dict(A=A, phi=phi, rho=r, gate=g, S=S, kept=top_b(S, B))

