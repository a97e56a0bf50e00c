"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: numbers the
paper prints, closed forms worked by hand (fixtures under tests/golden/),
invariants, library routines for special cases, and the literal-loop twin.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special

from oracle import literal as O1
from oracle import stlite_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def frac(s):
    return float(Fraction(s)) if isinstance(s, str) else float(s)


# ---------------------------------------------------------------- budget ----

def test_budget_paper_instantiation():
    g = golden("f1_instantiation.json")
    assert O.budget(g["W"], *g["rho"]) == g["floor_rho_W"]          # floor(0.76 * 2592) = 1969
    assert O.budget(g["N"], *g["beta"]) == g["B"]                   # 20% of 12000 = 2400


def test_budget_rational_not_float():
    # 0.29 * 100 is 28.999999999999996 in binary floating point; the rational budget is 29.
    assert math.floor(0.29 * 100) == 28
    assert O.budget(100, 29, 100) == 29
    assert O.budget(912, 1, 5) == 182
    assert O.budget(150528, 1, 5) == 30105
    assert O.budget(77, 1, 1) == 77
    with pytest.raises(ValueError):
        O.budget(10, 3, 2)


def test_f1_marginal_rate_paper_numbers():
    """Part (iii) of the F1 proposition with the paper's numbers: when the floor(rho W)
    redundant tokens outrank all others, top-B keeps exactly B - floor(rho W) of the
    N - floor(rho W) non-redundant ones: 431 / 10031 (printed as about 4.3%)."""
    g = golden("f1_instantiation.json")
    N, B, nred = g["N"], g["B"], g["floor_rho_W"]
    rng = np.random.default_rng(5)
    S = rng.uniform(0.0, 1.0, N)
    red = rng.choice(N, nred, replace=False)
    S[red] += 2.0
    kept = O.select_topk(S, B)
    nonred = np.setdiff1d(np.arange(N), red)
    got = Fraction(len(np.intersect1d(kept, nonred)), len(nonred))
    assert got == Fraction(g["marginal_num"], g["marginal_den"])
    assert round(100 * float(got), 1) == g["marginal_percent"]


# ------------------------------------------------------------ base score ----

def _q_k_for_logits(z, d=128):
    """One query and keys along e1 so that q . k_i / sqrt(d) = z_i."""
    L = len(z)
    K = np.zeros((L, d))
    K[:, 0] = z
    Q = np.zeros((1, 1, d))
    Q[0, 0, 0] = math.sqrt(d)
    return Q, K


def test_base_score_worked_example():
    g = golden("base_score_example.json")
    z = [{"0": 0.0, "ln2": math.log(2), "ln3": math.log(3)}[s] for s in g["logits"]]
    Q, K = _q_k_for_logits(z)
    np.testing.assert_allclose(O.base_score(Q, K), [frac(a) for a in g["A"]], rtol=1e-14)


def test_base_score_uniform_logits_closed_form():
    """All logits equal: each window row spreads 1/(p+1) over keys 0..p, so
    A_i = sum_{p >= max(i, L-delta)} 1/(p+1) (causal window, reading R1)."""
    L, delta, G, d = 37, 6, 3, 128
    Q = np.zeros((G, delta, d))
    K = np.random.default_rng(1).standard_normal((L, d))
    want = np.array([sum(1.0 / (p + 1) for p in range(max(i, L - delta), L)) for i in range(L)])
    np.testing.assert_allclose(O.base_score(Q, K), want, rtol=1e-13)


def test_base_score_single_row_is_library_softmax():
    rng = np.random.default_rng(2)
    L, d = 50, 128
    Q = rng.standard_normal((1, 1, d))
    K = rng.standard_normal((L, d))
    want = scipy.special.softmax(K @ Q[0, 0] / math.sqrt(d))
    np.testing.assert_allclose(O.base_score(Q, K), want, rtol=1e-12)


def test_base_score_mass_equals_window():
    rng = np.random.default_rng(3)
    for (L, delta, G) in [(40, 8, 7), (100, 1, 2), (9, 9, 1)]:
        A = O.base_score(rng.standard_normal((G, delta, 128)), rng.standard_normal((L, 128)))
        assert abs(A.sum() - delta) < 1e-11
        assert (A > 0).all()


def test_base_score_gqa_mean_of_heads():
    """Reading R2: a group's A_base is the mean of its heads' single-head scores."""
    rng = np.random.default_rng(4)
    Q = rng.standard_normal((3, 4, 128))
    K = rng.standard_normal((30, 128))
    per = [O.base_score(Q[g:g + 1], K) for g in range(3)]
    np.testing.assert_allclose(O.base_score(Q, K), np.mean(per, axis=0), rtol=1e-13)


def test_f1_part_i_bound_and_part_ii_eviction():
    """F1 proposition, Part (i): the window query gives i* at most
    1/(1 + floor(rho W) e^Delta) when floor(rho W) keys beat it by Delta; the bound
    is reached when every other key is negligible.  Part (ii): with B <= floor(rho W)
    a plain top-B (SnapKV mode) evicts i*."""
    g = golden("f1_instantiation.json")
    delta_gap = g["Delta"]
    n_red = 40
    L = 300
    z = np.full(L, -60.0)
    istar = 17
    z[istar] = 0.0
    red = np.arange(L - n_red, L)
    z[red] = delta_gap
    Q, K = _q_k_for_logits(z)
    A = O.base_score(Q, K)
    bound = 1.0 / (1.0 + n_red * math.exp(delta_gap))
    assert A[istar] <= bound * (1 + 1e-12)
    assert A[istar] == pytest.approx(bound, rel=1e-12)   # the other keys add < 1e-20
    # Part (ii), at B = floor(rho W) and below.
    for B in (n_red, n_red - 7):
        S = O.integrate(A, np.zeros(L), np.ones(L, np.uint8), np.zeros(L, bool), 0.0)
        assert istar not in set(O.select_topk(S, B))
    # The printed instantiation: 1 / (1 + 1969 e^2.1) is 6.2e-5.
    inst = 1.0 / (1.0 + g["floor_rho_W"] * math.exp(g["Delta"]))
    assert float(f"{inst:.{g['attn_bound_sig_digits'] - 1}e}") == g["attn_bound"]


# ------------------------------------------------------------------- CSS ----

def _grid(cells, d=128):
    e = np.eye(d)
    return np.array([[c(e) for c in row] for row in cells]).reshape(-1, d)


def test_css_golden_patterns():
    g = golden("css_patterns.json")["patterns"]
    e1 = lambda e: e[0]
    e2 = lambda e: e[1]
    ne1 = lambda e: -e[0]
    grids = {
        "identical": [[e1] * 3] * 3,
        "centre_e1_ring_e2": [[e2, e2, e2], [e2, e1, e2], [e2, e2, e2]],
        "checkerboard": [[e1, ne1, e1], [ne1, e1, ne1], [e1, ne1, e1]],
    }
    for name, cells in grids.items():
        want = np.array([[frac(x) for x in row] for row in g[name]["phi"]]).reshape(-1)
        got = O.css_frame(_grid(cells), 3, 3)
        np.testing.assert_allclose(got, want, atol=1e-15, err_msg=name)


def test_css_border_counts_and_degenerate_grids():
    rng = np.random.default_rng(6)
    assert O.css_frame(rng.standard_normal((1, 128)), 1, 1).tolist() == [0.0]
    X = rng.standard_normal((2, 128))
    c = X[0] @ X[1] / np.linalg.norm(X[0]) / np.linalg.norm(X[1])
    np.testing.assert_allclose(O.css_frame(X, 1, 2), [1 - c, 1 - c], rtol=1e-14)
    # a zero key has cosine 0 with everything (R6)
    X = rng.standard_normal((9, 128))
    X[4] = 0
    phi = O.css_frame(X, 3, 3)
    assert phi[4] == 1.0


def test_css_range_and_scale_invariance():
    rng = np.random.default_rng(7)
    X = rng.standard_normal((5 * 7, 128))
    phi = O.css_frame(X, 5, 7)
    assert (phi >= 0).all() and (phi <= 2).all()
    scales = rng.uniform(0.1, 10.0, size=(35, 1))
    np.testing.assert_allclose(O.css_frame(X * scales, 5, 7), phi, rtol=1e-12, atol=1e-14)


# ------------------------------------------------------------------- TSG ----

def test_tsg_golden_example():
    g = golden("tsg_example.json")
    e = np.eye(128)
    hist_vecs = [e[0], (e[0] + e[1]) / math.sqrt(2), -e[0], e[2]]
    K = np.array(hist_vecs + [e[0], e[1]])
    hist = np.arange(4)
    cur = np.array([4, 5])
    rho = O.tsg_rho(K, hist, cur)
    want = [{"1": 1.0, "1/sqrt2": 1 / math.sqrt(2), "0": 0.0}[s] for s in g["rho"]]
    np.testing.assert_allclose(rho, want, atol=1e-15)
    for B, gate in g["gate_by_budget"].items():
        got, tau = O.tsg_gate(rho, hist, 6, int(B))
        assert got[:4].tolist() == gate, B
        assert got[4:].tolist() == [1, 1]            # current frame exempt


def test_tsg_count_invariant_and_threshold():
    rng = np.random.default_rng(8)
    L = 200
    K = rng.standard_normal((L, 128))
    hist = np.arange(0, 150)
    cur = np.arange(150, 190)
    rho = O.tsg_rho(K, hist, cur)
    for B in (0, 1, 37, 149, 150, 500):
        gate, tau = O.tsg_gate(rho, hist, L, B)
        m = min(B, len(hist))
        assert gate[hist].sum() == m
        assert gate[150:].all()
        if 0 < m:
            r32 = rho.astype(np.float32)
            assert (r32[gate[hist] == 1] <= np.float32(tau)).all()
            assert (r32[gate[hist] == 0] >= np.float32(tau)).all()


def test_tsg_rho_brute_force_and_snap():
    rng = np.random.default_rng(9)
    K = rng.standard_normal((30, 128))
    K[3] = K[25] * 2.5            # exact duplicate direction of a current-frame key
    K[4] = K[26] + 1e-3 * rng.standard_normal(128)  # near duplicate: cos > 1 - 1e-4
    hist = np.arange(0, 20)
    cur = np.arange(20, 30)
    rho = O.tsg_rho(K, hist, cur)
    for t, i in enumerate(hist):
        best = max(K[i] @ K[j] / np.linalg.norm(K[i]) / np.linalg.norm(K[j]) for j in cur)
        if best < 1 - 1e-4:
            assert rho[t] == pytest.approx(best, abs=1e-14)
    assert rho[3] == 1.0 and rho[4] == 1.0




# ------------------------------------------- CSS neighbourhood-size ablation ----

def _span(x, n, r):
    """(length, position of x) of the in-grid window [x - r, x + r] of a size-n axis."""
    lo, hi = max(0, x - r), min(n - 1, x + r)
    return hi - lo + 1, x - lo


@pytest.mark.parametrize("k", [5, 7, 9])
def test_css_wide_literal_twin(k):
    rng = np.random.default_rng(30 + k)
    frames = [(0, 1, 1), (1, 2, 3), (7, 6, 7), (49, 10, 4), (89, 3, 11)]
    K = rng.standard_normal((89 + 33 + 5, 8))
    K[3] = 0.0                       # a zero key: its cosines are 0 (R6)
    got = O.css_saliency(K, frames, k)
    want = O1.css(K.tolist(), frames, k)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12)
    assert got[0] == 0.0 and (got[-5:] == 0).all()   # 1x1 frame and text


@pytest.mark.parametrize("k", [5, 7, 9])
def test_css_wide_spike_closed_form(k):
    """A grid of e2 with one cell e1: that cell has Phi = 1; a cell whose k x k
    window holds it has Phi = 1/n (n = its in-grid neighbour count: one
    orthogonal neighbour among n); every other cell has Phi = 0."""
    rows, cols, u0, v0, r = 9, 13, 3, 9, k // 2
    K = np.tile(np.eye(4)[1], (rows * cols, 1))
    K[u0 * cols + v0] = np.eye(4)[0]
    phi = O.css_frame(K, rows, cols, k).reshape(rows, cols)
    for u in range(rows):
        for v in range(cols):
            n = _span(u, rows, r)[0] * _span(v, cols, r)[0] - 1
            if (u, v) == (u0, v0):
                want = 1.0
            elif abs(u - u0) <= r and abs(v - v0) <= r:
                want = 1.0 / n
            else:
                want = 0.0
            assert phi[u, v] == pytest.approx(want, abs=1e-15), (u, v)


@pytest.mark.parametrize("k", [3, 5, 7, 9])
def test_css_wide_checkerboard_closed_form(k):
    """+-e1 checkerboard: cos = +1 with cells of the centre's parity, -1 with the
    others.  Over an a x b window with the centre at (i, j), the cells of parity
    p number ceil(a/2) ceil(b/2) + floor(a/2) floor(b/2) for p = 0, so
    Phi = 1 - (same - opp) / (a b - 1) with same = (count of the centre's parity) - 1."""
    rows, cols, r = 7, 10, k // 2
    sign = np.array([[1.0 if (u + v) % 2 == 0 else -1.0 for v in range(cols)] for u in range(rows)])
    K = sign.reshape(-1, 1) * np.eye(3)[0]
    phi = O.css_frame(K, rows, cols, k).reshape(rows, cols)
    for u in range(rows):
        for v in range(cols):
            (a, i), (b, j) = _span(u, rows, r), _span(v, cols, r)
            even = -(-a // 2) * -(-b // 2) + (a // 2) * (b // 2)
            same = (even if (i + j) % 2 == 0 else a * b - even) - 1
            opp = a * b - 1 - same
            assert phi[u, v] == pytest.approx(1 - (same - opp) / (a * b - 1), abs=1e-14), (k, u, v)


def test_css_wide_whole_grid_and_defaults():
    """k at least twice the grid's extent: every cell averages its cosines with
    all other cells (full Gram matrix less the diagonal); a uniform frame has
    Phi = 0 at every k; k = 3 is the default; other sizes are rejected."""
    rng = np.random.default_rng(33)
    X = rng.standard_normal((12, 16))
    U = X / np.linalg.norm(X, axis=1, keepdims=True)
    G = U @ U.T
    want = 1 - (G.sum(axis=1) - np.diag(G)) / 11
    np.testing.assert_allclose(O.css_frame(X, 3, 4, 9), want, atol=1e-14)
    np.testing.assert_allclose(O.css_frame(X, 3, 4, 7), want, atol=1e-14)
    Y = np.tile(rng.standard_normal(16), (30, 1))
    for k in (3, 5, 7, 9):
        np.testing.assert_allclose(O.css_frame(Y, 5, 6, k), 0.0, atol=1e-15)
    frames = [(0, 4, 5), (20, 3, 3)]
    Z = rng.standard_normal((35, 16))
    np.testing.assert_array_equal(O.css_saliency(Z, frames, 3), O.css_saliency(Z, frames))
    for bad in (1, 4, 11):
        with pytest.raises(ValueError):
            O.css_frame(Z[:20], 4, 5, bad)

# ------------------------------------------------ TSG similarity variants ----

def test_tsg_similarity_literal_twin_and_cosine_route():
    rng = np.random.default_rng(21)
    K = rng.standard_normal((24, 16)) * rng.uniform(0.2, 3.0, (24, 1))  # mixed magnitudes
    K[2] = K[20]                                # exact duplicate of a current-frame key
    K[5] = K[21] + 1e-4 * rng.standard_normal(16)   # d^2 ~ 1.6e-7, well inside the snap
    hist, cur = np.arange(0, 16), np.arange(16, 24)
    for sim in ("dot", "neg_l2"):
        got = O.tsg_similarity(K, hist, cur, sim)
        want = O1.tsg_similarity(K.tolist(), hist.tolist(), cur.tolist(), sim)
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(O.tsg_similarity(K, hist, cur, "cosine"), O.tsg_rho(K, hist, cur))
    nl2 = O.tsg_similarity(K, hist, cur, "neg_l2")
    assert nl2[2] == 0.0 and nl2[5] == 0.0 and (nl2 <= 0).all()
    # the dot product is not magnitude invariant: a longer current key can beat the duplicate
    dot = O.tsg_similarity(K, hist, cur, "dot")
    assert dot[2] >= K[20] @ K[20]
    assert dot[2] == pytest.approx(max(K[20] @ K[j] for j in cur), rel=1e-15)
    with pytest.raises(ValueError):
        O.tsg_similarity(K, hist, cur, "manhattan")
    assert O.tsg_similarity(K, hist[:0], cur, "dot").shape == (0,)


def test_tsg_similarity_closed_forms():
    """Orthonormal keys: dot = 0 and -L2 = -sqrt(2) between distinct axes; k_i = c e_j
    gives dot = c and -L2 = -|c - 1|.  On unit-norm keys the three metrics order
    tokens alike: dot = cos and -L2 = -sqrt(2 - 2 cos)."""
    E = np.eye(8)
    K = np.vstack([E[4], E[5], 3.0 * E[0], 0.5 * E[1], E[0], E[1]])
    hist, cur = np.arange(0, 4), np.arange(4, 6)
    np.testing.assert_allclose(O.tsg_similarity(K, hist, cur, "dot"), [0, 0, 3.0, 0.5], atol=0)
    np.testing.assert_allclose(O.tsg_similarity(K, hist, cur, "neg_l2"),
                               [-math.sqrt(2), -math.sqrt(2), -2.0, -0.5], rtol=1e-15)
    rng = np.random.default_rng(22)
    U = rng.standard_normal((40, 32))
    U /= np.linalg.norm(U, axis=1, keepdims=True)
    hist, cur = np.arange(0, 30), np.arange(30, 40)
    cosr = O.tsg_rho(U, hist, cur)
    assert (cosr < 1 - 1e-4).all()
    np.testing.assert_allclose(O.tsg_similarity(U, hist, cur, "dot"), cosr, atol=1e-14)
    np.testing.assert_allclose(O.tsg_similarity(U, hist, cur, "neg_l2"),
                               -np.sqrt(2 - 2 * cosr), atol=1e-12)


def test_tsg_similarity_scale_behaviour_and_l2_snap_edge():
    """Dot scales with c^2 and -L2 with |c| when all keys are scaled by c; the cosine
    is scale free.  The negative-L2 snap fires at d^2 <= 1e-5 ||k_i||^2 exactly."""
    rng = np.random.default_rng(23)
    K = rng.standard_normal((20, 16))
    hist, cur = np.arange(0, 12), np.arange(12, 20)
    c = 2.0 ** 3
    np.testing.assert_allclose(O.tsg_similarity(c * K, hist, cur, "dot"),
                               c * c * O.tsg_similarity(K, hist, cur, "dot"), rtol=1e-14)
    np.testing.assert_allclose(O.tsg_similarity(c * K, hist, cur, "neg_l2"),
                               c * O.tsg_similarity(K, hist, cur, "neg_l2"), rtol=1e-12)
    np.testing.assert_allclose(O.tsg_rho(c * K, hist, cur), O.tsg_rho(K, hist, cur), atol=1e-14)
    # k_i = (1, 0, ...), current key (1, t, 0, ...): d^2 = t^2, ||k_i||^2 = 1
    for t, snapped in ((math.sqrt(0.9e-5), True), (math.sqrt(1.1e-5), False)):
        K2 = np.zeros((2, 4))
        K2[0, 0] = 1.0
        K2[1, 0], K2[1, 1] = 1.0, t
        r = O.tsg_similarity(K2, np.array([0]), np.array([1]), "neg_l2")[0]
        assert (r == 0.0) if snapped else r == pytest.approx(-t, rel=1e-9)


def test_tsg_fixed_gate_hand_example():
    """tau = 0.85, the fixed-threshold control of the necessity table: a historical
    token is kept iff float32(rho) <= float32(0.85); text and current frame keep 1."""
    L = 9
    hist = np.array([0, 1, 2, 3, 5, 6])
    rho = np.array([0.2, 0.85, 0.8500001, 1.0, 0.85 + 1e-12, -0.3])
    gate = O.tsg_fixed_gate(rho, hist, L, 0.85)
    # 0.85 + 1e-12 rounds to float32(0.85) and is kept (decided in float32, R-dec);
    # 0.8500001 is a distinct float32 above it and is dropped.
    assert gate.tolist() == [1, 1, 0, 0, 1, 1, 1, 1, 1]
    assert O.tsg_fixed_gate(rho, hist, L, 1.0).tolist() == [1] * L
    assert O.tsg_fixed_gate(rho, hist, L, -1.0).tolist() == [0, 0, 0, 0, 1, 0, 0, 1, 1]
    assert O.tsg_fixed_gate(rho[:0], hist[:0], 4, 0.5).tolist() == [1] * 4


def _frames_seq(rng, n_frames, rows, cols, text, dup_of_last=None):
    """Build a small sequence (keys fp32-representable as bf16) with frames+text."""
    d = 128
    frames, chunks, off = [], [], 0
    for f in range(n_frames):
        chunks.append(rng.standard_normal((rows * cols, d)))
        frames.append((off, rows, cols))
        off += rows * cols
        chunks.append(rng.standard_normal((text, d)))
        off += text
    K = np.concatenate(chunks)
    if dup_of_last is not None:   # historical frame dup_of_last becomes a copy of the current frame
        o, r, c = frames[dup_of_last]
        oc = frames[-1][0]
        K[o:o + r * c] = K[oc:oc + r * c]
    return K, frames


def test_duplicate_frame_gated_out_and_never_kept():
    """A historical frame equal to the current frame has rho = 1 everywhere; with at
    least m other historical tokens below the snap band it is gated out entirely,
    so none of its tokens can be kept."""
    rng = np.random.default_rng(10)
    K, frames = _frames_seq(rng, 4, 4, 5, 6, dup_of_last=1)
    L = K.shape[0]
    hist, cur, text = O.split_tokens(L, frames)
    rho = O.tsg_rho(K, hist, cur)
    o, r, c = frames[1]
    dup_tokens = np.arange(o, o + r * c)
    in_dup = np.isin(hist, dup_tokens)
    assert (rho[in_dup] == 1.0).all()
    B = O.budget(L, 1, 5)
    m = min(B, len(hist))
    assert (rho[~in_dup] < 1 - 1e-4).sum() >= m
    gate, _ = O.tsg_gate(rho, hist, L, B)
    assert gate[dup_tokens].sum() == 0
    A = np.full(L, 1.0 / L)
    visual = np.zeros(L, bool)
    visual[hist] = True
    visual[cur] = True
    S = O.integrate(A, O.css_saliency(K, frames), gate, visual, 1.0)
    assert not np.isin(O.select_topk(S, B), dup_tokens).any()


def test_single_frame_tsg_is_noop():
    rng = np.random.default_rng(11)
    L, d = 60, 128
    Kb = np.asarray(rng.integers(0x3c00, 0x3f80, size=(L, d)), np.uint16)
    Kb[::2] |= 0x8000
    Vb = np.asarray(rng.integers(0, 0xFFFF, size=(L, d)), np.uint16)
    Qb = np.asarray(rng.integers(0x3c00, 0x3f80, size=(2, 4, d)), np.uint16)
    frames = [(0, 5, 8)]
    on = O.compress_unit(Qb, Kb, Vb, frames, (1, 5))
    off = O.compress_unit(Qb, Kb, Vb, frames, (1, 5), use_tsg=False)
    assert on["kept"].tolist() == off["kept"].tolist()
    assert on["gate"].all()


# ------------------------------------------------------- integrate/select ----

def test_select_properties_brute_force():
    rng = np.random.default_rng(12)
    for trial in range(30):
        L = int(rng.integers(1, 40))
        S = rng.choice([0.0, 0.25, 0.5, 1.0], size=L) if trial % 2 else rng.uniform(0, 1, L)
        B = int(rng.integers(0, L + 1))
        kept = O.select_topk(S, B)
        assert len(kept) == B and (np.diff(kept) > 0).all()
        ks = set(kept.tolist())
        for i in ks:
            for j in range(L):
                if j not in ks:
                    assert S[i] > S[j] or (S[i] == S[j] and i < j)


def test_beta_one_keeps_everything_and_snapkv_mode():
    rng = np.random.default_rng(13)
    L, d = 48, 128
    Kb = np.asarray(rng.integers(0x3c00, 0x3f80, size=(L, d)), np.uint16)
    Kb[1::3] |= 0x8000
    Vb = np.asarray(rng.integers(0, 0xFFFF, size=(L, d)), np.uint16)
    Qb = np.asarray(rng.integers(0x3c00, 0x3f80, size=(1, 3, d)), np.uint16)
    frames = [(0, 3, 4), (16, 3, 4)]
    full = O.compress_unit(Qb, Kb, Vb, frames, (1, 1))
    assert full["kept"].tolist() == list(range(L))
    assert (full["k_out"] == Kb).all() and (full["v_out"] == Vb).all()
    # SnapKV mode (alpha = 0, TSG off) keeps the B largest A_base.
    snap = O.compress_unit(Qb, Kb, Vb, frames, (1, 4), use_css=False, use_tsg=False)
    A = snap["A"].astype(np.float32)
    thr = np.sort(A)[::-1][snap["B"] - 1]
    assert (A[snap["kept"]] >= thr).all()
    assert (A[np.setdiff1d(np.arange(L), snap["kept"])] <= thr).all()


def test_integrate_modal_cases():
    A = np.array([0.1, 0.2, 0.3, 0.4])
    phi = np.array([0.5, 0.6, 0.7, 0.8])
    gate = np.array([1, 0, 1, 0], np.uint8)
    visual = np.array([False, False, True, True])
    S = O.integrate(A, phi, gate, visual, 2.0)
    np.testing.assert_allclose(S, [0.1, 0.2, 0.3 + 1.4, 0.0])


# --------------------------------------------------- literal twin (O1 = O2) --

@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_literal_twin_agrees(seed):
    rng = np.random.default_rng(100 + seed)
    d = 128
    rows, cols = [(2, 3), (3, 3), (1, 4), (4, 2)][seed]
    nfr = [3, 2, 1, 3][seed]
    text = [4, 3, 7, 2][seed]
    chunks, frames, off = [], [], 0
    for f in range(nfr):
        frames.append((off, rows, cols))
        chunks.append(rng.standard_normal((rows * cols, d)) / math.sqrt(d))
        off += rows * cols
        chunks.append(rng.standard_normal((text, d)) / math.sqrt(d))
        off += text
    K = np.concatenate(chunks)
    if nfr > 1:   # one exact copy of a current-frame key in the history (snap class)
        K[frames[0][0]] = K[frames[-1][0] + 1]
    L = K.shape[0]
    Kb = np.asarray(np.round(K * 64), np.int64)   # coarse values: exact in bf16
    K = Kb / 64.0
    G, delta = [2, 7, 1, 3][seed], [3, 2, 4, 1][seed]
    Q = np.round(rng.standard_normal((G, delta, d)) * 8) / 64.0
    B = O.budget(L, [1, 1, 2, 3][seed], [5, 3, 5, 4][seed])
    alpha = [1.0, 0.5, 2.0, 1.0][seed]
    lit = O1.compress([[list(map(float, r)) for r in g] for g in Q],
                      [list(map(float, r)) for r in K], frames, B, alpha)
    A = O.base_score(Q, K)
    np.testing.assert_allclose(A, lit["A"], rtol=1e-12, atol=0)
    hist, cur, text_idx = O.split_tokens(L, frames)
    phi = O.css_saliency(K, frames)
    np.testing.assert_allclose(phi, lit["phi"], rtol=1e-12, atol=1e-13)
    rho = O.tsg_rho(K, hist, cur)
    np.testing.assert_allclose(rho, [lit["rho"][int(i)] for i in hist], atol=1e-13)
    gate, _ = O.tsg_gate(rho, hist, L, B)
    assert gate.tolist() == lit["gate"]
    visual = np.zeros(L, bool)
    visual[hist] = True
    visual[cur] = True
    S = O.integrate(A, phi, gate, visual, alpha)
    np.testing.assert_allclose(S, lit["S"], rtol=1e-12, atol=1e-14)
    assert O.select_topk(S, B).tolist() == lit["kept"]


@pytest.mark.filterwarnings("ignore::RuntimeWarning")
def test_bf16_widening_matches_torch():
    torch = pytest.importorskip("torch")
    bits = np.arange(0, 1 << 16, dtype=np.uint16)
    finite = ((bits >> 7) & 0xFF) != 0xFF
    want = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(O.bf16_to_f64(bits)[finite], want[finite])


# ------------------------------------------- decode attention over a cache --

def test_decode_single_row_and_empty_cache():
    rng = np.random.default_rng(21)
    Q = rng.standard_normal((3, 128))
    K = rng.standard_normal((1, 128))
    V = rng.standard_normal((1, 128))
    # softmax over one row is 1: every query returns that row's value
    np.testing.assert_array_equal(O.decode_attention(Q, K, V), np.repeat(V, 3, axis=0))
    assert not O.decode_attention(Q, K[:0], V[:0]).any()


def test_decode_uniform_logits_is_mean_of_values():
    rng = np.random.default_rng(22)
    K = rng.standard_normal((37, 128))
    V = rng.standard_normal((37, 128))
    out = O.decode_attention(np.zeros((2, 128)), K, V)
    np.testing.assert_allclose(out, np.repeat(V.mean(axis=0, keepdims=True), 2, axis=0), rtol=1e-13, atol=1e-15)


def test_decode_two_level_logits_closed_form():
    """Keys along e1 give logits a (rows in A) and b (rows in B): the output is
    the mean of A's values weighted e^a against B's weighted e^b."""
    rng = np.random.default_rng(23)
    d, a, b = 128, 2.5, -1.0
    inA = rng.random(40) < 0.3
    K = np.zeros((40, d))
    K[:, 0] = np.where(inA, a, b)
    Q = np.zeros((1, d))
    Q[0, 0] = math.sqrt(d)
    V = rng.standard_normal((40, d))
    want = (math.exp(a) * V[inA].sum(0) + math.exp(b) * V[~inA].sum(0)) / (
        math.exp(a) * inA.sum() + math.exp(b) * (~inA).sum())
    np.testing.assert_allclose(O.decode_attention(Q, K, V)[0], want, rtol=1e-12, atol=1e-14)


def test_decode_library_softmax_and_invariants():
    rng = np.random.default_rng(24)
    Q = rng.standard_normal((7, 128)) * 0.5
    K = rng.standard_normal((50, 128))
    V = rng.standard_normal((50, 128))
    out = O.decode_attention(Q, K, V)
    P = scipy.special.softmax(Q @ K.T / math.sqrt(128), axis=1)
    np.testing.assert_allclose(out, P @ V, rtol=1e-12, atol=1e-13)
    # permuting the cached rows changes nothing; shifting every value by c shifts the output by c
    perm = rng.permutation(50)
    np.testing.assert_allclose(O.decode_attention(Q, K[perm], V[perm]), out, rtol=1e-12, atol=1e-13)
    c = rng.standard_normal(128)
    np.testing.assert_allclose(O.decode_attention(Q, K, V + c), out + c, rtol=1e-12, atol=1e-12)
    # a convex combination of the values: inside their per-dimension range
    assert (out <= V.max(0) + 1e-12).all() and (out >= V.min(0) - 1e-12).all()


def test_decode_literal_twin_agrees():
    rng = np.random.default_rng(25)
    Q = rng.standard_normal((3, 16))
    K = rng.standard_normal((11, 16))
    V = rng.standard_normal((11, 16))
    lit = O1.decode_attention(Q.tolist(), K.tolist(), V.tolist())
    np.testing.assert_allclose(O.decode_attention(Q, K, V), lit, rtol=1e-12, atol=1e-14)


def test_decode_over_compacted_cache_at_beta_one_is_full_decode():
    """At beta = 1 the compacted cache is the full cache in token order."""
    rng = np.random.default_rng(26)
    L, d = 40, 128
    Kb = np.asarray(rng.integers(0x3c00, 0x3f80, size=(L, d)), np.uint16)
    Kb[1::3] |= 0x8000
    Vb = np.asarray(rng.integers(0x3000, 0x4000, size=(L, d)), np.uint16)
    Qb = np.asarray(rng.integers(0x3c00, 0x3f80, size=(1, 3, d)), np.uint16)
    res = O.compress_unit(Qb, Kb, Vb, [(0, 3, 4), (16, 3, 4)], (1, 1))
    Qd = O.bf16_to_f64(Qb[0, :2])
    full = O.decode_attention(Qd, O.bf16_to_f64(Kb), O.bf16_to_f64(Vb))
    comp = O.decode_attention(Qd, O.bf16_to_f64(res["k_out"]), O.bf16_to_f64(res["v_out"]))
    np.testing.assert_array_equal(full, comp)


# ------------------------------------------------------- cache hit rate ----

def test_decode_attention_scores_definition():
    rng = np.random.default_rng(40)
    G, L, d = 3, 17, 8
    Q, K = rng.standard_normal((G, d)), rng.standard_normal((L, d))
    a = O.decode_attention_scores(Q, K)
    np.testing.assert_allclose(a, O1.decode_scores(Q.tolist(), K.tolist()), atol=1e-15)
    # the decode query sees every cached key: window scoring with delta = 1 at
    # the last position is the same distribution
    np.testing.assert_allclose(a, O.base_score(Q[:, None, :], K), atol=1e-15)
    np.testing.assert_allclose(a, scipy.special.softmax(Q @ K.T / math.sqrt(d), axis=1).mean(axis=0), atol=1e-15)
    assert a.sum() == pytest.approx(1.0, abs=1e-14)
    np.testing.assert_allclose(O.decode_attention_scores(np.zeros((2, d)), K), np.full(L, 1 / L), atol=1e-16)
    # two logit levels: keys e1 (logit x) and 0 (logit 0) under q = x sqrt(d) e1
    K2 = np.zeros((5, d))
    K2[[1, 3], 0] = 1.0
    x = 0.7
    q = np.zeros((1, d))
    q[0, 0] = x * math.sqrt(d)
    hi = math.exp(x) / (2 * math.exp(x) + 3)
    np.testing.assert_allclose(O.decode_attention_scores(q, K2), [(1 - 2 * hi) / 3, hi, (1 - 2 * hi) / 3, hi,
                                                                  (1 - 2 * hi) / 3], atol=1e-15)


def test_cache_hit_rate_definition_and_random_expectation():
    assert O.cache_hit_rate(np.array([1, 2, 3]), np.array([2, 3, 4])) == pytest.approx(2 / 3)
    assert O.cache_hit_rate(np.array([5, 6]), np.array([5, 6])) == 1.0
    assert O.cache_hit_rate(np.array([0, 1]), np.array([5, 6])) == 0.0
    assert math.isnan(O.cache_hit_rate(np.array([], int), np.array([], int)))
    assert O1.hit_rate([1, 2, 3], [2, 3, 4]) == O.cache_hit_rate(np.array([1, 2, 3]), np.array([2, 3, 4]))
    # the paper's footnote: random selection hits beta in expectation (hypergeometric mean B^2/L / B)
    rng = np.random.default_rng(41)
    L, B = 500, 100
    oracle = O.chr_oracle_set(rng.uniform(size=L), B)
    rates = [O.cache_hit_rate(np.sort(rng.choice(L, B, replace=False)), oracle) for _ in range(4000)]
    sd = math.sqrt((B / L) * (1 - B / L) * (L - B) / (L - 1) / B) / math.sqrt(len(rates))
    assert abs(np.mean(rates) - B / L) < 5 * sd


def test_chr_oracle_set_brute_force_and_snapkv_identity():
    """I* is the top-B by (attention desc, index asc); SnapKV voting with a
    one-query window equal to the decode query keeps exactly I* (CHR = 1)."""
    rng = np.random.default_rng(42)
    a = np.round(rng.uniform(size=40), 1)      # many ties
    for B in (0, 1, 7, 40):
        want = sorted(sorted(range(40), key=lambda i: (-np.float32(a[i]), i))[:B])
        assert O.chr_oracle_set(a, B).tolist() == want
    G, L, d = 4, 60, 16
    Q, K = rng.standard_normal((G, d)), rng.standard_normal((L, d))
    B = O.budget(L, 1, 5)
    oracle = O.chr_oracle_set(O.decode_attention_scores(Q, K), B)
    snap = O.select_topk(O.base_score(Q[:, None, :], K), B)
    assert O.cache_hit_rate(snap, oracle) == 1.0



def test_uniform_base_prior_closed_forms():
    """A constant A: with no CSS and no gate the top-B is the first B tokens
    (index tie-break); with Phi it ranks visual tokens by Phi, text at the
    constant, and gated-out visual tokens last (S = 0)."""
    L, B, c = 12, 5, 0.25
    A = np.full(L, c)
    visual = np.zeros(L, bool)
    visual[2:10] = True
    assert O.select_topk(O.integrate(A, np.zeros(L), np.ones(L, np.uint8), visual, 1.0), B).tolist() == [0, 1, 2, 3, 4]
    phi = np.zeros(L)
    phi[[3, 7, 8]] = [0.5, 0.9, 0.1]
    gate = np.ones(L, np.uint8)
    gate[7] = 0
    S = O.integrate(A, phi, gate, visual, 1.0)
    # scores: 3 -> 0.75, 8 -> 0.35, the other visual and text tokens -> 0.25, token 7 -> 0
    assert O.select_topk(S, B).tolist() == [0, 1, 2, 3, 8]


# ----------------------------------------------- concatenated-head key space ----

def _concat_case(seed, H=2, G=2, delta=3, d=128):
    rng = np.random.default_rng(200 + seed)
    frames = [(0, 2, 3), (10, 2, 3), (20, 3, 2)]
    L = 30
    Kb = np.round(rng.standard_normal((H, L, d)) / math.sqrt(d) * 64) / 64.0   # exact in bf16
    Kb[:, 2] = Kb[:, 21]           # a token equal to a current-frame token in every head (snap class)
    Q = np.round(rng.standard_normal((H * G, delta, d)) * 8) / 64.0
    to_bits = lambda x: (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.uint16)
    return frames, L, to_bits(Q), to_bits(Kb), to_bits(rng.standard_normal((H, L, d)))


@pytest.mark.parametrize("seed", [0, 1])
def test_concat_literal_twin(seed):
    frames, L, qb, kb, vb = _concat_case(seed, H=[2, 4][seed], G=[2, 1][seed])
    out = O.compress_layer_concat(qb, kb, vb, frames, (1, 4), 1.0)
    Q, K = O.bf16_to_f64(qb), O.bf16_to_f64(kb)
    H = K.shape[0]
    G = Q.shape[0] // H
    lit = O1.compress_concat([Q[h * G:(h + 1) * G].tolist() for h in range(H)], [K[h].tolist() for h in range(H)],
                             frames, out["B"], 1.0)
    np.testing.assert_allclose(out["A"], lit["A"], rtol=1e-12, atol=0)
    np.testing.assert_allclose(out["phi"], lit["phi"], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(out["rho"], [lit["rho"][int(i)] for i in out["hist"]], atol=1e-13)
    assert out["gate"].tolist() == lit["gate"]
    assert out["kept"].tolist() == lit["kept"]
    assert out["rho"][list(out["hist"]).index(2)] == 1.0
    assert (out["k_out"] == kb[:, out["kept"]]).all() and out["k_out"].shape == (H, out["B"], 128)


def test_concat_one_head_is_the_per_head_procedure():
    frames, L, qb, kb, vb = _concat_case(2, H=1, G=3)
    cat = O.compress_layer_concat(qb, kb, vb, frames, (1, 4), 0.5)
    one = O.compress_unit(qb, kb[0], vb[0], frames, (1, 4), 0.5)
    for k in ("A", "phi", "rho", "S"):
        np.testing.assert_array_equal(cat[k], one[k])
    assert cat["kept"].tolist() == one["kept"].tolist() and cat["gate"].tolist() == one["gate"].tolist()


def test_concat_identical_heads_match_one_head():
    """Every kv head with the same keys and the same queries: the concatenated
    cosines equal one head's, the mean A equals one head's A, and so the kept set
    is the per-head one."""
    frames, L, qb, kb, vb = _concat_case(3, H=1, G=2)
    kb4 = np.repeat(kb, 4, axis=0)
    qb4 = np.tile(qb, (4, 1, 1))
    cat = O.compress_layer_concat(qb4, kb4, np.repeat(vb, 4, axis=0), frames, (1, 3), 1.0)
    one = O.compress_unit(qb, kb[0], vb[0], frames, (1, 3), 1.0)
    np.testing.assert_allclose(cat["A"], one["A"], rtol=1e-14)
    np.testing.assert_allclose(cat["phi"], one["phi"], atol=1e-14)
    np.testing.assert_allclose(cat["rho"], one["rho"], atol=1e-14)
    assert cat["kept"].tolist() == one["kept"].tolist()



# ------------------------------------------- packed varlen batch entry point --

def _bits(x):
    """bf16 bit patterns of float values that bf16 holds exactly."""
    f = np.asarray(x, dtype=np.float32)
    b = f.view(np.uint32)
    assert ((b & 0xFFFF) == 0).all(), "value not exact in bf16"
    return (b >> 16).astype(np.uint16)


def test_compress_sequence_packed_batch_matches_hand_slices():
    """compress_sequence on a packed batch of three sequences (ragged lengths,
    one text-only) equals compress_unit and the literal twin run on arrays
    sliced by hand: the contiguous GQA group of query heads kv*G .. kv*G+G-1,
    the sequence's own token range and frames with local offsets.  The local
    frames and the per-head queries are built first and packed afterwards, so
    an interleaved head slice, a wrong sequence offset or frames left absolute
    give different inputs to the two sides."""
    rng = np.random.default_rng(2024)
    d, G, Hkv, n_layers, delta = 128, 2, 2, 2, 3
    beta, alpha = (1, 3), 1.0
    # local layouts: (frames as (local offset, rows, cols), length)
    seqs = [([(2, 2, 3), (10, 2, 3), (19, 3, 2)], 29),   # text, frames, text between, trailing text
            ([], 11),                                        # text only
            ([(0, 3, 3), (12, 3, 3)], 25)]                  # frame first, current frame then text
    lens = [L for _, L in seqs]
    cu_seqlens = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    cu_frames = np.concatenate([[0], np.cumsum([len(f) for f, _ in seqs])]).astype(np.int32)
    frame_meta = np.array([(int(cu_seqlens[s]) + o, r, c) for s, (fr, _) in enumerate(seqs) for o, r, c in fr],
                          np.int32).reshape(-1, 3)
    Lt = int(cu_seqlens[-1])
    coarse = lambda *shape: np.round(rng.standard_normal(shape) * 8) / 64.0   # exact in bf16
    # distinct queries per (layer, sequence, query head), keys/values per (layer, kv head)
    Qf = coarse(n_layers, len(seqs), G * Hkv, delta, d)
    Kf = coarse(n_layers, Hkv, Lt, d)
    Vf = coarse(n_layers, Hkv, Lt, d)
    # one current-frame key copied into the history of sequence 0 (the snap class)
    a0 = int(cu_seqlens[0])
    Kf[:, :, a0 + 2] = Kf[:, :, a0 + 19 + 1]
    q_bits, k_bits, v_bits = _bits(Qf), _bits(Kf), _bits(Vf)
    for s, (frames_local, L) in enumerate(seqs):
        a = int(cu_seqlens[s])
        assert O.seq_frames_local(cu_seqlens, cu_frames, frame_meta, s) == frames_local
        for layer in range(n_layers):
            for kv in range(Hkv):
                got = O.compress_sequence(q_bits, k_bits, v_bits, cu_seqlens, cu_frames, frame_meta, s,
                                          layer, kv, G, beta, alpha)
                Qg = np.stack([Qf[layer, s, kv * G + g] for g in range(G)])     # [G, delta, d]
                Ks, Vs = Kf[layer, kv, a:a + L], Vf[layer, kv, a:a + L]
                ref = O.compress_unit(_bits(Qg), _bits(Ks), _bits(Vs), frames_local, beta, alpha)
                lit = O1.compress([[list(map(float, r)) for r in g] for g in Qg],
                                  [list(map(float, r)) for r in Ks], frames_local, O.budget(L, *beta), alpha)
                where = (s, layer, kv)
                assert got["B"] == ref["B"] == O.budget(L, *beta), where
                np.testing.assert_array_equal(got["A"], ref["A"])
                np.testing.assert_allclose(got["A"], lit["A"], rtol=1e-12, atol=0)
                np.testing.assert_allclose(got["phi"], lit["phi"], rtol=1e-12, atol=1e-13)
                assert got["gate"].tolist() == lit["gate"], where
                assert got["kept"].tolist() == lit["kept"], where
                assert (got["kept_abs"] == got["kept"] + a).all() and got["offset"] == a
                np.testing.assert_array_equal(got["k_out"], _bits(Ks[lit["kept"]]))
                np.testing.assert_array_equal(got["v_out"], _bits(Vs[lit["kept"]]))
    # an interleaved head grouping (query head kv + Hkv * g) picks other queries
    Qi = np.stack([Qf[0, 0, kv_g] for kv_g in (1, 1 + Hkv)])
    Qc = np.stack([Qf[0, 0, 1 * G + g] for g in range(G)])
    assert not np.array_equal(Qi, Qc)


# ------------------------------------------------- recompression per step ----

def test_trajectory_cache_hit_rate_average_by_hand():
    """Eq. chr averages the per-step rates over the T steps: hit rates 1/2, 1/3
    and 3/3 average to (1/2 + 1/3 + 1) / 3 = 11/18; a step with an empty oracle
    set (B = 0) is not an evaluation step."""
    rates = [O.cache_hit_rate(np.array([1, 4]), np.array([1, 2])),          # 1 of 2
             O.cache_hit_rate(np.array([0, 5, 9]), np.array([5, 6, 7])),    # 1 of 3
             O.cache_hit_rate(np.array([2, 3, 8]), np.array([2, 3, 8]))]    # 3 of 3
    assert rates == [0.5, 1 / 3, 1.0]
    assert O.trajectory_cache_hit_rate(rates) == pytest.approx(11 / 18, abs=1e-15)
    empty = O.cache_hit_rate(np.array([], int), np.array([], int))
    assert O.trajectory_cache_hit_rate(rates + [empty]) == pytest.approx(11 / 18, abs=1e-15)
    assert math.isnan(O.trajectory_cache_hit_rate([empty]))
    assert O.trajectory_cache_hit_rate([Fraction(1, 4), 0.75]) == 0.5


def _trajectory_fixture(seed=7):
    """A hand-built trajectory: 4 frames of 2 x 3 patches, 3 text tokens after
    each, keys with a frame copied forward (the snap class), per-step window
    queries (G = 2, delta = 3) and decode queries; exact bf16 values."""
    rng = np.random.default_rng(seed)
    d, G, delta, nf, R, C, T = 128, 2, 3, 4, 2, 3, 3
    frames = [(f * (R * C + T), R, C) for f in range(nf)]
    L = nf * (R * C + T)
    coarse = lambda *shape: np.round(rng.standard_normal(shape) * 8) / 64.0
    K, V = coarse(L, d), coarse(L, d)
    K[frames[2][0]:frames[2][0] + 6] = K[frames[1][0]:frames[1][0] + 6]   # frame 2 repeats frame 1
    K[frames[3][0] + 4] = K[frames[0][0] + 1]                             # a patch seen in frame 0 returns
    Qs = coarse(nf, G, delta, d)
    Qd = coarse(nf, G, d)
    ends = [o + R * C + T for o, _, _ in frames]
    return frames, ends, K, V, Qs, Qd, G


def test_recompress_steps_each_step_is_its_own_prefix():
    """Step t is the procedure on the first L_t = (t + 1)(R C + text) rows with
    frames 0..t (frame t current): the same as compress_unit and the literal
    twin on that prefix sliced by hand; its oracle set is the top-B_t of the
    literal decode attention over the prefix, and its rate a plain count."""
    frames, ends, K, V, Qs, Qd, G = _trajectory_fixture()
    beta = (1, 3)
    steps = [0, 1, 2, 3]
    got = O.recompress_steps(_bits(Qs), _bits(Qd), _bits(K), _bits(V), frames, ends, steps, beta)
    rates = []
    for i, t in enumerate(steps):
        L_t = (t + 1) * 9
        assert ends[t] == L_t
        fr = frames[:t + 1]
        ref = O.compress_unit(_bits(Qs[t]), _bits(K[:L_t]), _bits(V[:L_t]), fr, beta)
        g = got["steps"][i]
        assert g["B"] == L_t // 3 == ref["B"]
        np.testing.assert_array_equal(g["kept"], ref["kept"])
        np.testing.assert_array_equal(g["A"], ref["A"])
        lit = O1.compress([[list(map(float, r)) for r in Qs[t, h]] for h in range(G)],
                          [list(map(float, r)) for r in K[:L_t]], fr, L_t // 3)
        assert g["kept"].tolist() == lit["kept"]
        assert g["gate"].tolist() == lit["gate"]
        if t == 0:
            assert (g["gate"] == 1).all(), "a single frame has no history: TSG is a no-op"
        a_lit = O1.decode_scores([list(map(float, Qd[t, h])) for h in range(G)],
                                 [list(map(float, r)) for r in K[:L_t]])
        star = O1.top_b(a_lit, L_t // 3)
        assert g["star"].tolist() == star
        hits = sum(1 for x in star if x in set(lit["kept"]))
        assert g["chr"] == hits / len(star)
        rates.append(hits / len(star))
    assert got["rates"] == rates
    assert got["chr"] == pytest.approx(sum(rates) / len(rates), abs=1e-15)


def test_recompress_steps_packed_batch_equals_single_runs():
    """The steps packed as one varlen batch (sequence i = the prefix of step
    steps[i], frames with absolute offsets) give, through compress_sequence,
    exactly the single-step runs; the last step is the whole trajectory."""
    frames, ends, K, V, Qs, Qd, G = _trajectory_fixture(8)
    beta = (2, 5)
    steps = [1, 3, 2]
    single = O.recompress_steps(_bits(Qs[steps]), _bits(Qd[steps]), _bits(K), _bits(V), frames, ends,
                                steps, beta)
    lens = [ends[t] for t in steps]
    cu_seqlens = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    cu_frames = np.concatenate([[0], np.cumsum([t + 1 for t in steps])]).astype(np.int32)
    frame_meta = np.array([(int(cu_seqlens[i]) + o, r, c) for i, t in enumerate(steps)
                           for (o, r, c) in frames[:t + 1]], np.int32)
    Kp = np.concatenate([K[:n] for n in lens])[None, None]       # [1 layer, 1 kv head, sum L, d]
    Vp = np.concatenate([V[:n] for n in lens])[None, None]
    Qp = Qs[steps][None]                                          # [1 layer, steps, G heads, delta, d]
    for i, t in enumerate(steps):
        got = O.compress_sequence(_bits(Qp), _bits(Kp), _bits(Vp), cu_seqlens, cu_frames, frame_meta, i,
                                  0, 0, G, beta)
        ref = single["steps"][i]
        for key in ("A", "phi", "rho", "gate", "S", "kept", "k_out", "v_out"):
            np.testing.assert_array_equal(got[key], ref[key], err_msg=f"step {t} {key}")
    whole = O.compress_unit(_bits(Qs[3]), _bits(K), _bits(V), frames, beta)
    np.testing.assert_array_equal(single["steps"][1]["kept"], whole["kept"])


# ------------------------------------------------ Mean-Attention prior ----

def test_mean_attention_closed_forms():
    """Pooling of width w = 2r + 1 with zero padding and divisor w: a constant
    c stays c wherever the whole window lies inside the sequence and is
    c (i + r + 1) / w at distance i < r from the start (mirror at the end); a
    single spike becomes a box of height 1/w; width 1 is the identity; mass at
    least r from both ends is preserved; reversing the sequence reverses it."""
    for w in (1, 3, 7, 9):
        r = (w - 1) // 2
        L = 25
        c = 0.375
        got = O.mean_attention(np.full(L, c), w)
        for i in range(L):
            edge = min(i, L - 1 - i)
            want = c if edge >= r else c * (edge + r + 1) / w
            assert got[i] == pytest.approx(want, rel=1e-15), (w, i)
        spike = np.zeros(L)
        spike[12] = 1.0
        box = O.mean_attention(spike, w)
        assert np.array_equal(box, np.where(np.abs(np.arange(L) - 12) <= r, 1.0 / w, 0.0))
        rng = np.random.default_rng(w)
        A = rng.uniform(size=L)
        A[:r] = 0
        A[L - r:] = 0
        assert O.mean_attention(A, w).sum() == pytest.approx(A.sum(), rel=1e-13)
        B = rng.uniform(size=L)
        assert np.allclose(O.mean_attention(B[::-1], w), O.mean_attention(B, w)[::-1], rtol=1e-14, atol=0)
    A = np.random.default_rng(3).uniform(size=11)
    assert np.array_equal(O.mean_attention(A, 1), A)
    for bad in (0, 2, -1):
        with pytest.raises(ValueError):
            O.mean_attention(A, bad)


def test_mean_attention_is_library_zero_padded_box_filter():
    """The definition equals a library routine on every length, including
    sequences shorter than the window: scipy's 1D correlation with a box of
    1/w taps and constant-zero boundaries; and the literal twin."""
    import scipy.ndimage
    rng = np.random.default_rng(17)
    for L in (1, 2, 3, 6, 40):
        A = rng.uniform(size=L) * 1e-3
        for w in (1, 3, 5, 7, 11):
            lib = scipy.ndimage.correlate1d(A, np.full(w, 1.0 / w), mode="constant", cval=0.0)
            np.testing.assert_allclose(O.mean_attention(A, w), lib, rtol=1e-13, atol=1e-300)
            np.testing.assert_allclose(O.mean_attention(A, w), O1.mean_pool(list(A), w), rtol=1e-14, atol=0)


def test_mean_attention_prior_through_the_procedure():
    """compress_unit with the Mean-Attention prior ranks on the pooled A: the
    literal twin (pooling inside its loop version of the procedure) agrees on
    the gate and the kept set, S uses A_mean, and width 1 reproduces the
    window prior exactly."""
    rng = np.random.default_rng(99)
    d, G, delta = 128, 2, 3
    frames = [(3, 2, 3), (12, 2, 3)]
    L = 24
    coarse = lambda *shape: np.round(rng.standard_normal(shape) * 8) / 64.0
    Q, K, V = coarse(G, delta, d), coarse(L, d), coarse(L, d)
    for w in (3, 5):
        got = O.compress_unit(_bits(Q), _bits(K), _bits(V), frames, (1, 3), 1.0, mean_width=w)
        np.testing.assert_allclose(got["A_mean"], O.mean_attention(got["A"], w), rtol=0, atol=0)
        lit = O1.compress([[list(map(float, r)) for r in Q[g]] for g in range(G)],
                          [list(map(float, r)) for r in K], frames, L // 3, 1.0, mean_width=w)
        assert got["kept"].tolist() == lit["kept"]
        np.testing.assert_allclose(got["A_mean"], lit["A"], rtol=1e-12, atol=0)
        vis = got["visual"]
        np.testing.assert_array_equal(got["S"][~vis], got["A_mean"][~vis])
    one = O.compress_unit(_bits(Q), _bits(K), _bits(V), frames, (1, 3), 1.0, mean_width=1)
    plain = O.compress_unit(_bits(Q), _bits(K), _bits(V), frames, (1, 3), 1.0)
    np.testing.assert_array_equal(one["kept"], plain["kept"])
    np.testing.assert_array_equal(one["S"], plain["S"])
