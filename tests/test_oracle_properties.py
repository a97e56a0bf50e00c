"""Property tests of the fp64 oracle (hypothesis): invariants that hold for any
input, each checked against a brute-force or exact-arithmetic restatement.

  budget          B = floor(L * num / den) in exact rationals
  select_topk     |kept| = B, ascending, equal to sorting (float32 S desc, index asc)
  tsg_gate        exactly min(B, |hist|) admitted; every admitted rho (float32) <= every
                  rejected one, and among equal rho the lower index is admitted first;
                  non-historical tokens keep gate 1
  base_score      A >= 0 and sum_i A_i = delta (each softmax row sums to one)
  css_saliency    Phi in [0, 2], 0 on text, invariant to positive rescaling of any key
  decode scores   a distribution over the cache (non-negative, sums to one)
  cache_hit_rate  in [0, 1], 1 for I_keep = I*, symmetric in its arguments when |kept| = |I*|
"""
import math
from fractions import Fraction

import numpy as np
from hypothesis import given, settings, strategies as st

from oracle import stlite_oracle as O

SETTINGS = settings(max_examples=60, deadline=None)


@SETTINGS
@given(st.integers(0, 10 ** 7), st.integers(1, 1000), st.integers(1, 1000))
def test_budget_exact(L, a, b):
    num, den = min(a, b), max(a, b)
    assert O.budget(L, num, den) == math.floor(Fraction(L * num, den))


@SETTINGS
@given(st.lists(st.sampled_from([0.0, 0.25, 0.5, 1.0, 1.0 + 2 ** -30, 3.0, -1.0]), min_size=1, max_size=40),
       st.data())
def test_select_topk_is_sorted_brute_force(S, data):
    S = np.asarray(S)
    B = data.draw(st.integers(0, len(S)))
    kept = O.select_topk(S, B)
    want = sorted(sorted(range(len(S)), key=lambda i: (-float(np.float32(S[i])), i))[:B])
    assert kept.tolist() == want


@SETTINGS
@given(st.integers(1, 30), st.data())
def test_tsg_gate_count_order_and_ties(n_hist, data):
    L = n_hist + data.draw(st.integers(0, 10))
    hist = np.sort(np.asarray(data.draw(st.permutations(range(L))))[:n_hist])
    rho = np.asarray(data.draw(st.lists(st.sampled_from([-0.5, 0.0, 0.3, 0.3 + 1e-9, 0.7, 1.0]),
                                        min_size=n_hist, max_size=n_hist)))
    B = data.draw(st.integers(0, L))
    gate, tau = O.tsg_gate(rho, hist, L, B)
    m = min(B, n_hist)
    assert int(gate[hist].sum()) == m
    others = np.setdiff1d(np.arange(L), hist)
    assert (gate[others] == 1).all()
    r32 = rho.astype(np.float32)
    adm, rej = gate[hist] == 1, gate[hist] == 0
    if adm.any() and rej.any():
        assert r32[adm].max() <= r32[rej].min()
        # equal rho on both sides: the admitted ones have the lower indices
        t = r32[adm].max()
        if (r32[rej] == t).any():
            assert hist[adm & (r32 == t)].max() < hist[rej & (r32 == t)].min()
    if m > 0:
        assert np.float32(tau) == r32[adm].max()
    else:
        assert math.isnan(tau)


@SETTINGS
@given(st.integers(1, 3), st.integers(1, 6), st.integers(8, 40), st.integers(0, 2 ** 31 - 1))
def test_base_score_mass_and_sign(G, delta, L, seed):
    rng = np.random.default_rng(seed)
    d = 16
    Q = rng.standard_normal((G, delta, d)) * rng.uniform(0.1, 4.0)
    K = rng.standard_normal((L, d))
    A = O.base_score(Q, K)
    assert (A >= 0).all()
    assert abs(A.sum() - delta) <= 1e-12 * delta


@SETTINGS
@given(st.integers(1, 6), st.integers(1, 6), st.integers(0, 5), st.integers(0, 2 ** 31 - 1))
def test_css_range_text_and_key_scaling(rows, cols, text, seed):
    rng = np.random.default_rng(seed)
    n = rows * cols
    K = rng.standard_normal((text + n + text, 8))
    frames = [(text, rows, cols)]
    phi = O.css_saliency(K, frames)
    assert (phi >= -1e-15).all() and (phi <= 2 + 1e-15).all()
    assert (phi[:text] == 0).all() and (phi[text + n:] == 0).all()
    K2 = K.copy()
    K2[text:text + n] *= rng.uniform(0.01, 100.0, size=(n, 1))
    np.testing.assert_allclose(O.css_saliency(K2, frames), phi, atol=1e-12)


@SETTINGS
@given(st.integers(1, 4), st.integers(1, 50), st.integers(0, 2 ** 31 - 1))
def test_decode_scores_distribution(G, L, seed):
    rng = np.random.default_rng(seed)
    a = O.decode_attention_scores(rng.standard_normal((G, 16)) * 3, rng.standard_normal((L, 16)))
    assert (a >= 0).all() and abs(a.sum() - 1) <= 1e-12


@SETTINGS
@given(st.integers(1, 60), st.data())
def test_cache_hit_rate_bounds(L, data):
    B = data.draw(st.integers(1, L))
    a = np.sort(np.asarray(data.draw(st.permutations(range(L))))[:B])
    b = np.sort(np.asarray(data.draw(st.permutations(range(L))))[:B])
    r = O.cache_hit_rate(a, b)
    assert 0.0 <= r <= 1.0 and r == O.cache_hit_rate(b, a)
    assert O.cache_hit_rate(a, a) == 1.0
