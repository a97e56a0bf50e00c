"""The seeded input generator: layouts of the five workloads, determinism, and
the redundancy structure the generator promises."""
import numpy as np

from paper_2603_00188_amd import workload as W


def test_layout_sizes():
    want = {0: (912, 3), 1: (3392, 1), 2: (62720, 20), 3: (150528, 48)}
    for i, (L, F) in want.items():
        lay = W.make_layout(W.config(i))
        assert lay.total_tokens == L and len(lay.frame_meta) == F
        assert lay.cu_seqlens.tolist() == [0, L]
    lay4 = W.make_layout(W.config(4))
    assert lay4.n_seqs == 8
    for s in range(8):
        nf = lay4.cu_frames[s + 1] - lay4.cu_frames[s]
        assert 6 <= nf <= 24
        fm = lay4.seq_frames(s)
        assert (fm[:, 0] >= lay4.cu_seqlens[s]).all()
        assert (fm[:, 0] + fm[:, 1] * fm[:, 2] <= lay4.cu_seqlens[s + 1]).all()


def test_deterministic_and_layer_regeneration():
    w = W.config(0)
    s1, k1, v1, q1 = W.make_inputs(w)
    s2, k2, v2, q2 = W.make_inputs(w)
    assert (k1 == k2).all() and (v1 == v2).all() and (q1 == q2).all()
    w2 = W.config(1).with_layers(3)
    _, k, v, q = W.make_inputs(w2)
    _, k1, v1, q1 = W.make_inputs(w2, layers=[2])
    assert (k[2] == k1[0]).all() and (v[2] == v1[0]).all() and (q[2] == q1[0]).all()


def test_redundancy_structure():
    w = W.config(3).with_layers(1)
    scene = W.make_scene(w)
    assert sum(scene.duplicate) == round(0.3 * 48)
    for f in range(1, 48):
        same = (scene.frame_emb[f] == scene.frame_emb[f - 1]).all(axis=1).mean()
        if scene.duplicate[f]:
            assert same == 1.0
        else:
            assert 0.6 < same < 0.999
    # config 0: two 2x3 rectangles resampled per transition
    sc0 = W.make_scene(W.config(0))
    for f in (1, 2):
        changed = (~(sc0.frame_emb[f] == sc0.frame_emb[f - 1]).all(axis=1)).sum()
        assert 6 <= changed <= 12


def test_bf16_rounding_is_rne():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(100000).astype(np.float32)
    ties = ((np.arange(512, dtype=np.uint32) + 0x3F00) << 16) | 0x8000
    x[:512] = ties.view(np.float32)
    got = W.to_bf16_bits(x)
    assert (got == W.to_bf16_bits_reference(x)).all()
    # ties go to the even mantissa
    assert (got[:512] & 1 == 0).all()
    back = W.bf16_bits_to_f32(got)
    assert (np.abs(back - x) <= np.abs(x) * 2.0 ** -8).all()


def test_step_inputs_are_prefixes_of_the_trajectory():
    """Sequence i of the per-step batch is the trajectory's first L_t rows
    (frames 0..t and the text after each), frame t is its current frame, and
    the draws are deterministic and per step (a step regenerates alone); anchors lie on patches that changed between
    their frame and the step's current frame."""
    w = W.config(0)
    base = W.make_inputs(w)
    si = W.make_step_inputs(w, base=base)
    scene, kb, vb, _ = base
    fm0 = scene.layout.seq_frames(0)
    assert si.steps == [0, 1, 2]
    ends = list(fm0[1:, 0]) + [scene.layout.total_tokens]
    assert list(np.diff(si.layout.cu_seqlens)) == ends
    for i, t in enumerate(si.steps):
        a, n = int(si.layout.cu_seqlens[i]), ends[t]
        assert np.array_equal(si.k[:, :, a:a + n], kb[:, :, :n])
        assert np.array_equal(si.v[:, :, a:a + n], vb[:, :, :n])
        fr = si.layout.seq_frames(i)
        assert len(fr) == t + 1
        assert np.array_equal(fr[:, 0] - a, fm0[:t + 1, 0]) and np.array_equal(fr[:, 1:], fm0[:t + 1, 1:])
        if si.anchor[i] is not None:
            f, u0, v0, h, ww = si.anchor[i]
            assert f < t
            c = int(fm0[f, 2])
            cells = [(u0 + x) * c + (v0 + y) for x in range(h) for y in range(ww)]
            ef, et = scene.frame_emb[f][cells], scene.frame_emb[t][cells]
            assert (ef != et).any(axis=1).any(), "the anchor shows content the current frame lost"
    assert si.anchor[0] is None
    again = W.make_step_inputs(w, base=base)
    assert np.array_equal(si.q, again.q) and np.array_equal(si.q_dec, again.q_dec)
    # the decode query is not one of the window queries
    for i in range(len(si.steps)):
        for g in range(w.n_q_heads):
            assert not (si.q[0, i, g] == si.q_dec[0, i, g][None, :]).all(axis=1).any()
    sub = W.make_step_inputs(w, steps=[2, 0], base=base)
    assert np.array_equal(sub.q[:, 0], si.q[:, 2]) and np.array_equal(sub.q_dec[:, 1], si.q_dec[:, 0])
    assert list(np.diff(sub.layout.cu_seqlens)) == [ends[2], ends[0]]
