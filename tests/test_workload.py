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


def _centre(rect):
    u0, v0, h, ww = rect
    return u0 + h // 2, v0 + ww // 2


def test_gui_screen_structure():
    """The gui screen model: the same layout as the named workload, flat
    textured panels (neighbouring background patches of one panel have cosine
    about 1 / (1 + (1/3)^2) = 0.9), independent element patches over about a
    quarter of the screen, transitions that keep every other patch, a query
    target centred on an element patch, and CSS saliency (the oracle's, Eq.
    css_calc) that tells elements from background."""
    from oracle import stlite_oracle as O
    w = W.config(2).with_layers(1)
    g = w.with_screen("gui")
    assert w.screen == "iid" and g.name == "long_horizon_gui"
    assert W.make_scene(w).content is None
    sc, k, _, _ = W.make_inputs(g)
    lay = sc.layout
    assert np.array_equal(lay.frame_meta, W.make_layout(w).frame_meta)
    assert len(sc.content) == len(lay.frame_meta)
    for f, (off, r, c) in enumerate(lay.frame_meta):
        ct = sc.content[f].reshape(r, c)
        assert 0.12 < ct.mean() < 0.35
        e = sc.frame_emb[f].reshape(r, c, -1)
        cs = (e[:, :-1] * e[:, 1:]).sum(-1) / (np.linalg.norm(e[:, :-1], axis=-1) * np.linalg.norm(e[:, 1:], axis=-1))
        pan = W.gui_panels(r, c)
        bg = ~ct[:, :-1] & ~ct[:, 1:] & (pan[:, :-1] == pan[:, 1:])
        el = ct[:, :-1] & ct[:, 1:]
        assert 0.85 < cs[bg].mean() < 0.95
        assert abs(cs[el].mean()) < 0.15
        if f:
            same = (sc.frame_emb[f] == sc.frame_emb[f - 1]).all(axis=1)
            assert np.array_equal(sc.content[f][same], sc.content[f - 1][same])
            assert 0.6 < same.mean() < 0.999
    off, r, c = (int(x) for x in lay.frame_meta[-1])
    u, v = _centre(sc.element[0])
    assert sc.content[-1].reshape(r, c)[u, v]
    phi = O.css_frame(O.bf16_to_f64(k[0, 0, off:off + r * c]), r, c)
    ct = sc.content[-1]
    assert phi[ct].mean() > 0.9 and phi[~ct].mean() < 0.45


def test_gui_step_targets_and_anchors():
    """Per-step inputs on gui screens: each step's element is centred on an
    element patch of its current frame, and each anchor on an element patch of
    the earlier frame that the current frame has changed."""
    w = W.config(3).with_layers(1).with_screen("gui")
    si = W.make_step_inputs(w, steps=[0, 3, 20, 47], pack=False)
    scene = W.make_scene(w)
    fm = scene.layout.seq_frames(0)
    n_anchor = 0
    for i, t in enumerate(si.steps):
        r, c = int(fm[t, 1]), int(fm[t, 2])
        u, v = _centre(si.element[i])
        assert scene.content[t].reshape(r, c)[u, v]
        if si.anchor[i] is not None:
            f, u0, v0, h, ww = si.anchor[i]
            p = (u0 + h // 2) * c + (v0 + ww // 2)
            assert f < t and scene.content[f][p]
            assert (scene.frame_emb[f][p] != scene.frame_emb[t][p]).any()
            n_anchor += 1
    assert n_anchor >= 2
