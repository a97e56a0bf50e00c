"""GPU parity: the HIP pass (through the C ABI) against the fp64 oracle.

Small workloads are compared on every unit; the full-size workloads run the
whole pass in the benchmark's launch configuration and are compared on sampled
(layer, kv head, sequence) units, which the oracle computes one by one.
"""
import dataclasses

import numpy as np
import pytest

from paper_2603_00188_amd import workload as W

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _H():
    from tests import gpu_harness as H
    return H


def test_config0_all_units(torch_cuda):
    H = _H()
    H.log("config 0 (tiny, 912 tokens, 4 units): run")
    case = H.Case(W.config(0))
    res = case.run()
    for kv in range(4):
        st = H.compare_unit(case, res, 0, kv, 0)
        H.log(f"config 0 kv {kv}: {st}")


def test_config1_all_units(torch_cuda):
    H = _H()
    H.log("config 1 (single step, 3392 tokens, 112 units): run")
    case = H.Case(W.config(1))
    res = case.run()
    worst = {}
    for layer in range(28):
        for kv in range(4):
            st = H.compare_unit(case, res, layer, kv, 0)
            for k, v in st.items():
                worst[k] = max(worst.get(k, 0), v)
    H.log(f"config 1 worst: {worst}")
    # single frame: TSG is a no-op, every token eligible
    assert res["gate"].all()


def _small(seqs, G=7, Hkv=2, window=8, beta=(1, 5), layers=2, seed=11, red=None, alpha=1.0,
           element=((1, 2), (1, 3))):
    return W.Workload("small", layers, G * Hkv, Hkv, window, beta, tuple(tuple(s) for s in seqs),
                      red or W.Redundancy(frac=(0.1, 0.3), n_rects=(1, 3)), element, seed=seed, alpha=alpha)


F, T = W.FRAME, W.TEXT
SMALL = {
    # ragged multi-sequence batch: odd grids, text-only and single-frame sequences, a 1x1 frame
    "ragged": _small([[(F, 5, 7), (T, 13), (F, 5, 7), (T, 9), (F, 5, 7), (T, 21)],
                      [(T, 40)],
                      [(F, 3, 1), (T, 5), (F, 1, 1), (T, 3), (F, 4, 9), (T, 70)],
                      [(T, 7), (F, 9, 17), (T, 11)]], window=5),
    # several key tiles and a ragged tail in every kernel
    "tiles": _small([[(F, 12, 21), (T, 37), (F, 12, 21), (T, 37), (F, 12, 21), (T, 150)]],
                    G=4, Hkv=3, window=16, beta=(3, 10)),
    # GQA group of 1 and of 8, window 1 and 64
    "g1w1": _small([[(F, 6, 6), (T, 4), (F, 6, 6), (T, 4)]], G=1, Hkv=4, window=1, beta=(1, 3)),
    "g8w64": _small([[(F, 10, 11), (T, 70), (F, 10, 11), (T, 70)]], G=8, Hkv=1, window=64, beta=(1, 4)),
    # exact duplicate frames (many ties at rho = 1 and at the gate threshold)
    "dups": _small([[(F, 8, 8), (T, 6)] * 5 + [(F, 8, 8), (T, 40)]], beta=(1, 2),
                   red=W.Redundancy(frac=(0.05, 0.1), n_rects=(1, 1), dup_frac=0.6)),
    # budgets at the edges: everything kept, almost nothing kept
    "beta_one": _small([[(F, 4, 5), (T, 10), (F, 4, 5), (T, 10)], [(T, 25)]], beta=(1, 1)),
    "beta_tiny": _small([[(F, 4, 5), (T, 10), (F, 4, 5), (T, 10)], [(T, 25)]], beta=(1, 30)),
    "alpha2": _small([[(F, 7, 9), (T, 20), (F, 7, 9), (T, 20)]], alpha=2.0),
    # window rows over 2, 3, 5 and 6 waves of 32-row blocks, with padding rows in the last block
    "g2w40": _small([[(F, 9, 10), (T, 30), (F, 9, 10), (T, 60)]], G=2, Hkv=2, window=40, layers=1),
    "g3w60": _small([[(F, 9, 10), (T, 30), (F, 9, 10), (T, 90)]], G=3, Hkv=2, window=60, layers=1),
    "g5w60": _small([[(F, 9, 10), (T, 30), (F, 9, 10), (T, 90)]], G=5, Hkv=1, window=60, layers=1),
    "g6w64": _small([[(F, 9, 10), (T, 30), (F, 9, 10), (T, 90)]], G=6, Hkv=1, window=64, layers=1),
    # 14 row blocks (the balanced 8-wave layout, two blocks split by key block between two waves):
    # several key chunks per sequence, a short second sequence, and 28 padding rows in a split block
    "g7w64": _small([[(F, 20, 30), (T, 100)] * 4, [(T, 50), (F, 9, 10), (T, 77)]], G=7, Hkv=1, window=64, layers=1),
    "g7w60": _small([[(F, 20, 30), (T, 100)] * 3, [(F, 5, 6), (T, 300)]], G=7, Hkv=2, window=60, layers=1),
    # 13 row blocks: the only block count that takes the plain 7-wave layout
    "g13w32": _small([[(F, 9, 10), (T, 30), (F, 9, 10), (T, 90)]], G=13, Hkv=1, window=32, layers=1),
    # the largest GQA group decode takes (16, no padded heads) at the largest window-row count (512)
    "g16w32": _small([[(F, 10, 12), (T, 40), (F, 10, 12), (T, 60)], [(T, 20), (F, 6, 7), (T, 35)]],
                     G=16, Hkv=2, window=32, layers=1),
    # more frames in one sequence than the selection kernels keep in LDS (1024)
    "many_frames": _small([[(F, 2, 3), (T, 1)] * 1100 + [(T, 20)]], G=2, Hkv=1, layers=1, beta=(1, 3)),
    # gui screens (flat textured panels and element patches): clusters of close Phi, rho and S values
    # around the gate threshold and the top-B cut, with exact duplicate frames and a second trajectory
    "gui": _small([[(F, 18, 32), (T, 40)] * 5, [(F, 12, 20), (T, 30)] * 3], G=7, Hkv=2, window=32,
                  beta=(1, 4), red=W.Redundancy(frac=(0.05, 0.2), n_rects=(1, 4), dup_frac=0.3),
                  element=((1, 3), (2, 4))).with_screen("gui"),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_small_all_units(torch_cuda, name):
    H = _H()
    w = SMALL[name]
    H.log(f"small {name}: L={w.total_tokens} seqs={len(w.seqs)} G={w.group} window={w.window}")
    case = H.Case(w)
    res = case.run()
    for layer in range(w.n_layers):
        for kv in range(w.n_kv_heads):
            for s in range(case.lay.n_seqs):
                H.compare_unit(case, res, layer, kv, s)


def test_zero_keys_and_snapkv_mode(torch_cuda):
    """Zero key rows (cosine 0 by convention) and the SnapKV special case
    (no CSS term, no gate) against the oracle with the same switches."""
    H = _H()
    w = SMALL["ragged"]
    case = H.Case(w)
    for off, r, c in case.lay.frame_meta[:3]:
        case.k[:, :, off + 1] = 0          # one zero key in each of the first frames
    case.k[:, :, int(case.lay.frame_meta[-1][0]) + 2] = 0
    import torch
    case.dk.copy_(torch.from_numpy(case.k.view(np.int16)))
    res = case.run()
    for layer in range(w.n_layers):
        for kv in range(w.n_kv_heads):
            for s in range(case.lay.n_seqs):
                H.compare_unit(case, res, layer, kv, s)
    res = case.run(alpha=0.0, css=False, tsg=False)
    for layer in range(w.n_layers):
        for kv in range(w.n_kv_heads):
            for s in range(case.lay.n_seqs):
                H.compare_unit(case, res, layer, kv, s, css=False, tsg=False)


def test_stage_threshold_and_select_exact(torch_cuda):
    """Stage-isolated: gate and top-B fed with the oracle's own (fp32-rounded)
    rho, A, Phi must reproduce the oracle's integer decisions exactly."""
    import torch
    H = _H()
    from oracle import stlite_oracle as O
    from paper_2603_00188_amd import stlite as S
    w = SMALL["dups"]
    case = H.Case(w)
    U, L = case.prob.units, case.prob.total_tokens
    rho = np.zeros((U, L), np.float32)
    A = np.zeros((U, L), np.float32)
    phi = np.zeros((U, L), np.float32)
    refs = {}
    for layer in range(w.n_layers):
        for kv in range(w.n_kv_heads):
            u = layer * w.n_kv_heads + kv
            for s in range(case.lay.n_seqs):
                r = case.oracle(layer, kv, s)
                a = int(case.lay.cu_seqlens[s])
                rho[u, a + r["hist"]] = r["rho"]
                A[u, a:a + len(r["A"])] = r["A"]
                phi[u, a:a + len(r["A"])] = r["phi"]
                refs[(u, s)] = r
    dev = lambda x: torch.from_numpy(x).cuda()
    drho, dA, dphi = dev(rho), dev(A), dev(phi)
    out = case.out
    S.stlite_tsg_threshold(case.prob, drho, out.tau, out.gate, out.ws_tsg)
    torch.cuda.synchronize()
    gate = out.gate.cpu().numpy()
    for (u, s), r in refs.items():
        a, b = int(case.lay.cu_seqlens[s]), int(case.lay.cu_seqlens[s + 1])
        g_ref, tau_ref = O.tsg_gate(rho[u, a:b][r["hist"]].astype(np.float64), r["hist"], b - a, r["B"])
        assert (gate[u, a:b] == g_ref).all(), (u, s)
    S.stlite_select_topk(case.prob, dA, dphi, out.gate, 1.0, out.kept, out.score, out.ws)
    torch.cuda.synchronize()
    kept = out.kept.cpu().numpy()
    score = out.score.cpu().numpy()
    for (u, s), r in refs.items():
        a, b = int(case.lay.cu_seqlens[s]), int(case.lay.cu_seqlens[s + 1])
        g = gate[u, a:b]
        s32 = np.where(r["visual"], np.where(g > 0, A[u, a:b] + phi[u, a:b], np.float32(0)), A[u, a:b])
        assert (score[u, a:b] == s32).all(), (u, s)
        want = O.select_topk(s32.astype(np.float64), r["B"]) + a
        cb = case.cu_budget
        assert (kept[u, cb[s]:cb[s + 1]] == want).all(), (u, s)


# Layouts of the stage-exact selection tests: (frames, (rows, cols), text) per sequence.
STAGE_LAYOUTS = {
    # segments of 27,300 and 5,935 tokens: one work-group per segment keeps them on chip
    "short": ((13, (40, 50), 100), (5, (30, 37), 77)),
    # a 168,000-token segment, longer than the on-chip selection holds: every
    # segment of the call takes the splitter selection by default
    "long": ((80, (40, 50), 100), (5, (30, 37), 77)),
    # a 336,000-token segment: about 9.7 % of it (32,600 keys at beta = 1/5, more at 1/2) lies
    # between the splitters, more than one resolving batch (24,576), so resolve reloads the
    # candidate list batch by batch
    "huge": ((160, (40, 50), 100), (5, (30, 37), 77)),
    # a 1,050,000-token segment: more tiles (4,102) than resolve counts in LDS (4,096), so the
    # taken counts per tile go through global atomics
    "giant": ((500, (40, 50), 100), (5, (30, 37), 77)),
}

# (layout, selection path forced through STLITE_SELECT_PATH; None = the default)
STAGE_CASES = [("short", None), ("long", None), ("long", "four_pass"), ("long", "split_exact"),
               ("short", "split"), ("short", "split_exact"), ("short", "four_pass"),
               ("huge", None), ("huge", "split_exact"), ("giant", None)]


@pytest.mark.parametrize("layout,path", STAGE_CASES)
@pytest.mark.parametrize("values", ["few", "many", "spread"])
def test_stage_exact_many_parts_and_ties(torch_cuda, monkeypatch, layout, path, values):
    """Stage-isolated on long sequences, with inputs drawn from a few values
    (long runs of equal keys straddling wave, tile and part boundaries; the
    splitters land on tied keys), from a few hundred (the k-th key among the
    splitter candidates, with hundreds of ties there) or from a few thousand
    (tens of ties at the k-th key): gate, tau, S and kept lists must equal the
    oracle's exactly, on every selection path."""
    import torch
    from oracle import stlite_oracle as O
    from paper_2603_00188_amd import stlite as S
    if path:
        monkeypatch.setenv("STLITE_SELECT_PATH", path)
    seqs, metas, cu = [], [], [0]
    for nf, (r, c), nt in STAGE_LAYOUTS[layout]:
        off = cu[-1]
        fm = []
        for _ in range(nf):
            fm.append((off, r, c))
            off += r * c + nt
        metas.append(fm)
        cu.append(off)
    cu_seqlens = np.array(cu, np.int32)
    cu_frames = np.array([0, len(metas[0]), len(metas[0]) + len(metas[1])], np.int32)
    frame_meta = np.array(metas[0] + metas[1], np.int32)
    n_layers, hkv = 1, 2
    for beta in ((1, 5), (1, 2)):
        cu_budget = S.budgets(cu_seqlens, *beta)
        prob = S.Problem(n_layers, hkv, hkv, 8, cu_seqlens, cu_frames, frame_meta, cu_budget)
        U, L = prob.units, prob.total_tokens
        rng = np.random.default_rng(5)
        if values == "few":
            rho = rng.choice(np.float32([0.1, 0.25, 0.5, 0.75, 1.0]), size=(U, L)).astype(np.float32)
            A = rng.choice(np.float32([1e-4, 2e-4, 5e-4]), size=(U, L)).astype(np.float32)
            phi = rng.choice(np.float32([0.9, 1.0, 1.1]), size=(U, L)).astype(np.float32)
        elif values == "spread":
            rho = rng.choice(np.linspace(0.2, 0.4, 2000, dtype=np.float32), size=(U, L)).astype(np.float32)
            A = rng.choice(np.linspace(1e-4, 5e-4, 1500, dtype=np.float32), size=(U, L)).astype(np.float32)
            phi = rng.choice(np.linspace(0.9, 1.1, 1700, dtype=np.float32), size=(U, L)).astype(np.float32)
        else:
            rho = rng.choice(np.linspace(0.2, 0.4, 300, dtype=np.float32), size=(U, L)).astype(np.float32)
            A = rng.choice(np.linspace(1e-4, 5e-4, 200, dtype=np.float32), size=(U, L)).astype(np.float32)
            phi = rng.choice(np.linspace(0.9, 1.1, 250, dtype=np.float32), size=(U, L)).astype(np.float32)
        out = S.Buffers(prob)
        dev = lambda x: torch.from_numpy(x).cuda()
        S.stlite_tsg_threshold(prob, dev(rho), out.tau, out.gate, out.ws_tsg)
        S.stlite_select_topk(prob, dev(A), dev(phi), out.gate, 1.0, out.kept, out.score, out.ws)
        torch.cuda.synchronize()
        gate, tau, kept = out.gate.cpu().numpy(), out.tau.cpu().numpy(), out.kept.cpu().numpy()
        score = out.score.cpu().numpy()
        for u in range(U):
            for s in range(2):
                a, b = int(cu_seqlens[s]), int(cu_seqlens[s + 1])
                fm = metas[s]
                vis = np.zeros(b - a, bool)
                for off, r, c in fm:
                    vis[off - a:off - a + r * c] = True
                hist = np.concatenate([np.arange(off - a, off - a + r * c) for off, r, c in fm[:-1]])
                B = int(cu_budget[s + 1] - cu_budget[s])
                g_ref, tau_ref = O.tsg_gate(rho[u, a:b][hist].astype(np.float64), hist, b - a, B)
                assert (gate[u, a:b] == g_ref).all(), (beta, u, s)
                assert np.float32(tau[u, s]) == np.float32(tau_ref), (beta, u, s)
                s32 = np.where(vis, np.where(g_ref > 0, A[u, a:b] + phi[u, a:b], np.float32(0)), A[u, a:b])
                assert np.array_equal(score[u, a:b], s32), (beta, u, s)
                want = O.select_topk(s32.astype(np.float64), B) + a
                assert (kept[u, cu_budget[s]:cu_budget[s + 1]] == want).all(), (beta, u, s)


@pytest.mark.parametrize("path", [None, "split", "split_exact", "four_pass"])
def test_stage_tie_group_covers_sample_band(torch_cuda, monkeypatch, path):
    """A tie group holding most of a long segment and the k-th key: the
    gate's rho equal to 0.5 on 95 % of the history, and the top-B's S = 0 on
    every historical token (the gate passed in is all zeros there), with B
    above the count of positive scores.  The splitters drawn from such a
    sample fall on the same key; gate, tau and kept lists must still equal
    the oracle's exactly."""
    import torch
    from oracle import stlite_oracle as O
    from paper_2603_00188_amd import stlite as S
    if path:
        monkeypatch.setenv("STLITE_SELECT_PATH", path)
    nf, (r, c), nt = 80, (40, 50), 100
    fm, off = [], 0
    for _ in range(nf):
        fm.append((off, r, c))
        off += r * c + nt
    cu_seqlens = np.array([0, off], np.int32)
    cu_frames = np.array([0, nf], np.int32)
    frame_meta = np.array(fm, np.int32)
    cu_budget = S.budgets(cu_seqlens, 1, 5)
    prob = S.Problem(1, 2, 2, 8, cu_seqlens, cu_frames, frame_meta, cu_budget)
    U, L = prob.units, prob.total_tokens
    B = int(cu_budget[1])
    vis = np.zeros(L, bool)
    for o, rr, cc in fm:
        vis[o:o + rr * cc] = True
    hist = np.concatenate([np.arange(o, o + rr * cc) for o, rr, cc in fm[:-1]])
    rng = np.random.default_rng(9)
    rho = np.zeros((U, L), np.float32)
    rho[:, hist] = np.where(rng.random((U, len(hist))) < 0.95, np.float32(0.5),
                            rng.uniform(0.0, 1.0, (U, len(hist))).astype(np.float32))
    A = rng.uniform(1e-5, 1e-3, (U, L)).astype(np.float32)
    phi = rng.uniform(0.5, 1.5, (U, L)).astype(np.float32)
    gate_in = np.ones((U, L), np.uint8)
    gate_in[:, hist] = 0
    out = S.Buffers(prob)
    dev = lambda x: torch.from_numpy(x).cuda()
    S.stlite_tsg_threshold(prob, dev(rho), out.tau, out.gate, out.ws_tsg)
    S.stlite_select_topk(prob, dev(A), dev(phi), dev(gate_in), 1.0, out.kept, out.score, out.ws)
    torch.cuda.synchronize()
    gate, tau, kept = out.gate.cpu().numpy(), out.tau.cpu().numpy(), out.kept.cpu().numpy()
    n_pos = int(np.count_nonzero(~vis)) + int(fm[-1][1] * fm[-1][2])
    assert B > n_pos  # the k-th largest S is one of the zeros
    for u in range(U):
        g_ref, tau_ref = O.tsg_gate(rho[u][hist].astype(np.float64), hist, L, B)
        assert (gate[u] == g_ref).all(), u
        assert np.float32(tau[u, 0]) == np.float32(tau_ref), u
        s32 = np.where(vis, np.where(gate_in[u] > 0, A[u] + phi[u], np.float32(0)), A[u])
        want = O.select_topk(s32.astype(np.float64), B)
        assert (kept[u, :B] == want).all(), u


@pytest.mark.parametrize("path", ["four_pass", "split", "split_exact"])
def test_selection_paths_agree(torch_cuda, monkeypatch, path):
    """The whole pass on the small cases (ragged batches, sequences shorter
    than a tile, a 1 x 1 frame, a zero budget) under each forced selection
    path gives the same bits as under the default path."""
    H = _H()
    for name in ("ragged", "tiles", "dups", "beta_tiny"):
        case = H.Case(SMALL[name])
        monkeypatch.delenv("STLITE_SELECT_PATH", raising=False)
        ref = case.run()
        monkeypatch.setenv("STLITE_SELECT_PATH", path)
        got = case.run()
        for key in ("gate", "tau", "kept", "score", "k_out", "v_out"):
            assert np.array_equal(got[key], ref[key], equal_nan=True), (name, path, key)


@pytest.mark.parametrize("path", [None, "split"])
@pytest.mark.parametrize("css, tsg", [(True, False), (False, True)], ids=["css_only", "tsg_only"])
def test_component_ablations(torch_cuda, monkeypatch, path, css, tsg):
    """The one-component variants of the procedure: CSS without the gate
    (every visual token admitted, the top-B reads Phi and no gate) and the
    gate without CSS (no Phi term, the top-B reads the gate and no Phi),
    against the oracle with the same switches, under the default and the
    splitter selection."""
    H = _H()
    if path:
        monkeypatch.setenv("STLITE_SELECT_PATH", path)
    else:
        monkeypatch.delenv("STLITE_SELECT_PATH", raising=False)
    for name in ("ragged", "dups", "gui"):
        w = SMALL[name]
        case = H.Case(w)
        res = case.run(css=css, tsg=tsg)
        for layer in range(w.n_layers):
            for kv in range(w.n_kv_heads):
                for s in range(case.lay.n_seqs):
                    H.compare_unit(case, res, layer, kv, s, css=css, tsg=tsg)


def test_split_tsg_matches_fused(torch_cuda):
    """stlite_tsg_rho followed by stlite_tsg_threshold reproduces stlite_tsg_gate
    bit for bit (rho, gate and tau)."""
    import torch
    H = _H()
    from paper_2603_00188_amd import stlite as S
    for name in ("ragged", "dups", "beta_tiny"):
        case = H.Case(SMALL[name])
        out = case.out
        S.stlite_tsg_gate(case.prob, case.dk, out.rho, out.tau, out.gate, out.ws_tsg)
        torch.cuda.synchronize()
        fused = (out.rho.cpu().numpy(), out.gate.cpu().numpy(), out.tau.cpu().numpy())
        out.rho.fill_(7.0)
        out.gate.fill_(9)
        out.tau.fill_(7.0)
        S.stlite_tsg_rho(case.prob, case.dk, out.rho, out.ws_tsg)
        S.stlite_tsg_threshold(case.prob, out.rho, out.tau, out.gate, out.ws_tsg)
        torch.cuda.synchronize()
        split = (out.rho.cpu().numpy(), out.gate.cpu().numpy(), out.tau.cpu().numpy())
        for a, b in zip(fused, split):
            assert np.array_equal(a, b, equal_nan=True), name


def test_overlapped_streams_match_serial(torch_cuda):
    """compress() with score, TSG and CSS on three concurrent streams gives
    the same bits as the serial pass."""
    H = _H()
    case = H.Case(SMALL["ragged"])
    r1 = case.run()
    r2 = case.run(overlap=True)
    for k in r1:
        assert np.array_equal(r1[k], r2[k], equal_nan=True), k


def test_determinism(torch_cuda):
    H = _H()
    case = H.Case(SMALL["tiles"])
    r1 = case.run()
    r2 = case.run()
    for k in r1:
        assert np.array_equal(r1[k], r2[k], equal_nan=True), k


def _full(idx, beta=None, samples=((0, 0, 0), (27, 3, 0)), screen="iid"):
    H = _H()
    w = W.config(idx, beta).with_screen(screen)
    H.log(f"config {idx} {w.name}: generate L={w.total_tokens} x {w.n_layers} layers")
    case = H.Case(w)
    H.log(f"config {idx}: run")
    res = case.run()
    for (layer, kv, s) in samples:
        st = H.compare_unit(case, res, layer, kv, s)
        H.log(f"config {idx} beta {w.beta} unit ({layer},{kv},{s}): {st}")
    return case, res


@pytest.mark.timeout(900)
def test_config2_sampled(torch_cuda):
    H = _H()
    case, res = _full(2, (1, 5), samples=((3, 1, 0), (20, 3, 0)))
    for beta, units in (((1, 10), ((14, 2), (27, 0))), ((2, 5), ((14, 2), (0, 3)))):
        import dataclasses as dc
        w = dc.replace(case.w, beta=beta)
        case2 = H.Case.__new__(H.Case)
        case2.__dict__.update(case.__dict__)
        case2.w = w
        from paper_2603_00188_amd import stlite as S
        case2.cu_budget = S.budgets(case.lay.cu_seqlens, *beta)
        case2.prob = S.Problem(case.n_layers, w.n_q_heads, w.n_kv_heads, w.window, case.lay.cu_seqlens,
                               case.lay.cu_frames, case.lay.frame_meta, case2.cu_budget)
        case2.out = S.Buffers(case2.prob)
        res2 = case2.run()
        for layer, kv in units:
            st = H.compare_unit(case2, res2, layer, kv, 0)
            H.log(f"config 2 beta {beta} unit ({layer},{kv},0): {st}")


@pytest.mark.timeout(900)
def test_config2_gui_sampled(torch_cuda):
    """The long-horizon workload (62,720 tokens) on gui screens, in the
    benchmark's launch configuration."""
    _full(2, samples=((0, 0, 0), (13, 2, 0), (27, 3, 0)), screen="gui")


@pytest.mark.timeout(900)
def test_config3_sampled(torch_cuda):
    """The 150,528-token trajectory in the benchmark's launch configuration,
    and decode attention over its full and compacted caches."""
    H = _H()
    # first, last and middle layers; every kv head twice
    samples = ((0, 0, 0), (4, 1, 0), (9, 2, 0), (13, 3, 0), (14, 0, 0), (18, 1, 0), (23, 2, 0), (27, 3, 0))
    case, res = _full(3, samples=samples)
    dec = H.run_decode(case)
    for unit in samples:
        H.log(f"config 3 decode unit {unit}: worst error / tolerance {H.compare_decode(case, res, dec, *unit):.3g}")


@pytest.mark.timeout(900)
def test_config4_sampled(torch_cuda):
    """The ragged batch of 8 trajectories, and decode attention over its caches."""
    H = _H()
    # four units spread over layers and kv heads, each compared on all 8 sequences
    samples = tuple((layer, kv, s) for layer, kv in ((0, 0), (7, 1), (13, 2), (27, 3)) for s in range(8))
    case, res = _full(4, samples=samples)
    dec = H.run_decode(case)
    for unit in samples:
        H.log(f"config 4 decode unit {unit}: worst error / tolerance {H.compare_decode(case, res, dec, *unit):.3g}")


# Spike workloads: (workload, query head of kv head 0 that the spike aligns with).  g7w64 has 14
# row blocks (the balanced 8-wave layout); head 6's rows 384..447 form blocks 12 and 13, each
# split by key block between two waves.
SPIKE_CASES = {
    "g4w16": (lambda: _small([[(F, 12, 21), (T, 37), (F, 12, 21), (T, 37), (F, 12, 21), (T, 150)]],
                             G=4, Hkv=3, window=16, beta=(3, 10), layers=1), 0),
    "g7w64": (lambda: _small([[(F, 20, 30), (T, 100)] * 4], G=7, Hkv=1, window=64, beta=(3, 10), layers=1), 6),
}
# The exact pass at the other wave layouts: one 32-row block (1 wave), 6 blocks (3 waves) and
# 13 blocks (the plain 7-wave layout); key chunks of >= 1024 keys keep the spike keys
# 200, 460 and 700 out of the first tile of their chunk.
SPIKE_LAYOUTS = dict(SPIKE_CASES, **{
    "g1w1": (lambda: _small([[(F, 20, 30), (T, 100)] * 2], G=1, Hkv=2, window=1, beta=(3, 10), layers=1), 0),
    "g3w60": (lambda: _small([[(F, 20, 30), (T, 100)] * 2], G=3, Hkv=1, window=60, beta=(3, 10), layers=1), 2),
    "g13w32": (lambda: _small([[(F, 20, 30), (T, 100)] * 2], G=13, Hkv=1, window=32, beta=(3, 10), layers=1), 12),
})


@pytest.mark.parametrize("name", list(SPIKE_LAYOUTS))
def test_logit_spike_takes_exact_pass(torch_cuda, name):
    """Keys aligned with a window query, far into a chunk, push that query's
    logits about 150 log2 units above the chunk's first tile, so that the lean
    first pass's fp32 sums overflow: it flags those chunks and the exact pass
    recomputes them."""
    import torch
    H = _H()
    from oracle import stlite_oracle as O
    from paper_2603_00188_amd import workload as W2
    make, head = SPIKE_LAYOUTS[name]
    w = make()
    case = H.Case(w)
    q = O.bf16_to_f64(case.q[0, 0, head, 0])        # window position 0 of the head
    unit_dir = q / np.linalg.norm(q)
    spike = W2.to_bf16_bits((700.0 * unit_dir).astype(np.float32))
    for j in (200, 460, 700):                       # not in the first tile of their chunk; both key blocks
        case.k[0, 0, j] = spike
    case.dk.copy_(torch.from_numpy(case.k.view(np.int16)))
    res = case.run()
    for kv in range(w.n_kv_heads):
        H.compare_unit(case, res, 0, kv, 0)
    A = res["a_base"][0]
    med = float(np.median(A[: int(case.lay.cu_seqlens[1])]))
    assert A[200] > 100 * med and A[460] > 100 * med, "spike keys should carry most of the head's window mass"


@pytest.mark.parametrize("name", list(SPIKE_CASES))
def test_logit_spike_in_first_tile_takes_exact_pass(torch_cuda, name):
    """A key aligned with one window query, inside the first tile of its chunk,
    lifts the lean first pass's offset of that query's group of eight rows
    about 150 log2 units above the other seven rows' logits: their sums
    underflow, the chunk is flagged and the exact pass recomputes it."""
    import torch
    H = _H()
    from oracle import stlite_oracle as O
    from paper_2603_00188_amd import workload as W2
    make, head = SPIKE_CASES[name]
    w = make()
    case = H.Case(w)
    q = O.bf16_to_f64(case.q[0, 0, head, 3])        # window position 3 of the head
    unit_dir = q / np.linalg.norm(q)
    spike = W2.to_bf16_bits((700.0 * unit_dir).astype(np.float32))
    for j in ((10, 270) if name == "g4w16" else (10, 1034)):  # first tile of chunks 0 and 1
        case.k[0, 0, j] = spike
    case.dk.copy_(torch.from_numpy(case.k.view(np.int16)))
    res = case.run()
    for kv in range(w.n_kv_heads):
        H.compare_unit(case, res, 0, kv, 0)
