"""GPU parity of the TSG variants of the paper's ablations against the fp64
oracle: the dot-product and negative-L2 similarities (similarity-metric
ablation) and the fixed-threshold gate (component-necessity controls), all
through the C ABI.

Tolerances (bf16 keys, exact bf16 products, 128-term fp32 sums with
gamma_128 = 128 * 2^-24 ~ 7.6e-6):
  cosine      the same bits as stlite_tsg_rho
  dot         |d| <= 1e-5 ||k_i|| max_j ||k_j||: each candidate's error is at
              most gamma_128 sum_c |k_ic k_jc| <= gamma_128 ||k_i|| ||k_j||, and
              a max of values each within e is within e
  neg_l2      compared as squared distances, |rho_gpu^2 - rho_ref^2| <= e2 with
              e2 = 3e-5 (||k_i||^2 + max_j ||k_j||^2) (the product error above
              twice, two fp32 sums of squares, three roundings); where the
              unsnapped squared distance lies within e2 of the snap edge
              1e-5 ||k_i||^2, either side of the snap is accepted
  fixed gate  bit-exact against the oracle's fixed gate on the GPU's rho (both
              decide float32 rho <= float32 tau); against the oracle's own rho
              it may differ only where |rho_ref - tau| <= 1e-3 max(|rho_ref|, 1e-2)
  adaptive gate on a variant rho: bit-exact (gate and tau) against the
              oracle's gate on the GPU's rho
"""
import numpy as np
import pytest

from paper_2603_00188_amd import workload as W

pytestmark = pytest.mark.gpu

DOT_TOL = 1e-5
L2_TOL = 3e-5
SIMS = {"cosine": 0, "dot": 1, "neg_l2": 2}


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _mods():
    from oracle import stlite_oracle as O
    from paper_2603_00188_amd import stlite as S
    from tests import gpu_harness as H
    from tests.test_gpu_parity import SMALL
    return O, S, H, SMALL


def _units(case):
    """(unit, layer, kv, seq, token offset, L_s, hist, cur) of every unit and sequence."""
    O = _mods()[0]
    lay = case.lay
    for layer in range(case.n_layers):
        for kv in range(case.w.n_kv_heads):
            u = layer * case.w.n_kv_heads + kv
            for s in range(lay.n_seqs):
                a, b = int(lay.cu_seqlens[s]), int(lay.cu_seqlens[s + 1])
                frames = O.seq_frames_local(lay.cu_seqlens, lay.cu_frames, lay.frame_meta, s)
                hist, cur, _ = O.split_tokens(b - a, frames)
                yield u, layer, kv, s, a, b - a, hist, cur


def _similarity(case, sim):
    import torch
    S = _mods()[1]
    rho = torch.full((case.prob.units, case.prob.total_tokens), 7.0, dtype=torch.float32, device="cuda")
    S.stlite_tsg_similarity(case.prob, SIMS[sim], case.dk, rho, case.out.ws_tsg)
    torch.cuda.synchronize()
    return rho


def check_similarity(case, rho_gpu, sim, layer, kv, s, rows=None):
    """Compare rho of one unit and sequence (or of the listed historical rows)."""
    O = _mods()[0]
    lay = case.lay
    u = layer * case.w.n_kv_heads + kv
    a, b = int(lay.cu_seqlens[s]), int(lay.cu_seqlens[s + 1])
    frames = O.seq_frames_local(lay.cu_seqlens, lay.cu_frames, lay.frame_meta, s)
    hist, cur, _ = O.split_tokens(b - a, frames)
    where = f"{case.w.name} {sim} layer {layer} kv {kv} seq {s}"
    g = rho_gpu[u, a:b]
    if rows is None:
        off = np.ones(b - a, bool)
        off[hist] = False
        assert (g[off] == 0).all(), f"{where}: rho not 0 off the history"
    else:
        hist = hist[rows]
    if len(hist) == 0:
        return 0.0
    K = O.bf16_to_f64(case.k[layer, kv, a:b])
    ref = O.tsg_similarity(K, hist, cur, sim)
    got = g[hist].astype(np.float64)
    n = (K * K).sum(axis=1)
    ncur = n[cur].max()
    if sim == "dot":
        lim = DOT_TOL * np.sqrt(n[hist] * ncur)
        err = np.abs(got - ref)
    else:
        assert (got <= 0).all(), f"{where}: -L2 above 0"
        e2 = L2_TOL * (n[hist] + ncur)
        Kc = K[cur]
        d2 = np.array([((K[i] - Kc) ** 2).sum(axis=1).min() for i in hist])  # unsnapped
        edge = np.abs(d2 - O.L2_SNAP * n[hist]) <= e2
        err = np.abs(got * got - ref * ref)
        lim = np.where(edge, np.maximum(e2, O.L2_SNAP * n[hist] + e2), e2)
    ratio = err / lim
    i = int(np.argmax(ratio))
    assert ratio[i] <= 1.0, f"{where}: row {hist[i]} gpu {got[i]!r} ref {ref[i]!r} err/tol {ratio[i]:.3g}"
    return float(ratio[i])


@pytest.mark.parametrize("name", ["ragged", "tiles", "dups", "g8w64"])
def test_similarity_variants_small(torch_cuda, name):
    O, S, H, SMALL = _mods()
    w = SMALL[name]
    H.log(f"tsg similarity {name}: L={w.total_tokens}")
    case = H.Case(w)
    S.stlite_tsg_rho(case.prob, case.dk, case.out.rho, case.out.ws_tsg)
    base = case.out.rho.cpu().numpy()
    cos = _similarity(case, "cosine").cpu().numpy()
    assert np.array_equal(cos, base), f"{name}: the cosine variant differs from stlite_tsg_rho"
    for sim in ("dot", "neg_l2"):
        rho = _similarity(case, sim).cpu().numpy()
        worst = 0.0
        for u, layer, kv, s, a, L, hist, cur in _units(case):
            worst = max(worst, check_similarity(case, rho, sim, layer, kv, s))
        H.log(f"tsg similarity {name} {sim}: worst err/tol {worst:.3g}")


def test_duplicates_snap_under_every_similarity(torch_cuda):
    """Exact duplicate frames: rho = 1 (cosine) and exactly 0 (negative L2) on
    every copied token; the dot product is at least the copy's ||k||^2."""
    O, S, H, SMALL = _mods()
    case = H.Case(SMALL["dups"])
    nl2 = _similarity(case, "neg_l2").cpu().numpy()
    cos = _similarity(case, "cosine").cpu().numpy()
    dot = _similarity(case, "dot").cpu().numpy()
    n_zero = 0
    for u, layer, kv, s, a, L, hist, cur in _units(case):
        K = O.bf16_to_f64(case.k[layer, kv, a:a + L])
        copies = [i for i in hist if (K[cur] == K[i]).all(axis=1).any()]
        assert all(nl2[u, a + i] == 0.0 and cos[u, a + i] == 1.0 for i in copies)
        for i in copies:
            n_i = (K[i] * K[i]).sum()
            assert dot[u, a + i] >= n_i - DOT_TOL * np.sqrt(n_i * (K[cur] ** 2).sum(axis=1).max())
        n_zero += len(copies)
    assert n_zero > 0


def test_variant_rho_feeds_adaptive_gate(torch_cuda):
    """stlite_tsg_threshold on a dot or -L2 rho: the oracle's gate and tau_red on
    the same rho, bit for bit."""
    import torch
    O, S, H, SMALL = _mods()
    for name in ("ragged", "dups", "beta_tiny"):
        case = H.Case(SMALL[name])
        for sim in ("dot", "neg_l2"):
            rho = _similarity(case, sim)
            tau = torch.full((case.prob.units, case.prob.n_seqs), 7.0, dtype=torch.float32, device="cuda")
            gate = torch.full((case.prob.units, case.prob.total_tokens), 9, dtype=torch.uint8, device="cuda")
            S.stlite_tsg_threshold(case.prob, rho, tau, gate, case.out.ws_tsg)
            torch.cuda.synchronize()
            r, t, g = rho.cpu().numpy(), tau.cpu().numpy(), gate.cpu().numpy()
            for u, layer, kv, s, a, L, hist, cur in _units(case):
                B = int(case.cu_budget[s + 1] - case.cu_budget[s])
                want, tau_ref = O.tsg_gate(r[u, a:a + L][hist].astype(np.float64), hist, L, B)
                assert np.array_equal(g[u, a:a + L], want), f"{name} {sim} unit {u} seq {s}: gate"
                if min(B, len(hist)) > 0:
                    assert t[u, s] == np.float32(tau_ref), f"{name} {sim} unit {u} seq {s}: tau"
                else:
                    assert np.isnan(t[u, s])


@pytest.mark.parametrize("name", ["ragged", "tiles", "dups"])
def test_fixed_gate(torch_cuda, name):
    import torch
    O, S, H, SMALL = _mods()
    case = H.Case(SMALL[name])
    S.stlite_tsg_rho(case.prob, case.dk, case.out.rho, case.out.ws_tsg)
    torch.cuda.synchronize()
    rho = case.out.rho.cpu().numpy()
    present = float(rho[0][rho[0] != 0][0]) if (rho[0] != 0).any() else 0.5
    gate = torch.empty((case.prob.units, case.prob.total_tokens), dtype=torch.uint8, device="cuda")
    for tau in (0.85, 0.5, present, float("inf"), -float("inf"), -2.0):
        gate.fill_(9)
        S.stlite_tsg_fixed_gate(case.prob, case.out.rho, tau, gate)
        torch.cuda.synchronize()
        g = gate.cpu().numpy()
        flips = 0
        for u, layer, kv, s, a, L, hist, cur in _units(case):
            want = O.tsg_fixed_gate(rho[u, a:a + L][hist].astype(np.float64), hist, L, tau)
            assert np.array_equal(g[u, a:a + L], want), f"{name} tau {tau} unit {u} seq {s}"
            if tau == 0.85 and len(hist):
                K = O.bf16_to_f64(case.k[layer, kv, a:a + L])
                ref_rho = O.tsg_rho(K, hist, cur)
                ref = O.tsg_fixed_gate(ref_rho, hist, L, tau)
                diff = np.flatnonzero(g[u, a:a + L] != ref)
                r_of = np.full(L, np.nan)
                r_of[hist] = ref_rho
                band = 1e-3 * np.maximum(np.abs(r_of[diff]), 1e-2)
                assert (np.abs(r_of[diff] - tau) <= band).all(), f"{name} unit {u} seq {s}: flips off the band"
                flips += len(diff)
        if tau == float("inf"):
            assert g.all()
        H.log(f"fixed gate {name} tau {tau}: ok (band flips vs oracle rho {flips})")


@pytest.mark.timeout(900)
def test_similarity_variants_trajectory_sampled(torch_cuda):
    """The 150,528-token trajectory (two of its layers): dot and -L2 rho on 1024
    sampled historical rows of four units against the oracle."""
    O, S, H, SMALL = _mods()
    w = W.config(3)
    H.log(f"tsg similarity trajectory: generate L={w.total_tokens} x 2 layers")
    case = H.Case(w, layers=[0, 27])
    rng = np.random.default_rng(2603)
    for sim in ("dot", "neg_l2"):
        H.log(f"tsg similarity trajectory {sim}: run")
        rho = _similarity(case, sim).cpu().numpy()
        for layer, kv in ((0, 0), (0, 3), (1, 1), (1, 2)):
            a, b = int(case.lay.cu_seqlens[0]), int(case.lay.cu_seqlens[1])
            frames = O.seq_frames_local(case.lay.cu_seqlens, case.lay.cu_frames, case.lay.frame_meta, 0)
            hist, _, _ = O.split_tokens(b - a, frames)
            rows = np.sort(rng.choice(len(hist), size=min(1024, len(hist)), replace=False))
            r = check_similarity(case, rho, sim, layer, kv, 0, rows=rows)
            H.log(f"tsg similarity trajectory {sim} layer {layer} kv {kv}: worst err/tol {r:.3g}")


@pytest.mark.parametrize("name", ["ragged", "dups"])
def test_uniform_base_prior(torch_cuda, name):
    """The uniform base prior: stlite_select_topk with a constant a_base, on the
    GPU's own Phi and gate, against the oracle's top-B of the same scores."""
    import torch
    O, S, H, SMALL = _mods()
    case = H.Case(SMALL[name])
    res = case.run()
    out = case.out
    const = torch.full_like(out.a_base, 0.125)
    kept = torch.empty_like(out.kept)
    S.stlite_select_topk(case.prob, const, out.phi, out.gate, case.w.alpha, kept, None, out.ws)
    torch.cuda.synchronize()
    kept = kept[:, :case.prob.total_budget].cpu().numpy()
    cb = case.cu_budget
    for u, layer, kv, s, a, L, hist, cur in _units(case):
        frames = O.seq_frames_local(case.lay.cu_seqlens, case.lay.cu_frames, case.lay.frame_meta, s)
        _, _, text = O.split_tokens(L, frames)
        visual = np.ones(L, bool)
        visual[text] = False
        Sref = O.integrate(np.full(L, 0.125), res["phi"][u, a:a + L].astype(np.float64),
                           res["gate"][u, a:a + L], visual, case.w.alpha)
        B = int(cb[s + 1] - cb[s])
        got = kept[u, cb[s]:cb[s + 1]] - a
        want = O.select_topk(Sref, B)
        sym = np.setxor1d(got, want)
        if len(sym):
            sB = np.sort(Sref.astype(np.float32))[::-1][B - 1]
            assert (np.abs(Sref[sym] - sB) <= 1e-6 * abs(sB)).all(), f"{name} unit {u} seq {s}"


@pytest.mark.timeout(900)
def test_variants_ragged_batch_sampled(torch_cuda):
    """The ragged batch of 8 trajectories (two of its layers): dot and -L2 rho on
    sampled rows of sampled sequences, and the fixed gate on every unit."""
    import torch
    O, S, H, SMALL = _mods()
    w = W.config(4)
    H.log(f"tsg variants ragged batch: generate L={w.total_tokens} x 2 layers")
    case = H.Case(w, layers=[0, 27])
    rng = np.random.default_rng(4)
    for sim in ("dot", "neg_l2"):
        rho = _similarity(case, sim).cpu().numpy()
        for layer, kv, s in ((0, 0, 0), (0, 2, 3), (1, 1, 5), (1, 3, 7)):
            a, b = int(case.lay.cu_seqlens[s]), int(case.lay.cu_seqlens[s + 1])
            frames = O.seq_frames_local(case.lay.cu_seqlens, case.lay.cu_frames, case.lay.frame_meta, s)
            hist, _, _ = O.split_tokens(b - a, frames)
            rows = np.sort(rng.choice(len(hist), size=min(512, len(hist)), replace=False))
            rr = check_similarity(case, rho, sim, layer, kv, s, rows=rows)
            H.log(f"tsg variants ragged batch {sim} unit ({layer},{kv},{s}): worst err/tol {rr:.3g}")
    S.stlite_tsg_rho(case.prob, case.dk, case.out.rho, case.out.ws_tsg)
    gate = torch.empty((case.prob.units, case.prob.total_tokens), dtype=torch.uint8, device="cuda")
    S.stlite_tsg_fixed_gate(case.prob, case.out.rho, 0.85, gate)
    torch.cuda.synchronize()
    rho, g = case.out.rho.cpu().numpy(), gate.cpu().numpy()
    for u, layer, kv, s, a, L, hist, cur in _units(case):
        want = O.tsg_fixed_gate(rho[u, a:a + L][hist].astype(np.float64), hist, L, 0.85)
        assert np.array_equal(g[u, a:a + L], want), (u, s)

