"""GPU parity of the CSS neighbourhood-size ablation (k x k windows, k = 5, 7,
9) against the fp64 oracle, through stlite_css_saliency_nbhd.

Tolerance: as for the 3 x 3 path, |d| <= 1e-3 max(|Phi_ref|, 1e-2) on visual
tokens (the cosines are exact bf16 products summed in fp32 and scaled by
1-ulp inverse norms, an error of order 1e-6 in H; 1 - H cancels, hence the
floor), and exactly 0 on text.  nbhd = 3 gives the bits of stlite_css_saliency.
"""
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


def _mods():
    from oracle import stlite_oracle as O
    from paper_2603_00188_amd import stlite as S
    from tests import gpu_harness as H
    from tests.test_gpu_parity import SMALL
    return O, S, H, SMALL


def _phi(case, nbhd):
    import torch
    S = _mods()[1]
    phi = torch.full((case.prob.units, case.prob.total_tokens), 7.0, dtype=torch.float32, device="cuda")
    S.stlite_css_saliency_nbhd(case.prob, nbhd, case.dk, phi)
    torch.cuda.synchronize()
    return phi.cpu().numpy()


def check_phi(case, phi, nbhd, layer, kv, s, frames_only=None):
    O, S, H, _ = _mods()
    lay = case.lay
    u = layer * case.w.n_kv_heads + kv
    a, b = int(lay.cu_seqlens[s]), int(lay.cu_seqlens[s + 1])
    frames = O.seq_frames_local(lay.cu_seqlens, lay.cu_frames, lay.frame_meta, s)
    K = O.bf16_to_f64(case.k[layer, kv, a:b])
    where = f"{case.w.name} nbhd {nbhd} layer {layer} kv {kv} seq {s}"
    g = phi[u, a:b]
    if frames_only is None:
        ref = O.css_saliency(K, frames, nbhd)
        _, _, text = O.split_tokens(b - a, frames)
        visual = np.ones(b - a, bool)
        visual[text] = False
        assert (g[text] == 0).all(), f"{where}: phi not 0 on text"
        return H._rel_check("phi", g[visual], ref[visual], 1e-2, H.COS_TOL, where)
    worst = 0.0
    for fi in frames_only:
        off, r, c = frames[fi]
        ref = O.css_frame(K[off:off + r * c], r, c, nbhd)
        worst = max(worst, H._rel_check("phi", g[off:off + r * c], ref, 1e-2, H.COS_TOL, f"{where} frame {fi}"))
    return worst


@pytest.mark.parametrize("name", ["ragged", "tiles", "g8w64", "dups"])
def test_css_nbhd_small_all_units(torch_cuda, name):
    O, S, H, SMALL = _mods()
    w = SMALL[name]
    H.log(f"css nbhd {name}: L={w.total_tokens}")
    case = H.Case(w)
    base = _phi(case, 3)
    S.stlite_css_saliency(case.prob, case.dk, case.out.phi)
    assert np.array_equal(base, case.out.phi.cpu().numpy()), f"{name}: nbhd 3 differs from stlite_css_saliency"
    for nbhd in (5, 7, 9):
        phi = _phi(case, nbhd)
        worst = 0.0
        for layer in range(case.n_layers):
            for kv in range(w.n_kv_heads):
                for s in range(case.lay.n_seqs):
                    worst = max(worst, check_phi(case, phi, nbhd, layer, kv, s))
        H.log(f"css nbhd {name} k={nbhd}: worst rel err {worst:.3g}")


def test_css_nbhd_tiny_config(torch_cuda):
    """Three 16 x 16 frames with text between them."""
    O, S, H, _ = _mods()
    case = H.Case(W.config(0))
    for nbhd in (5, 7, 9):
        phi = _phi(case, nbhd)
        for kv in range(4):
            check_phi(case, phi, nbhd, 0, kv, 0)


@pytest.mark.timeout(900)
def test_css_nbhd_trajectory_sampled(torch_cuda):
    """The 150,528-token trajectory (two of its layers, 36 x 80 frames): sampled
    frames of four units against the oracle."""
    O, S, H, _ = _mods()
    w = W.config(3)
    H.log(f"css nbhd trajectory: generate L={w.total_tokens} x 2 layers")
    case = H.Case(w, layers=[0, 27])
    for nbhd in (5, 9):
        phi = _phi(case, nbhd)
        for layer, kv, frames in ((0, 0, (0, 47)), (0, 3, (20,)), (1, 1, (46,)), (1, 2, (5,))):
            r = check_phi(case, phi, nbhd, layer, kv, 0, frames_only=frames)
            H.log(f"css nbhd trajectory k={nbhd} layer {layer} kv {kv}: worst rel err {r:.3g}")


@pytest.mark.timeout(900)
def test_css_nbhd_ragged_batch_sampled(torch_cuda):
    """The ragged batch of 8 trajectories (two of its layers): sampled frames of
    sampled sequences at k = 7, text exactly 0 everywhere."""
    O, S, H, _ = _mods()
    w = W.config(4)
    H.log(f"css nbhd ragged batch: generate L={w.total_tokens} x 2 layers")
    case = H.Case(w, layers=[0, 27])
    phi = _phi(case, 7)
    lay = case.lay
    for s in range(lay.n_seqs):
        a, b = int(lay.cu_seqlens[s]), int(lay.cu_seqlens[s + 1])
        frames = O.seq_frames_local(lay.cu_seqlens, lay.cu_frames, lay.frame_meta, s)
        _, _, text = O.split_tokens(b - a, frames)
        assert (phi[:, a:b][:, text] == 0).all(), s
    for layer, kv, s, fr in ((0, 0, 0, (0, 5)), (0, 3, 4, (2,)), (1, 1, 7, (1,)), (1, 2, 6, (3,))):
        r = check_phi(case, phi, 7, layer, kv, s, frames_only=fr)
        H.log(f"css nbhd ragged batch unit ({layer},{kv},{s}): worst rel err {r:.3g}")

