"""GPU parity of the concatenated key space (reading R3b: D = n_kv_heads * 128,
one kept set per layer) against the fp64 oracle's compress_layer_concat.

Tolerances are the per-head pass's: A_layer |d| <= 1e-3 |ref| (a mean of
per-head A, each within that bound); Phi and rho |d| <= 1e-3 max(|ref|, 1e-2);
gate bit-exact outside the 1e-4 tie band around tau; kept bit-exact outside the
1e-4 band around the B-th score (re-scored with the GPU's gate after a band
flip); K', V' exact copies of the rows the GPU kept, for every head.
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


def _mods():
    from oracle import stlite_oracle as O
    from paper_2603_00188_amd import stlite as S
    from tests import gpu_harness as H
    from tests.test_gpu_parity import SMALL, _small
    return O, S, H, SMALL, _small


def run_concat(case):
    import torch
    O, S, H, _, _ = _mods()
    pl = S.layer_problem(case.prob)
    r = S.compress_concat(case.prob, pl, case.dq, case.dk, case.dv, alpha=case.w.alpha)
    torch.cuda.synchronize()
    Bt = case.prob.total_budget
    out = {k: v.cpu().numpy() for k, v in r.items()}
    out["kept"] = out["kept"][:, :Bt]
    out["k_out"] = r["k_out"][:, :Bt].cpu().numpy().view(np.uint16)
    out["v_out"] = r["v_out"][:, :Bt].cpu().numpy().view(np.uint16)
    return out


def compare_layer(case, res, layer, s):
    O, S, H, _, _ = _mods()
    w = case.w
    lay = case.lay
    a, b = int(lay.cu_seqlens[s]), int(lay.cu_seqlens[s + 1])
    frames = O.seq_frames_local(lay.cu_seqlens, lay.cu_frames, lay.frame_meta, s)
    ref = O.compress_layer_concat(case.q[layer, s], case.k[layer, :, a:b], case.v[layer, :, a:b], frames, w.beta,
                                  w.alpha)
    where = f"{w.name} concat layer {layer} seq {s}"
    st = {"A": H._rel_check("A_layer", res["a_layer"][layer, a:b], ref["A"], 1e-30, H.A_RTOL, where)}
    vis = ref["visual"]
    st["phi"] = H._rel_check("phi", res["phi"][layer, a:b][vis], ref["phi"][vis], 1e-2, H.COS_TOL, where)
    assert (res["phi"][layer, a:b][~vis] == 0).all(), f"{where}: phi not 0 on text"
    hist = ref["hist"]
    st["rho"] = H._rel_check("rho", res["rho"][layer, a:b][hist], ref["rho"], 1e-2, H.COS_TOL, where)
    gpu_gate = res["gate"][layer, a:b]
    diff = np.flatnonzero(gpu_gate != ref["gate"])
    if len(diff):
        rho_of = np.full(b - a, np.nan)
        rho_of[hist] = ref["rho"]
        band = H.BAND * max(abs(ref["tau"]), 1e-2)
        assert (np.abs(rho_of[diff] - ref["tau"]) <= band).all(), f"{where}: gate differs outside the tie band"
    assert gpu_gate[hist].sum() == min(ref["B"], len(hist)), f"{where}: gate count"
    B = ref["B"]
    cb = case.cu_budget
    kept = res["kept"][layer, cb[s]:cb[s + 1]]
    assert len(kept) == B and (np.diff(kept) > 0).all() and (kept >= a).all() and (kept < b).all(), where
    S_ref = ref["S"]
    kept_ref = ref["kept"]
    if len(diff):
        S_ref = O.integrate(ref["A"], ref["phi"], gpu_gate, vis, w.alpha)
        kept_ref = O.select_topk(S_ref, B)
    sym = np.setxor1d(kept - a, kept_ref)
    if len(sym):
        sB = np.sort(S_ref.astype(np.float32))[::-1][B - 1]
        assert (np.abs(S_ref[sym] - sB) <= H.BAND * abs(sB)).all(), f"{where}: kept differs away from s_B"
    for h in range(w.n_kv_heads):
        u = layer * w.n_kv_heads + h
        assert (res["k_out"][u, cb[s]:cb[s + 1]] == case.k[layer, h][kept]).all(), f"{where}: K' head {h}"
        assert (res["v_out"][u, cb[s]:cb[s + 1]] == case.v[layer, h][kept]).all(), f"{where}: V' head {h}"
    st["kept_swaps"] = int(len(sym))
    return st


def _cases():
    O, S, H, SMALL, _small = _mods()
    F, T = W.FRAME, W.TEXT
    return {
        "ragged_h2": SMALL["ragged"],    # 2 kv heads, odd grids, text-only and 1x1 frames
        "g1w1_h4": SMALL["g1w1"],        # 4 kv heads, G = 1
        "tiles_h4": _small([[(F, 12, 21), (T, 37), (F, 12, 21), (T, 37), (F, 12, 21), (T, 150)]],
                           G=4, Hkv=4, window=16, beta=(3, 10)),
        "dups_h2": SMALL["dups"],        # exact duplicate frames
    }


@pytest.mark.parametrize("name", ["ragged_h2", "g1w1_h4", "tiles_h4", "dups_h2"])
def test_concat_small_all_layers(torch_cuda, name):
    O, S, H, _, _ = _mods()
    w = _cases()[name]
    H.log(f"concat {name}: L={w.total_tokens} Hkv={w.n_kv_heads}")
    case = H.Case(w)
    res = run_concat(case)
    worst = {}
    for layer in range(case.n_layers):
        for s in range(case.lay.n_seqs):
            for k, v in compare_layer(case, res, layer, s).items():
                worst[k] = max(worst.get(k, 0), v)
    H.log(f"concat {name}: {worst}")


def test_concat_tiny_config(torch_cuda):
    O, S, H, _, _ = _mods()
    case = H.Case(W.config(0))
    res = run_concat(case)
    H.log(f"concat tiny: {compare_layer(case, res, 0, 0)}")


def test_concat_unsupported_head_counts(torch_cuda):
    """3 and 1 kv heads are rejected before anything is enqueued."""
    import torch
    O, S, H, SMALL, _ = _mods()
    for name in ("tiles", "g8w64"):   # 3 and 1 kv heads
        case = H.Case(SMALL[name])
        phi = torch.empty((case.prob.n_layers, case.prob.total_tokens), dtype=torch.float32, device="cuda")
        with pytest.raises(S.StliteError) as e:
            S.stlite_css_saliency_concat(case.prob, case.dk, phi)
        assert e.value.status == S.ERR_UNSUPPORTED


@pytest.mark.timeout(900)
def test_concat_trajectory_sampled(torch_cuda):
    """The 150,528-token trajectory (two of its layers, four kv heads)."""
    O, S, H, _, _ = _mods()
    w = W.config(3)
    H.log(f"concat trajectory: generate L={w.total_tokens} x 2 layers")
    case = H.Case(w, layers=[0, 27])
    res = run_concat(case)
    for layer in (0, 1):
        H.log(f"concat trajectory layer {layer}: {compare_layer(case, res, layer, 0)}")
