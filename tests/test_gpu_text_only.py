"""A problem with no frames at all (two text-only sequences): every entry
point takes its frame-free path.  Against the oracle: Phi = 0, rho = 0,
gate = 1, the kept set is the top-B of A alone, decode and CHR as usual, and
every variant writes its defined zero / one outputs.
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


def test_text_only_problem_every_entry_point(torch_cuda):
    import torch
    from oracle import stlite_oracle as O
    from paper_2603_00188_amd import stlite as S
    from tests import gpu_harness as H
    from tests.test_gpu_parity import _small
    w = _small([[(W.TEXT, 70)], [(W.TEXT, 41)]], G=2, Hkv=2, window=6, beta=(1, 4))
    case = H.Case(w)
    assert len(case.lay.frame_meta) == 0
    res = case.run()
    for layer in range(w.n_layers):
        for kv in range(w.n_kv_heads):
            for s in range(case.lay.n_seqs):
                H.compare_unit(case, res, layer, kv, s)
    assert (res["phi"] == 0).all() and (res["rho"] == 0).all() and (res["gate"] == 1).all()
    p, U, L = case.prob, case.prob.units, case.prob.total_tokens
    f32 = dict(dtype=torch.float32, device="cuda")
    # variants: rho 0 everywhere, gate 1, Phi 0
    for sim in (S.SIM_COSINE, S.SIM_DOT, S.SIM_NEG_L2):
        rho = torch.full((U, L), 7.0, **f32)
        S.stlite_tsg_similarity(p, sim, case.dk, rho, case.out.ws_tsg)
        assert (rho.cpu().numpy() == 0).all(), sim
    gate = torch.full((U, L), 9, dtype=torch.uint8, device="cuda")
    S.stlite_tsg_fixed_gate(p, case.out.rho, 0.85, gate)
    assert (gate.cpu().numpy() == 1).all()
    for nb in (5, 7, 9):
        phi = torch.full((U, L), 7.0, **f32)
        S.stlite_css_saliency_nbhd(p, nb, case.dk, phi)
        assert (phi.cpu().numpy() == 0).all(), nb
    # concatenated key space: A mean of the heads, no frames, kept = top-B of A_layer
    pl = S.layer_problem(p)
    r = S.compress_concat(p, pl, case.dq, case.dk, case.dv, alpha=w.alpha)
    torch.cuda.synchronize()
    cb = case.cu_budget
    for layer in range(w.n_layers):
        for s in range(case.lay.n_seqs):
            a, b = int(case.lay.cu_seqlens[s]), int(case.lay.cu_seqlens[s + 1])
            ref = O.compress_layer_concat(case.q[layer, s], case.k[layer, :, a:b], case.v[layer, :, a:b], [],
                                          w.beta, w.alpha)
            H._rel_check("A_layer", r["a_layer"][layer, a:b].cpu().numpy(), ref["A"], 1e-30, H.A_RTOL, "concat")
            kept = r["kept"][layer, cb[s]:cb[s + 1]].cpu().numpy() - a
            sym = np.setxor1d(kept, ref["kept"])
            if len(sym):
                sB = np.sort(ref["S"].astype(np.float32))[::-1][ref["B"] - 1]
                assert (np.abs(ref["S"][sym] - sB) <= H.BAND * abs(sB)).all()
    assert (r["phi"].cpu().numpy() == 0).all() and (r["rho"].cpu().numpy() == 0).all()
    assert (r["gate"].cpu().numpy() == 1).all()
    # decode over both caches and the cache hit rate
    dec = H.run_decode(case)
    for layer in range(w.n_layers):
        for kv in range(w.n_kv_heads):
            for s in range(case.lay.n_seqs):
                H.compare_decode(case, res, dec, layer, kv, s)
    q_dec = torch.from_numpy(np.ascontiguousarray(W.decode_queries(case.q)).view(np.int16)).cuda()
    star, _ = S.oracle_set(S.decode_problem(p), q_dec, case.dk)
    hits = S.kept_overlap(p, case.out.kept, star)
    torch.cuda.synchronize()
    Bt = p.total_budget
    st, kp = star[:, :Bt].cpu().numpy(), case.out.kept[:, :Bt].cpu().numpy()
    for u in range(U):
        for s in range(case.lay.n_seqs):
            assert hits.cpu().numpy()[u, s] == len(np.intersect1d(kp[u, cb[s]:cb[s + 1]], st[u, cb[s]:cb[s + 1]]))
