"""Shared helpers of the GPU parity tests: run the HIP pass through the C ABI on
seeded workloads and compare it, unit by unit, with the fp64 oracle.

Tolerances (bf16 inputs, fp32 accumulation in the kernels):
  A_base, A_mean    |d| <= 1e-3 |ref| (A_mean sums positive A_base terms)
  Phi, rho          |d| <= 1e-3 max(|ref|, 1e-2)   (1 - cos cancels); Phi on
                    the tokens the GPU's gate admits, exactly 0 on the others
  gate              bit-exact, except historical tokens whose oracle rho lies
                    within 1e-4 max(|tau|, 1e-2) of the oracle's tau_red
  kept              exactly B per unit, ascending; tokens in the symmetric
                    difference must score within 1e-4 |s_B| of the oracle's
                    B-th score s_B (oracle S recomputed with the GPU gate when
                    a gate flip inside the band occurred)
  K', V'            bit-exact copies of the rows the GPU kept
  decode out        |d| <= 1e-4 sum_j p_j |v_j| + 1e-7 per element: the logits
                    are exact bf16 products summed in fp32, softmax and P V run
                    in fp32 over up to ~1.5e5 rows in chunks, an error of order
                    1e-6 .. 1e-5 of that scale
"""
from __future__ import annotations

import sys
import time

import numpy as np

from oracle import stlite_oracle as O
from paper_2603_00188_amd import stlite as S
from paper_2603_00188_amd import workload as W

A_RTOL = 1e-3
COS_TOL = 1e-3
BAND = 1e-4
DECODE_TOL = 1e-4


def log(msg: str):
    sys.__stdout__.write(f"[gpu-test {time.strftime('%H:%M:%S')}] {msg}\n")
    sys.__stdout__.flush()


class Case:
    """Seeded inputs of one workload, on the host and on the device."""

    def __init__(self, w: W.Workload, layers=None, device="cuda", inputs=None):
        """inputs = (layout, k, v, q) of already drawn arrays (e.g. the per-step
        batch of W.make_step_inputs, whose ``workload`` is then ``w``)."""
        import torch
        self.w = w
        if inputs is None:
            scene, self.k, self.v, self.q = W.make_inputs(w, layers)
            self.lay = scene.layout
        else:
            self.lay, self.k, self.v, self.q = inputs
        self.n_layers = self.k.shape[0]
        self.cu_budget = S.budgets(self.lay.cu_seqlens, *w.beta)
        self.prob = S.Problem(self.n_layers, w.n_q_heads, w.n_kv_heads, w.window, self.lay.cu_seqlens,
                              self.lay.cu_frames, self.lay.frame_meta, self.cu_budget, device=device)
        as_dev = lambda x: torch.from_numpy(x.view(np.int16)).to(device)
        self.dk, self.dv, self.dq = as_dev(self.k), as_dev(self.v), as_dev(self.q)
        self.out = S.Buffers(self.prob, device=device)

    def run(self, alpha=None, css=True, tsg=True, overlap=False, mean_width=0):
        import torch
        # Every output element the comparisons read must be written by the
        # pass: poison them first (NaN, a gate byte of 0xAB, kept index -1).
        o = self.out
        o.a_base.fill_(float("nan"))
        o.kept.fill_(-1)
        if css:
            o.phi.fill_(float("nan"))
        if tsg:
            o.rho.fill_(float("nan"))
            o.gate.fill_(0xAB)
        S.compress(self.prob, self.dq, self.dk, self.dv, self.out,
                   alpha=self.w.alpha if alpha is None else alpha, css=css, tsg=tsg, overlap=overlap,
                   mean_width=mean_width)
        torch.cuda.synchronize()
        o = self.out
        U = self.prob.units
        res = {n: getattr(o, n).cpu().numpy() for n in ("a_base", "phi", "rho", "tau", "gate", "score")}
        if mean_width:
            res["a_mean"] = o.a_mean.cpu().numpy().reshape(U, -1)
        Bt = self.prob.total_budget
        res["kept"] = o.kept[:, :Bt].cpu().numpy()
        res["k_out"] = o.k_out[:, :Bt].cpu().numpy().view(np.uint16)
        res["v_out"] = o.v_out[:, :Bt].cpu().numpy().view(np.uint16)
        for n in ("a_base", "phi", "rho", "score", "gate"):
            res[n] = res[n].reshape(U, -1)
        return res

    def oracle(self, layer: int, kv: int, s: int, alpha=None, css=True, tsg=True, mean_width=0):
        return O.compress_sequence(self.q, self.k, self.v, self.lay.cu_seqlens, self.lay.cu_frames,
                                   self.lay.frame_meta, s, layer, kv, self.w.group, self.w.beta,
                                   self.w.alpha if alpha is None else alpha, css, tsg, mean_width)


def _rel_check(name, got, ref, floor, tol, where):
    err = np.abs(got.astype(np.float64) - ref) / np.maximum(np.abs(ref), floor)
    if err.size and not (err <= tol).all():
        i = int(np.argmax(err))
        raise AssertionError(f"{where}: {name} rel err {err[i]:.3e} at {i}: gpu {got[i]!r} ref {ref[i]!r}")
    return float(err.max()) if err.size else 0.0


def compare_unit(case: Case, res, layer: int, kv: int, s: int, alpha=None, css=True, tsg=True,
                 ref=None):
    """Compare every stage of one (sequence, layer, kv head) unit with the oracle."""
    w = case.w
    u = layer * w.n_kv_heads + kv
    where = f"{w.name} layer {layer} kv {kv} seq {s}"
    a, b = int(case.lay.cu_seqlens[s]), int(case.lay.cu_seqlens[s + 1])
    if ref is None:
        ref = case.oracle(layer, kv, s, alpha, css, tsg)
    stats = {}
    stats["A"] = _rel_check("A_base", res["a_base"][u, a:b], ref["A"], 1e-30, A_RTOL, where)
    if "A_mean" in ref:  # sums of positive terms each within A_RTOL stay within A_RTOL
        stats["A_mean"] = _rel_check("A_mean", res["a_mean"][u, a:b], ref["A_mean"], 1e-30, A_RTOL, where)
    hist = ref["hist"]
    gate_ref = ref["gate"]
    gpu_gate = res["gate"][u, a:b]
    if css:
        # the gated CSS call writes Phi = 0 where the GPU's gate is 0 and the
        # ungated value elsewhere
        vis = ref["visual"]
        live = vis & (gpu_gate != 0) if tsg else vis
        stats["phi"] = _rel_check("phi", res["phi"][u, a:b][live], ref["phi"][live], 1e-2, COS_TOL, where)
        assert (res["phi"][u, a:b][~live] == 0).all(), f"{where}: phi not 0 on text or gated-out tokens"
    if tsg:
        stats["rho"] = _rel_check("rho", res["rho"][u, a:b][hist], ref["rho"], 1e-2, COS_TOL, where)
        nonhist = np.ones(b - a, bool)
        nonhist[hist] = False
        assert (res["rho"][u, a:b][nonhist] == 0).all(), f"{where}: rho not 0 off the history"
        diff = np.flatnonzero(gpu_gate != gate_ref)
        if len(diff):
            tau = ref["tau"]
            band = BAND * max(abs(tau), 1e-2)
            rho_of = np.full(b - a, np.nan)
            rho_of[hist] = ref["rho"]
            bad = diff[~(np.abs(rho_of[diff] - tau) <= band)]
            assert len(bad) == 0, f"{where}: gate differs outside the tie band at {bad[:10]}"
        assert gpu_gate[hist].sum() == min(ref["B"], len(hist)), f"{where}: gate count"
        assert (gpu_gate[np.setdiff1d(np.arange(b - a), hist)] == 1).all()
        if len(hist) and min(ref["B"], len(hist)) > 0:
            tg = res["tau"][u, s]
            assert abs(tg - ref["tau"]) <= BAND * max(abs(ref["tau"]), 1e-2) + 1e-6, f"{where}: tau"
        stats["gate_flips"] = int(len(diff))
    else:
        diff = []
    # kept set
    B = ref["B"]
    cb = case.cu_budget
    kept = res["kept"][u, cb[s]:cb[s + 1]]
    assert len(kept) == B
    assert (np.diff(kept) > 0).all() and (kept >= a).all() and (kept < b).all(), f"{where}: kept order/range"
    S_ref = ref["S"]
    if len(diff):  # re-score with the GPU's gate so that one band flip cannot cascade
        S_ref = O.integrate(ref.get("A_mean", ref["A"]), ref["phi"], gpu_gate, ref["visual"],
                            (w.alpha if alpha is None else alpha) if css else 0.0)
        kept_ref = O.select_topk(S_ref, B)
    else:
        kept_ref = ref["kept"]
    sym = np.setxor1d(kept - a, kept_ref)
    if len(sym):
        s32 = S_ref.astype(np.float32)
        sB = np.sort(s32)[::-1][B - 1]
        far = sym[~(np.abs(S_ref[sym] - sB) <= BAND * abs(sB))]
        assert len(far) == 0, f"{where}: kept differs away from the B-th score at {far[:10]}"
    stats["kept_swaps"] = int(len(sym))
    # compaction: exact copies of the rows the GPU kept
    kb = case.k[layer, kv][kept]
    vb = case.v[layer, kv][kept]
    assert (res["k_out"][u, cb[s]:cb[s + 1]] == kb).all(), f"{where}: K' not an exact copy"
    assert (res["v_out"][u, cb[s]:cb[s + 1]] == vb).all(), f"{where}: V' not an exact copy"
    return stats


def run_decode(case: Case):
    """Decode attention over the full and the compacted cache of the last run
    (the decode query of each head: its last window query)."""
    import torch
    q_dec = W.decode_queries(case.q)
    dq = torch.from_numpy(q_dec.view(np.int16)).to(case.dk.device)
    full = S.decode(case.prob, dq, case.dk, case.dv, S.CACHE_FULL)
    comp = S.decode(case.prob, dq, case.out.k_out, case.out.v_out, S.CACHE_COMPACT)
    torch.cuda.synchronize()
    return q_dec, full.cpu().numpy(), comp.cpu().numpy()


def compare_decode(case: Case, res, dec, layer: int, kv: int, s: int):
    """Both decode outputs of one (layer, kv head, sequence) against the oracle,
    the compacted one over the rows the GPU kept (their copies are checked
    bit-exact elsewhere).  Returns the worst error in units of the tolerance."""
    q_dec, full, comp = dec
    G = case.w.group
    heads = slice(kv * G, (kv + 1) * G)
    Q = O.bf16_to_f64(q_dec[layer, s, heads])
    a, b = int(case.lay.cu_seqlens[s]), int(case.lay.cu_seqlens[s + 1])
    u = layer * case.w.n_kv_heads + kv
    ba, bb = int(case.cu_budget[s]), int(case.cu_budget[s + 1])
    worst = 0.0
    for name, got, Kb, Vb in (("full", full, case.k[layer, kv, a:b], case.v[layer, kv, a:b]),
                              ("compact", comp, res["k_out"][u, ba:bb], res["v_out"][u, ba:bb])):
        K, V = O.bf16_to_f64(Kb), O.bf16_to_f64(Vb)
        ref = O.decode_attention(Q, K, V)
        scale = O.decode_attention(Q, K, np.abs(V))
        g = got[layer, s, heads].astype(np.float64)
        lim = DECODE_TOL * scale + 1e-7
        err = np.abs(g - ref)
        bad = err > lim
        if bad.any():
            i = np.argwhere(bad)[0]
            raise AssertionError(f"decode {name} unit ({layer},{kv},{s}) head {i[0]} dim {i[1]}: "
                                 f"got {g[tuple(i)]!r} ref {ref[tuple(i)]!r} tol {lim[tuple(i)]:.3g}")
        worst = max(worst, float((err / lim).max()) if err.size else 0.0)
    return worst
