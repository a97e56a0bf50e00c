"""GPU parity of recompression at every step of one trajectory (problem setup,
Eq. history_context; Eq. chr) against the fp64 oracle.

Step t compresses its own context: frames 0..t of the trajectory and the text
after each, L_t tokens, budget B_t = floor(beta L_t); its decode query sums the
keys of the step's element and of an earlier frame's changed region.  The steps
run either packed as one varlen batch (one sequence per step) or one problem
per step (how a serving loop calls the library); both are compared stage by
stage with the oracle under the tolerances of the pass (tests/gpu_harness.py),
and the per-step cache hit rates and their mean over the steps (Eq. chr) under
the tie-band slack of tests/test_gpu_chr.py.
"""
import dataclasses

import numpy as np
import pytest

from paper_2603_00188_amd import workload as W

pytestmark = pytest.mark.gpu

F, T = W.FRAME, W.TEXT


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _mods():
    from oracle import stlite_oracle as O
    from tests import gpu_harness as H
    from tests import test_gpu_chr as C
    return O, H, C


def _trajectory():
    """Six frames of 12 x 21 patches, text after each (the window in the last
    text run of every step), 30% duplicate frames, two layers, G = 4, Hkv = 2."""
    return W.Workload("steps_small", 2, 8, 2, 16, (3, 10),
                      (tuple([(F, 12, 21), (T, 37)] * 5 + [(F, 12, 21), (T, 60)]),),
                      W.Redundancy(frac=(0.05, 0.2), n_rects=(1, 3), dup_frac=0.3), ((1, 2), (1, 3)), seed=21)


def _step_case(H, w, t, base):
    """Step t of the trajectory as a problem of its own (one sequence)."""
    scene, kb, vb, _ = base
    wt = dataclasses.replace(w, seqs=(W.step_prefix_segments(w, t),))
    lay = W.make_layout(wt)
    n = lay.total_tokens
    si = W.make_step_inputs(w, steps=[t], base=base, pack=False)
    k = np.ascontiguousarray(kb[:, :, :n])
    v = np.ascontiguousarray(vb[:, :, :n])
    return H.Case(wt, inputs=(lay, k, v, si.q)), si.q_dec


def test_steps_packed_batch_all_units(torch_cuda):
    """Every step packed as one batch: all stages of every (step, unit)
    against the oracle, I* and both hit rates per unit, and the Eq. chr mean
    over the steps against the oracle's recompress_steps on the trajectory."""
    O, H, C = _mods()
    w = _trajectory()
    base = W.make_inputs(w)
    si = W.make_step_inputs(w, base=base)
    case = H.Case(si.workload, inputs=(si.layout, si.k, si.v, si.q))
    H.log(f"steps packed: {len(si.steps)} steps, L = {list(np.diff(si.layout.cu_seqlens))}")
    r = C.run_chr(case, si.q_dec)
    fm = base[0].layout.seq_frames(0)
    frames = [tuple(int(x) for x in f) for f in fm]
    ends = [int(x) for x in fm[1:, 0]] + [base[0].layout.total_tokens]
    gpu_rates = np.zeros((case.prob.units, len(si.steps)))
    for layer in range(w.n_layers):
        for kv in range(w.n_kv_heads):
            u = layer * w.n_kv_heads + kv
            traj = O.recompress_steps(si.q[layer, :, kv * w.group:(kv + 1) * w.group],
                                      si.q_dec[layer, :, kv * w.group:(kv + 1) * w.group],
                                      base[1][layer, kv], base[2][layer, kv], frames, ends, si.steps,
                                      w.beta, w.alpha)
            for i, t in enumerate(si.steps):
                ref = case.oracle(layer, kv, i)
                # the packed sequence is step t of the trajectory, bit for bit on the oracle side
                np.testing.assert_array_equal(ref["kept"], traj["steps"][i]["kept"])
                H.compare_unit(case, r["res"], layer, kv, i, ref=ref)
                got = C.check_chr_unit(case, r, layer, kv, i, ref=ref)
                gpu_rates[u, i] = got["st_lite"]
            # Eq. chr for this unit: the mean of its per-step rates
            assert O.trajectory_cache_hit_rate(gpu_rates[u]) == pytest.approx(np.mean(gpu_rates[u]), abs=1e-15)
            H.log(f"steps packed unit ({layer},{kv}): CHR gpu {np.mean(gpu_rates[u]):.4f} "
                  f"oracle {traj['chr']:.4f}")


def test_steps_one_problem_per_step(torch_cuda):
    """The serving pattern: each step's cache as a problem of its own."""
    O, H, C = _mods()
    w = _trajectory()
    base = W.make_inputs(w)
    for t in range(len(base[0].layout.frame_meta)):
        case, q_dec = _step_case(H, w, t, base)
        r = C.run_chr(case, q_dec)
        for layer in range(w.n_layers):
            for kv in range(w.n_kv_heads):
                ref = case.oracle(layer, kv, 0)
                H.compare_unit(case, r["res"], layer, kv, 0, ref=ref)
                C.check_chr_unit(case, r, layer, kv, 0, ref=ref)
        if t == 0:
            assert r["res"]["gate"].all(), "the first step has no history: TSG admits everything"


@pytest.mark.timeout(900)
def test_steps_trajectory_sampled(torch_cuda):
    """The 150,528-token trajectory recompressed at steps 0, 1, 23 and 47, one
    problem per step as the benchmark runs them, on sampled units."""
    O, H, C = _mods()
    w = W.config(3)
    H.log(f"steps trajectory: generate L={w.total_tokens} x {w.n_layers} layers")
    base = W.make_inputs(w, workers=16)
    for t in (0, 1, 23, 47):
        case, q_dec = _step_case(H, w, t, base)
        H.log(f"steps trajectory: step {t}, L_t = {case.lay.total_tokens}")
        r = C.run_chr(case, q_dec)
        for layer, kv in ((0, 0), (13, 2), (27, 3)):
            ref = case.oracle(layer, kv, 0)
            st = H.compare_unit(case, r["res"], layer, kv, 0, ref=ref)
            got = C.check_chr_unit(case, r, layer, kv, 0, ref=ref)
            H.log(f"steps trajectory step {t} unit ({layer},{kv}): {st} {got}")
        del case, r
