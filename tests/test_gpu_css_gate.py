"""GPU: CSS with the TSG gate (stlite_css_saliency with a gate) against the
ungated call on the same keys.

Where the gate admits a token, the gated Phi must be bit for bit the ungated
Phi; where the gate is 0 it must be exactly 0; text stays 0.  Gates come from
stlite_tsg_gate on the parity workloads, and from the caller: sparse random
gates, and gates that leave out whole row bands and whole frames, so that
the kernel's skip of unneeded cosines runs next to admitted rows.
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


def _check(case, gate_np, where):
    import torch
    from paper_2603_00188_amd import stlite as S
    out = case.out
    S.stlite_css_saliency(case.prob, case.dk, out.phi, None)
    torch.cuda.synchronize()
    ungated = out.phi.cpu().numpy().reshape(case.prob.units, -1)
    gate = torch.from_numpy(np.ascontiguousarray(gate_np, dtype=np.uint8)).cuda()
    out.phi.fill_(7.0)
    S.stlite_css_saliency(case.prob, case.dk, out.phi, gate)
    torch.cuda.synchronize()
    gated = out.phi.cpu().numpy().reshape(case.prob.units, -1)
    on = gate_np != 0
    assert np.array_equal(gated[on], ungated[on]), f"{where}: gated phi differs on admitted tokens"
    assert (gated[~on] == 0).all(), f"{where}: gated phi not 0 where the gate is 0"
    return int(on.sum())


@pytest.mark.parametrize("name", ["ragged", "tiles", "dups", "many_frames"])
def test_css_with_tsg_gate_matches_ungated(torch_cuda, name):
    import torch
    from tests import gpu_harness as H
    from tests.test_gpu_parity import SMALL
    from paper_2603_00188_amd import stlite as S
    case = H.Case(SMALL[name])
    out = case.out
    S.stlite_tsg_gate(case.prob, case.dk, out.rho, out.tau, out.gate, out.ws_tsg)
    torch.cuda.synchronize()
    gate = out.gate.cpu().numpy().reshape(case.prob.units, -1).copy()
    n = _check(case, gate, name)
    H.log(f"css gate {name}: {n} of {gate.size} tokens admitted")


def test_css_with_caller_gates(torch_cuda):
    from tests import gpu_harness as H
    from tests.test_gpu_parity import SMALL
    case = H.Case(SMALL["tiles"])
    U, L = case.prob.units, case.prob.total_tokens
    rng = np.random.default_rng(3)
    fm = case.lay.frame_meta
    gates = {
        "all_zero": np.zeros((U, L), np.uint8),
        "all_one": np.ones((U, L), np.uint8),
        "sparse_5pct": (rng.random((U, L)) < 0.05).astype(np.uint8),
        "values_2_255": np.where(rng.random((U, L)) < 0.3, rng.integers(2, 256, (U, L)), 0).astype(np.uint8),
    }
    bands = np.zeros((U, L), np.uint8)          # every frame: rows 5..6 only admitted
    frames = np.zeros((U, L), np.uint8)         # frame 1 fully admitted, the others not
    for f, (off, r, c) in enumerate(fm):
        bands[:, off + 5 * c: off + 7 * c] = 1
        if f == 1:
            frames[:, off:off + r * c] = 1
    gates["row_bands"] = bands
    gates["one_frame"] = frames
    corner = np.zeros((U, L), np.uint8)         # one admitted cell at each frame's last row and column
    for off, r, c in fm:
        corner[:, off + r * c - 1] = 1
        corner[:, off] = 1
    gates["corners"] = corner
    for name, g in gates.items():
        _check(case, g, name)


def test_css_gate_single_step_full_size(torch_cuda):
    """The single-step workload (one 36 x 80 frame, 28 layers): with a gate
    that admits a random half of the tokens."""
    from tests import gpu_harness as H
    case = H.Case(W.config(1))
    U, L = case.prob.units, case.prob.total_tokens
    g = (np.random.default_rng(9).random((U, L)) < 0.5).astype(np.uint8)
    _check(case, g, "single_step")
