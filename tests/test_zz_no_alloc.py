"""GPU: stlite_select_topk_noalloc (the selection with its workspace in the
library's static device array) against stlite_select_topk with a caller
workspace, through the C ABI, on two calls in a row -- the second on a
smaller problem, so the static array still holds the first call's words --
and on the full pass's own A, Phi and gate.  kept and S must agree bit for
bit."""
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


def _inputs(prob, seed):
    """A, Phi and gate drawn from few values, so that long runs of ties meet
    the budget boundary."""
    rng = np.random.default_rng(seed)
    U, L = prob.units, prob.total_tokens
    A = rng.choice(np.float32([1e-4, 2e-4, 5e-4, 3e-2]), size=(U, L)).astype(np.float32)
    phi = rng.choice(np.float32([0.9, 1.0, 1.1]), size=(U, L)).astype(np.float32)
    gate = (rng.random((U, L)) < 0.6).astype(np.uint8)
    return A, phi, gate


def _both(prob, A, phi, gate, alpha=1.0):
    import torch
    from paper_2603_00188_amd import stlite as S
    dev = lambda x: torch.from_numpy(np.ascontiguousarray(x)).cuda()
    dA, dphi, dgate = dev(A), dev(phi), dev(gate)
    Bt = max(prob.total_budget, 1)
    kept1 = torch.full((prob.units, Bt), -1, dtype=torch.int32, device="cuda")
    kept2 = torch.full_like(kept1, -2)
    s1 = torch.full((prob.units, prob.total_tokens), 7.0, dtype=torch.float32, device="cuda")
    s2 = torch.full_like(s1, 9.0)
    ws = torch.empty(max(prob.workspace_size(S.CALL_SELECT_TOPK), 256), dtype=torch.uint8, device="cuda")
    assert prob.workspace_size(S.CALL_SELECT_TOPK) <= S.NOALLOC_SCRATCH_BYTES
    S.stlite_select_topk(prob, dA, dphi, dgate, alpha, kept1, s1, ws)
    S.stlite_select_topk_noalloc(prob, dA, dphi, dgate, alpha, kept2, s2)
    torch.cuda.synchronize()
    Bt = prob.total_budget
    return (kept1[:, :Bt].cpu().numpy(), kept2[:, :Bt].cpu().numpy(), s1.cpu().numpy(), s2.cpu().numpy())


def test_noalloc_select_matches_workspace_call(torch_cuda):
    from paper_2603_00188_amd import stlite as S
    from tests import gpu_harness as H
    # first call: the single-step workload's layout (28 layers x 4 kv heads)
    w1 = W.config(1)
    case1 = H.Case(w1)
    for seed in (1, 2):
        k1, k2, s1, s2 = _both(case1.prob, *_inputs(case1.prob, seed))
        assert np.array_equal(k1, k2) and np.array_equal(s1, s2), f"single step, seed {seed}"
        H.log(f"noalloc: single step seed {seed}: {k1.size} kept entries agree")
    # second call, smaller: a ragged batch of four sequences, 2 layers x 2 kv heads
    from tests.test_gpu_parity import SMALL
    case2 = H.Case(SMALL["ragged"])
    assert case2.prob.workspace_size(S.CALL_SELECT_TOPK) < case1.prob.workspace_size(S.CALL_SELECT_TOPK)
    k1, k2, s1, s2 = _both(case2.prob, *_inputs(case2.prob, 3))
    assert np.array_equal(k1, k2) and np.array_equal(s1, s2), "ragged"
    # the pass's own A, Phi and gate on the ragged batch
    res = case2.run()
    A, phi, gate = (res[n].astype(t) for n, t in (("a_base", np.float32), ("phi", np.float32), ("gate", np.uint8)))
    k1, k2, s1, s2 = _both(case2.prob, A, phi, gate, case2.w.alpha)
    assert np.array_equal(k1, k2) and np.array_equal(s1, s2), "ragged, pass inputs"
    assert np.array_equal(k2, res["kept"]), "noalloc kept differs from the pass's kept"
