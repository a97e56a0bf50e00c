"""The pass captured into a HIP graph (stlite.capture_compress) replays to the
same bits as the eager pass: several replays, with eager work and host reads
between them, each compared with the eager outputs; inputs changed in place
between replays are picked up."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _outputs(out, Bt):
    return {"a_base": out.a_base.cpu().numpy(), "phi": out.phi.cpu().numpy(), "gate": out.gate.cpu().numpy(),
            "kept": out.kept[:, :Bt].cpu().numpy(), "k_out": out.k_out[:, :Bt].cpu().numpy().view(np.uint16),
            "v_out": out.v_out[:, :Bt].cpu().numpy().view(np.uint16)}


@pytest.mark.parametrize("name", ["ragged", "tiles", "dups"])
def test_graph_replays_match_eager(torch_cuda, name):
    torch = torch_cuda
    from paper_2603_00188_amd import stlite as S
    from tests import gpu_harness as H
    from tests.test_gpu_parity import SMALL
    case = H.Case(SMALL[name])
    Bt = case.prob.total_budget
    eager = case.run()
    graph = S.capture_compress(case.prob, case.dq, case.dk, case.dv, case.out, alpha=case.w.alpha)
    want = _outputs(case.out, Bt)
    assert np.array_equal(want["kept"], eager["kept"])
    for rep in range(3):
        for t in (case.out.a_base, case.out.phi, case.out.kept, case.out.k_out):
            t.fill_(7)  # eager work between the replays, and outputs poisoned
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = _outputs(case.out, Bt)
        for key in want:
            assert np.array_equal(got[key], want[key]), (name, rep, key)
    # new keys written in place: the replay computes the pass over them
    case.dk.copy_(torch.flip(case.dk, dims=[2]))
    case.k = np.ascontiguousarray(case.k[:, :, ::-1])
    graph.replay()
    torch.cuda.synchronize()
    flipped = _outputs(case.out, Bt)
    ref = case.run()
    assert np.array_equal(flipped["kept"], ref["kept"]) and np.array_equal(flipped["k_out"], ref["k_out"])
    for layer in range(case.n_layers):
        for kv in range(case.w.n_kv_heads):
            for s in range(case.lay.n_seqs):
                H.compare_unit(case, ref, layer, kv, s)
