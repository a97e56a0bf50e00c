"""GPU parity of the Mean-Attention base prior (the paper's base-scoring
ablation; reading R-mean: A_base pooled over `width` positions along each
sequence, zero padding, divisor width) and of the whole pass ranking on it,
against the fp64 oracle (compress_unit with mean_width).

Tolerances: A_mean |d| <= 1e-3 |ref| (a sum of positive A_base terms, each
within that bound, plus fp32 additions); the kept set, the gate and the
compacted rows under the rules of the pass (tests/gpu_harness.py).
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
    from tests import gpu_harness as H
    from tests.test_gpu_parity import SMALL
    return H, SMALL


def _all_units(H, case, width):
    res = case.run(mean_width=width)
    for layer in range(case.n_layers):
        for kv in range(case.w.n_kv_heads):
            for s in range(case.lay.n_seqs):
                H.compare_unit(case, res, layer, kv, s, ref=case.oracle(layer, kv, s, mean_width=width))
    return res


@pytest.mark.parametrize("width", [3, 7, 31])
def test_mean_attention_config0_all_units(torch_cuda, width):
    H, _ = _mods()
    case = H.Case(W.config(0))
    _all_units(H, case, width)


def test_mean_attention_config1_all_units(torch_cuda):
    H, _ = _mods()
    case = H.Case(W.config(1))
    H.log("mean attention: single step, 112 units, width 7")
    _all_units(H, case, 7)


@pytest.mark.parametrize("name,width", [("ragged", 7), ("ragged", 255), ("tiles", 9), ("dups", 5),
                                        ("beta_tiny", 3)])
def test_mean_attention_small(torch_cuda, name, width):
    """Ragged packed batches (text-only sequences, sequences shorter than the
    pooling window, a 1 x 1 frame) and the widest window."""
    H, SMALL = _mods()
    case = H.Case(SMALL[name])
    _all_units(H, case, width)


def test_mean_attention_width_one_is_a_copy(torch_cuda):
    """Width 1 writes A_base bit for bit, and the pass then keeps exactly what
    the window prior keeps."""
    H, SMALL = _mods()
    case = H.Case(SMALL["tiles"])
    plain = case.run()
    one = case.run(mean_width=1)
    assert np.array_equal(one["a_mean"], one["a_base"])
    assert np.array_equal(one["kept"], plain["kept"])


@pytest.mark.timeout(900)
def test_mean_attention_trajectory_sampled(torch_cuda):
    """The 150,528-token trajectory in the benchmark's launch configuration, on
    sampled units."""
    H, _ = _mods()
    w = W.config(3)
    H.log(f"mean attention trajectory: generate L={w.total_tokens} x {w.n_layers} layers")
    case = H.Case(w)
    res = case.run(mean_width=7)
    for layer, kv in ((0, 0), (13, 2), (27, 3)):
        st = H.compare_unit(case, res, layer, kv, 0, ref=case.oracle(layer, kv, 0, mean_width=7))
        H.log(f"mean attention trajectory unit ({layer},{kv}): {st}")
