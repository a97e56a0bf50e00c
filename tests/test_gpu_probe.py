"""GPU checks of the measurement probes (not part of the method): the read
probe touches every 16-byte word of its source exactly once, and the matrix
core probes run to completion with finite results."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def test_read_probe_reads_every_word_once(torch_cuda):
    """Lane l of the read probe XORs words l, l + stride, ... (stride = all
    lanes of the grid): its sink entry must equal that XOR computed on the
    host, for a source whose last stride is partial, under both cache
    policies."""
    torch = torch_cuda
    from paper_2603_00188_amd import stlite as S
    groups = 3
    stride = groups * 256
    n16 = stride * 7 + 123
    words = np.random.default_rng(3).integers(0, 2 ** 32, size=(n16, 4), dtype=np.uint32)
    src = torch.from_numpy(words.view(np.int32)).cuda()
    sink = torch.empty(stride, dtype=torch.float32, device="cuda")
    want = np.zeros(stride, np.uint32)
    for lane in range(stride):
        x = np.bitwise_xor.reduce(words[lane::stride], axis=0)
        want[lane] = x[0] ^ x[1] ^ x[2] ^ x[3]
    for nontemporal in (False, True):
        sink.fill_(0.0)
        S.stlite_probe_read(src, n16 * 16, sink, groups, nontemporal)
        torch.cuda.synchronize()
        got = sink.cpu().numpy().view(np.uint32)
        assert np.array_equal(got, want), nontemporal


def test_mfma_probes_finish_with_finite_sums(torch_cuda):
    torch = torch_cuda
    from paper_2603_00188_amd import stlite as S
    groups = 8
    gen = torch.Generator().manual_seed(0)
    ops = (torch.randn(groups * 256 * 128, generator=gen) * 0.25).to(torch.bfloat16).cuda().view(torch.int16)
    sink = torch.full((groups * 256,), float("nan"), dtype=torch.float32, device="cuda")
    for shape in (S.PROBE_MFMA_16X16X32, S.PROBE_MFMA_32X32X16, S.PROBE_MFMA_32X32X16_EXP2,
                  S.PROBE_MFMA_16X16X32_EXP2):
        sink.fill_(float("nan"))
        S.stlite_probe_mfma(shape, ops, sink, groups, 4)
        torch.cuda.synchronize()
        assert torch.isfinite(sink).all(), shape
