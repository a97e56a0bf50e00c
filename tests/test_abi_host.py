"""Host side of the C ABI, without a GPU: the library loads, exports every
function include/stlite.h declares, computes budgets exactly, and rejects
malformed problems before anything is launched."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2603_00188_amd import stlite as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "stlite.h")
HEADERS = sorted(os.path.join(ROOT, "include", f) for f in os.listdir(os.path.join(ROOT, "include"))
                 if f.endswith(".h"))

pytestmark = pytest.mark.skipif(not os.path.exists(S.LIB_PATH), reason="libstlite.so not built")

FAKE_DEV = 0x100000  # never dereferenced: validation reads only the host mirrors


def declared_functions():
    """Every function any include/*.h declares."""
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(stlite_[a-z_]+)\s*\(", src))
    return sorted(names)


def test_exports_match_header():
    lib = S.load()
    names = declared_functions()
    assert set(names) == set(S.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n
    assert lib.stlite_abi_version() == 2


def test_budget_exact():
    lib = S.load()
    assert lib.stlite_budget(2592, 76, 100) == 1969
    assert lib.stlite_budget(100, 29, 100) == 29
    assert lib.stlite_budget(150528, 1, 5) == 30105
    assert lib.stlite_budget(62720, 2, 5) == 25088
    assert lib.stlite_budget(7, 1, 1) == 7
    assert lib.stlite_budget(0, 1, 5) == 0
    assert lib.stlite_budget(10, 3, 2) == -1
    assert lib.stlite_budget(10, 0, 2) == -1
    assert lib.stlite_budget(-1, 1, 2) == -1
    big = 2 ** 40
    assert lib.stlite_budget(big, 2 ** 30 - 1, 2 ** 30) == (big * (2 ** 30 - 1)) // 2 ** 30


class HostProblem:
    """A _CProblem whose host mirrors are real and whose device pointers are fake."""

    def __init__(self, cu_seqlens, frames_per_seq, budgets, n_layers=2, n_q_heads=28, n_kv_heads=4,
                 window=8, head_dim=128):
        self.cu_seqlens = np.asarray(cu_seqlens, np.int32)
        self.cu_frames = np.asarray(np.concatenate([[0], np.cumsum([len(f) for f in frames_per_seq])]), np.int32)
        fm = [x for f in frames_per_seq for x in f]
        self.frame_meta = np.asarray(fm, np.int32).reshape(-1, 3) if fm else np.zeros((0, 3), np.int32)
        self.cu_budget = np.asarray(np.concatenate([[0], np.cumsum(budgets)]), np.int32)
        c = S._CProblem()
        c.n_layers, c.n_q_heads, c.n_kv_heads, c.head_dim = n_layers, n_q_heads, n_kv_heads, head_dim
        c.n_seqs, c.n_frames, c.window, c.reserved = len(cu_seqlens) - 1, len(fm), window, 0
        c.total_tokens = int(self.cu_seqlens[-1])
        c.total_budget = int(self.cu_budget[-1])
        c.cu_seqlens = c.cu_frames = c.cu_budget = FAKE_DEV
        c.frame_meta = FAKE_DEV if fm else None
        c.h_cu_seqlens = self.cu_seqlens.ctypes.data
        c.h_cu_frames = self.cu_frames.ctypes.data
        c.h_frame_meta = self.frame_meta.ctypes.data if fm else None
        c.h_cu_budget = self.cu_budget.ctypes.data
        self.c = c

    def validate(self):
        return S.load().stlite_validate(ctypes.byref(self.c))


def _one_huge_frame(p):
    # a single 2049 x 2048 frame (2^22 + 2048 patches) in a sequence long enough to hold it
    n = 2049 * 2048 + 40
    q = HostProblem([0, n], [[(0, 2049, 2048)]], [n // 5])
    p.__dict__.update(q.__dict__)


def good():
    # two sequences: [frame 4x5 | 10 text | frame 4x5 | 12 text], [30 text]
    return HostProblem([0, 72, 102], [[(0, 4, 5), (30, 4, 5)], []], [14, 6])


def test_valid_problem_and_workspace_sizes():
    p = good()
    assert p.validate() == S.OK, S.load().stlite_last_error()
    lib = S.load()
    n = ctypes.c_size_t(0)
    for call in range(6):
        assert lib.stlite_workspace_size(ctypes.byref(p.c), call, ctypes.byref(n)) == S.OK
        if call in (S.CALL_CSS_SALIENCY, S.CALL_COMPACT_KV):
            assert n.value == 0
        else:
            assert n.value > 0 and n.value % 256 == 0
    assert lib.stlite_workspace_size(ctypes.byref(p.c), 17, ctypes.byref(n)) == S.ERR_INVALID_ARG


@pytest.mark.parametrize("mutate, status, text", [
    (lambda p: setattr(p.c, "head_dim", 64), S.ERR_UNSUPPORTED, "head_dim"),
    (lambda p: setattr(p.c, "n_q_heads", 30), S.ERR_INVALID_ARG, "multiple"),
    (lambda p: setattr(p.c, "window", 0), S.ERR_INVALID_ARG, "window"),
    (lambda p: setattr(p.c, "window", 31), S.ERR_INVALID_ARG, "fewer than the window"),
    (lambda p: setattr(p.c, "window", 80), S.ERR_UNSUPPORTED, "G * window"),
    (lambda p: setattr(p.c, "reserved", 1), S.ERR_INVALID_ARG, "reserved"),
    (lambda p: setattr(p.c, "total_tokens", 103), S.ERR_INVALID_ARG, "total_tokens"),
    (lambda p: setattr(p.c, "total_budget", 19), S.ERR_INVALID_ARG, "total_budget"),
    (lambda p: setattr(p.c, "cu_seqlens", None), S.ERR_INVALID_ARG, "device"),
    (lambda p: setattr(p.c, "h_cu_budget", None), S.ERR_INVALID_ARG, "host"),
    (lambda p: p.frame_meta.__setitem__((1, 0), 10), S.ERR_INVALID_ARG, "overlaps"),
    (lambda p: p.frame_meta.__setitem__((1, 1), 9), S.ERR_INVALID_ARG, "leaves sequence"),
    (lambda p: p.frame_meta.__setitem__((0, 2), 0), S.ERR_INVALID_ARG, "empty grid"),
    (lambda p: _one_huge_frame(p), S.ERR_UNSUPPORTED, "at most 2^22"),
    (lambda p: p.cu_budget.__setitem__(1, 80), S.ERR_INVALID_ARG, "budget"),
    (lambda p: p.cu_frames.__setitem__(2, 1), S.ERR_INVALID_ARG, "cu_frames"),
])
def test_validation_rejects(mutate, status, text):
    p = good()
    mutate(p)
    assert p.validate() == status
    assert text in S.load().stlite_last_error().decode()


def test_last_error_is_per_thread():
    """Each host thread reads the message of its own last failure: several
    threads validate differently broken problems at once (ctypes releases the
    GIL during the calls) and each sees its own reason."""
    import threading
    cases = [(lambda p: setattr(p.c, "window", 0), "window"),
             (lambda p: setattr(p.c, "head_dim", 64), "head_dim"),
             (lambda p: setattr(p.c, "reserved", 1), "reserved"),
             (lambda p: setattr(p.c, "total_tokens", 103), "total_tokens")]
    lib = S.load()
    seen, errors = {}, []
    start = threading.Barrier(len(cases))

    def run(i, mutate, text):
        p = good()
        mutate(p)
        start.wait()
        for _ in range(200):
            if p.validate() == S.OK:
                errors.append((i, "validated"))
                return
            msg = lib.stlite_last_error().decode()
            if text not in msg:
                errors.append((i, msg))
                return
        seen[i] = text

    threads = [threading.Thread(target=run, args=(i, m, t)) for i, (m, t) in enumerate(cases)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors and len(seen) == len(cases), errors


def test_frame_of_exactly_2_22_patches_is_accepted():
    n = 2048 * 2048 + 40
    p = HostProblem([0, n], [[(0, 2048, 2048)]], [n // 5])
    assert p.validate() == S.OK, S.load().stlite_last_error()


def test_calls_fail_before_launch():
    lib = S.load()
    p = good()
    ref = ctypes.byref(p.c)
    # workspace missing / too small: nothing is enqueued, no GPU is touched
    assert lib.stlite_score_window(ref, FAKE_DEV, FAKE_DEV, FAKE_DEV, None, 0, None) == S.ERR_WORKSPACE
    assert lib.stlite_select_topk(ref, FAKE_DEV, None, None, 1.0, FAKE_DEV, None, FAKE_DEV, 16,
                                  None) == S.ERR_WORKSPACE
    n = ctypes.c_size_t(0)
    lib.stlite_workspace_size(ref, S.CALL_SELECT_TOPK, ctypes.byref(n))
    assert lib.stlite_select_topk(ref, FAKE_DEV, None, None, -1.0, FAKE_DEV, None, FAKE_DEV, n.value,
                                  None) == S.ERR_INVALID_ARG
    assert lib.stlite_select_topk(ref, FAKE_DEV, None, None, float("nan"), FAKE_DEV, None, FAKE_DEV,
                                  n.value, None) == S.ERR_INVALID_ARG
    assert lib.stlite_css_saliency(ref, None, None, FAKE_DEV, None) == S.ERR_INVALID_ARG
    assert lib.stlite_compact_kv(ref, FAKE_DEV + 8, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV,
                                 None) == S.ERR_INVALID_ARG
    assert lib.stlite_tsg_gate(ref, FAKE_DEV, None, None, None, None, 0, None) == S.ERR_WORKSPACE
    assert lib.stlite_tsg_rho(ref, FAKE_DEV, FAKE_DEV, None, 0, None) == S.ERR_WORKSPACE
    lib.stlite_workspace_size(ref, S.CALL_TSG_RHO, ctypes.byref(n))
    assert n.value > 0
    assert lib.stlite_tsg_rho(ref, FAKE_DEV, None, FAKE_DEV, n.value, None) == S.ERR_INVALID_ARG
    p.c.head_dim = 96
    assert lib.stlite_css_saliency(ref, FAKE_DEV, FAKE_DEV, FAKE_DEV, None) == S.ERR_UNSUPPORTED
    assert lib.stlite_status_string(S.ERR_HIP) == b"STLITE_ERR_HIP"


def test_budgets_helper_matches_oracle():
    from oracle import stlite_oracle as O
    cu = np.array([0, 912, 4304, 5000])
    got = S.budgets(cu, 1, 5)
    want = np.concatenate([[0], np.cumsum([O.budget(int(l), 1, 5) for l in np.diff(cu)])])
    assert got.tolist() == want.tolist()


def test_decode_workspace_and_rejections():
    """Decode attention: workspace per cache, and every malformed call fails
    before anything is enqueued."""
    lib = S.load()
    p = good()
    ref = ctypes.byref(p.c)
    n_full, n_comp = ctypes.c_size_t(0), ctypes.c_size_t(0)
    assert lib.stlite_workspace_size(ref, S.CALL_DECODE_FULL, ctypes.byref(n_full)) == S.OK
    assert lib.stlite_workspace_size(ref, S.CALL_DECODE_COMPACT, ctypes.byref(n_comp)) == S.OK
    assert n_full.value > 0 and n_full.value % 256 == 0 and 0 < n_comp.value <= n_full.value
    call = lambda cache, q, k, v, out, ws, nb: lib.stlite_decode_attention(ref, cache, q, k, v, out, ws, nb, None)
    assert call(S.CACHE_FULL, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV, None, 0) == S.ERR_WORKSPACE
    assert call(S.CACHE_FULL, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV, n_full.value - 1) == S.ERR_WORKSPACE
    assert call(2, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV, n_full.value) == S.ERR_INVALID_ARG
    assert call(S.CACHE_FULL, None, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV, n_full.value) == S.ERR_INVALID_ARG
    assert call(S.CACHE_COMPACT, FAKE_DEV, FAKE_DEV + 4, FAKE_DEV, FAKE_DEV, FAKE_DEV,
                n_comp.value) == S.ERR_INVALID_ARG
    # more than 16 query heads per kv head
    wide = HostProblem([0, 72, 102], [[(0, 4, 5), (30, 4, 5)], []], [14, 6], n_q_heads=68, n_kv_heads=4, window=4)
    nw = ctypes.c_size_t(0)
    assert lib.stlite_workspace_size(ctypes.byref(wide.c), S.CALL_DECODE_FULL, ctypes.byref(nw)) == S.OK
    assert lib.stlite_decode_attention(ctypes.byref(wide.c), S.CACHE_FULL, FAKE_DEV, FAKE_DEV, FAKE_DEV, FAKE_DEV,
                                       FAKE_DEV, nw.value, None) == S.ERR_UNSUPPORTED


def test_tsg_variant_rejections():
    """The similarity and fixed-threshold gate entry points reject malformed
    calls before anything is enqueued."""
    lib = S.load()
    p = good()
    ref = ctypes.byref(p.c)
    n = ctypes.c_size_t(0)
    assert lib.stlite_workspace_size(ref, S.CALL_TSG_RHO, ctypes.byref(n)) == S.OK
    sim = lambda s, k, rho, ws, nb: lib.stlite_tsg_similarity(ref, s, k, rho, ws, nb, None)
    assert sim(3, FAKE_DEV, FAKE_DEV, FAKE_DEV, n.value) == S.ERR_INVALID_ARG
    assert sim(-1, FAKE_DEV, FAKE_DEV, FAKE_DEV, n.value) == S.ERR_INVALID_ARG
    assert sim(S.SIM_DOT, FAKE_DEV, FAKE_DEV, FAKE_DEV, n.value - 1) == S.ERR_WORKSPACE
    assert sim(S.SIM_NEG_L2, None, FAKE_DEV, FAKE_DEV, n.value) == S.ERR_INVALID_ARG
    assert sim(S.SIM_NEG_L2, FAKE_DEV, None, FAKE_DEV, n.value) == S.ERR_INVALID_ARG
    assert sim(S.SIM_DOT, FAKE_DEV + 2, FAKE_DEV, FAKE_DEV, n.value) == S.ERR_INVALID_ARG
    fixed = lambda rho, tau, gate: lib.stlite_tsg_fixed_gate(ref, rho, tau, gate, None)
    assert fixed(None, 0.85, FAKE_DEV) == S.ERR_INVALID_ARG
    assert fixed(FAKE_DEV, 0.85, None) == S.ERR_INVALID_ARG
    assert fixed(FAKE_DEV, float("nan"), FAKE_DEV) == S.ERR_INVALID_ARG
    assert b"NaN" in lib.stlite_last_error()
    bad = good()
    bad.c.n_layers = 0
    assert lib.stlite_tsg_fixed_gate(ctypes.byref(bad.c), FAKE_DEV, 0.85, FAKE_DEV, None) != S.OK


def test_css_nbhd_rejections():
    lib = S.load()
    p = good()
    ref = ctypes.byref(p.c)
    for bad in (0, 1, 2, 4, 6, 11, -3):
        assert lib.stlite_css_saliency_nbhd(ref, bad, FAKE_DEV, FAKE_DEV, None) == S.ERR_INVALID_ARG
    assert b"nbhd" in lib.stlite_last_error()
    assert lib.stlite_css_saliency_nbhd(ref, 5, None, FAKE_DEV, None) == S.ERR_INVALID_ARG
    assert lib.stlite_css_saliency_nbhd(ref, 9, FAKE_DEV + 8, FAKE_DEV, None) == S.ERR_INVALID_ARG


def test_mean_attention_rejections():
    lib = S.load()
    p = good()
    ref = ctypes.byref(p.c)
    for bad in (0, 2, 8, -1, 257, 1001):
        assert lib.stlite_mean_attention(ref, FAKE_DEV, bad, FAKE_DEV + 4096, None) == S.ERR_INVALID_ARG
    assert b"width" in lib.stlite_last_error()
    assert lib.stlite_mean_attention(ref, None, 7, FAKE_DEV, None) == S.ERR_INVALID_ARG
    assert lib.stlite_mean_attention(ref, FAKE_DEV, 7, None, None) == S.ERR_INVALID_ARG
    assert lib.stlite_mean_attention(ref, FAKE_DEV, 7, FAKE_DEV, None) == S.ERR_INVALID_ARG
    assert b"alias" in lib.stlite_last_error()
    bad = good()
    bad.c.n_layers = 0
    assert lib.stlite_mean_attention(ctypes.byref(bad.c), FAKE_DEV, 7, FAKE_DEV + 4096, None) != S.OK


def test_kept_overlap_rejections():
    lib = S.load()
    p = good()
    ref = ctypes.byref(p.c)
    assert lib.stlite_kept_overlap(ref, FAKE_DEV, FAKE_DEV, None, None) == S.ERR_INVALID_ARG
    assert lib.stlite_kept_overlap(ref, None, FAKE_DEV, FAKE_DEV, None) == S.ERR_INVALID_ARG
    assert lib.stlite_kept_overlap(ref, FAKE_DEV, None, FAKE_DEV, None) == S.ERR_INVALID_ARG
    bad = good()
    bad.c.n_seqs = 0
    assert lib.stlite_kept_overlap(ctypes.byref(bad.c), FAKE_DEV, FAKE_DEV, FAKE_DEV, None) != S.OK


def test_probe_rejections():
    lib = S.load()
    assert lib.stlite_probe_mfma(4, FAKE_DEV, FAKE_DEV, 1, 1, None) == S.ERR_INVALID_ARG
    assert lib.stlite_probe_mfma(-1, FAKE_DEV, FAKE_DEV, 1, 1, None) == S.ERR_INVALID_ARG
    assert lib.stlite_probe_mfma(0, None, FAKE_DEV, 1, 1, None) == S.ERR_INVALID_ARG
    assert lib.stlite_probe_mfma(1, FAKE_DEV, None, 1, 1, None) == S.ERR_INVALID_ARG
    assert lib.stlite_probe_mfma(0, FAKE_DEV, FAKE_DEV, 0, 1, None) == S.ERR_INVALID_ARG
    assert lib.stlite_probe_mfma(1, FAKE_DEV, FAKE_DEV, 4, 0, None) == S.ERR_INVALID_ARG
    # the read probe: NULL pointers, an empty, unaligned or ragged source, no work-group
    assert lib.stlite_probe_read(None, 1024, FAKE_DEV, 1, 0, None) == S.ERR_INVALID_ARG
    assert lib.stlite_probe_read(FAKE_DEV, 1024, None, 1, 1, None) == S.ERR_INVALID_ARG
    assert lib.stlite_probe_read(FAKE_DEV, 0, FAKE_DEV, 1, 0, None) == S.ERR_INVALID_ARG
    assert lib.stlite_probe_read(FAKE_DEV, 1000, FAKE_DEV, 1, 0, None) == S.ERR_INVALID_ARG
    assert lib.stlite_probe_read(FAKE_DEV + 8, 1024, FAKE_DEV, 1, 0, None) == S.ERR_INVALID_ARG
    assert lib.stlite_probe_read(FAKE_DEV, 1024, FAKE_DEV, 0, 0, None) == S.ERR_INVALID_ARG



def test_concat_rejections_and_workspace():
    lib = S.load()
    p = good()   # 4 kv heads
    ref = ctypes.byref(p.c)
    n = ctypes.c_size_t(0)
    assert lib.stlite_workspace_size(ref, S.CALL_TSG_RHO_CONCAT, ctypes.byref(n)) == S.OK and n.value > 0
    assert lib.stlite_tsg_rho_concat(ref, FAKE_DEV, FAKE_DEV, FAKE_DEV, n.value - 1, None) == S.ERR_WORKSPACE
    assert lib.stlite_tsg_rho_concat(ref, None, FAKE_DEV, FAKE_DEV, n.value, None) == S.ERR_INVALID_ARG
    assert lib.stlite_css_saliency_concat(ref, FAKE_DEV, None, None) == S.ERR_INVALID_ARG
    assert lib.stlite_layer_mean(ref, None, FAKE_DEV, None) == S.ERR_INVALID_ARG
    three = HostProblem([0, 72, 102], [[(0, 4, 5), (30, 4, 5)], []], [14, 6], n_q_heads=27, n_kv_heads=3)
    r3 = ctypes.byref(three.c)
    n3 = ctypes.c_size_t(0)
    assert lib.stlite_workspace_size(r3, S.CALL_TSG_RHO_CONCAT, ctypes.byref(n3)) == S.OK
    assert lib.stlite_tsg_rho_concat(r3, FAKE_DEV, FAKE_DEV, FAKE_DEV, n3.value, None) == S.ERR_UNSUPPORTED
    assert lib.stlite_css_saliency_concat(r3, FAKE_DEV, FAKE_DEV, None) == S.ERR_UNSUPPORTED


def test_noalloc_select_rejects_oversized_problem():
    """stlite_select_topk_noalloc refuses a problem whose selection workspace
    exceeds its static buffer, before anything is enqueued (no GPU touched):
    28 layers x 4 kv heads over one 150,528-token sequence."""
    lib = S.load()
    L = 150528
    p = HostProblem([0, L], [[]], [L // 5], n_layers=28)
    n = ctypes.c_size_t(0)
    assert lib.stlite_workspace_size(ctypes.byref(p.c), S.CALL_SELECT_TOPK, ctypes.byref(n)) == S.OK
    assert n.value > S.NOALLOC_SCRATCH_BYTES
    st = lib.stlite_select_topk_noalloc(ctypes.byref(p.c), FAKE_DEV, None, None, 1.0, FAKE_DEV, None, None)
    assert st == S.ERR_WORKSPACE
    assert "static buffer" in lib.stlite_last_error().decode()
    p.c.head_dim = 64   # an invalid problem is reported as such first
    st = lib.stlite_select_topk_noalloc(ctypes.byref(p.c), FAKE_DEV, None, None, 1.0, FAKE_DEV, None, None)
    assert st == S.ERR_UNSUPPORTED
