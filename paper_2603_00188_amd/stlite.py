"""Python binding of libstlite (ctypes; argument marshalling only).

Every function here forwards to the C entry point of the same name declared in
include/stlite.h; all arithmetic runs in the library's gfx950 kernels.  PyTorch
provides device memory and the stream.  There is no fallback: if the library
is not built, ``load()`` raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libstlite.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = range(5)
(CALL_SCORE_WINDOW, CALL_TSG_GATE, CALL_CSS_SALIENCY, CALL_SELECT_TOPK, CALL_COMPACT_KV, CALL_TSG_THRESHOLD,
 CALL_TSG_RHO, CALL_DECODE_FULL, CALL_DECODE_COMPACT, CALL_TSG_RHO_CONCAT) = range(10)
CACHE_FULL, CACHE_COMPACT = 0, 1
SIM_COSINE, SIM_DOT, SIM_NEG_L2 = 0, 1, 2

EXPORTS = (
    "stlite_abi_version", "stlite_status_string", "stlite_last_error", "stlite_budget",
    "stlite_validate", "stlite_workspace_size", "stlite_score_window", "stlite_css_saliency",
    "stlite_tsg_gate", "stlite_tsg_rho", "stlite_tsg_threshold", "stlite_select_topk", "stlite_compact_kv",
    "stlite_decode_attention", "stlite_tsg_similarity", "stlite_tsg_fixed_gate",
    "stlite_css_saliency_nbhd", "stlite_kept_overlap", "stlite_probe_mfma", "stlite_probe_read",
    "stlite_layer_mean", "stlite_tsg_rho_concat", "stlite_css_saliency_concat", "stlite_compact_kv_layer",
    "stlite_select_topk_noalloc", "stlite_mean_attention",
)


class StliteError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status}: {detail}")
        self.status = status


class _CProblem(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
        ("n_seqs", ctypes.c_int32), ("n_frames", ctypes.c_int32),
        ("window", ctypes.c_int32), ("reserved", ctypes.c_int32),
        ("total_tokens", ctypes.c_int64), ("total_budget", ctypes.c_int64),
        ("cu_seqlens", ctypes.c_void_p), ("cu_frames", ctypes.c_void_p),
        ("frame_meta", ctypes.c_void_p), ("cu_budget", ctypes.c_void_p),
        ("h_cu_seqlens", ctypes.c_void_p), ("h_cu_frames", ctypes.c_void_p),
        ("h_frame_meta", ctypes.c_void_p), ("h_cu_budget", ctypes.c_void_p),
    ]


_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libstlite.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2603_00188_amd.build`")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER(_CProblem)
    vp, sz, i64, f32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int64, ctypes.c_float
    st = ctypes.c_int
    sig = {
        "stlite_abi_version": (ctypes.c_int32, []),
        "stlite_status_string": (ctypes.c_char_p, [st]),
        "stlite_last_error": (ctypes.c_char_p, []),
        "stlite_budget": (i64, [i64, i64, i64]),
        "stlite_validate": (st, [P]),
        "stlite_workspace_size": (st, [P, st, ctypes.POINTER(sz)]),
        "stlite_score_window": (st, [P, vp, vp, vp, vp, sz, vp]),
        "stlite_css_saliency": (st, [P, vp, vp, vp, vp]),
        "stlite_tsg_gate": (st, [P, vp, vp, vp, vp, vp, sz, vp]),
        "stlite_tsg_rho": (st, [P, vp, vp, vp, sz, vp]),
        "stlite_tsg_threshold": (st, [P, vp, vp, vp, vp, sz, vp]),
        "stlite_select_topk": (st, [P, vp, vp, vp, f32, vp, vp, vp, sz, vp]),
        "stlite_compact_kv": (st, [P, vp, vp, vp, vp, vp, vp]),
        "stlite_decode_attention": (st, [P, st, vp, vp, vp, vp, vp, sz, vp]),
        "stlite_tsg_similarity": (st, [P, st, vp, vp, vp, sz, vp]),
        "stlite_tsg_fixed_gate": (st, [P, vp, f32, vp, vp]),
        "stlite_css_saliency_nbhd": (st, [P, ctypes.c_int32, vp, vp, vp]),
        "stlite_kept_overlap": (st, [P, vp, vp, vp, vp]),
        "stlite_probe_mfma": (st, [st, vp, vp, ctypes.c_int32, ctypes.c_int32, vp]),
        "stlite_probe_read": (st, [vp, sz, vp, ctypes.c_int32, ctypes.c_int32, vp]),
        "stlite_layer_mean": (st, [P, vp, vp, vp]),
        "stlite_mean_attention": (st, [P, vp, ctypes.c_int32, vp, vp]),
        "stlite_tsg_rho_concat": (st, [P, vp, vp, vp, sz, vp]),
        "stlite_css_saliency_concat": (st, [P, vp, vp, vp]),
        "stlite_compact_kv_layer": (st, [P, vp, vp, vp, vp, vp, vp]),
        "stlite_select_topk_noalloc": (st, [P, vp, vp, vp, f32, vp, vp, vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int, where: str):
    if status != OK:
        raise StliteError(status, where, load().stlite_last_error().decode())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _nbytes(t) -> int:
    return 0 if t is None else t.numel() * t.element_size()


class Problem:
    """An stlite_problem plus the host and device copies of its layout arrays."""

    def __init__(self, n_layers: int, n_q_heads: int, n_kv_heads: int, window: int,
                 cu_seqlens, cu_frames, frame_meta, cu_budget, head_dim: int = 128,
                 device="cuda"):
        import torch
        self.h = {
            "cu_seqlens": np.ascontiguousarray(cu_seqlens, dtype=np.int32),
            "cu_frames": np.ascontiguousarray(cu_frames, dtype=np.int32),
            "frame_meta": np.ascontiguousarray(np.asarray(frame_meta, dtype=np.int32).reshape(-1, 3)),
            "cu_budget": np.ascontiguousarray(cu_budget, dtype=np.int32),
        }
        self.d = {k: torch.from_numpy(v.reshape(-1).copy()).to(device) for k, v in self.h.items()}
        n_seqs = len(self.h["cu_seqlens"]) - 1
        c = _CProblem()
        c.n_layers, c.n_q_heads, c.n_kv_heads, c.head_dim = n_layers, n_q_heads, n_kv_heads, head_dim
        c.n_seqs, c.n_frames, c.window, c.reserved = n_seqs, len(self.h["frame_meta"]), window, 0
        c.total_tokens = int(self.h["cu_seqlens"][-1])
        c.total_budget = int(self.h["cu_budget"][-1])
        for k in self.h:
            setattr(c, k, self.d[k].data_ptr() if self.d[k].numel() else None)
            setattr(c, "h_" + k, self.h[k].ctypes.data if self.h[k].size else None)
        self.c = c
        self.n_layers, self.n_q_heads, self.n_kv_heads, self.window = n_layers, n_q_heads, n_kv_heads, window
        self.n_seqs = n_seqs
        self.total_tokens = c.total_tokens
        self.total_budget = c.total_budget
        self.units = n_layers * n_kv_heads

    @property
    def ref(self):
        return ctypes.byref(self.c)

    def workspace_size(self, call: int) -> int:
        n = ctypes.c_size_t(0)
        _check(load().stlite_workspace_size(self.ref, call, ctypes.byref(n)), "stlite_workspace_size")
        return n.value


def budgets(cu_seqlens, beta_num: int, beta_den: int) -> np.ndarray:
    """cu_budget prefix sums with B_s = stlite_budget(L_s, beta)."""
    lib = load()
    L = np.diff(np.asarray(cu_seqlens, dtype=np.int64))
    B = [lib.stlite_budget(int(l), int(beta_num), int(beta_den)) for l in L]
    if any(b < 0 for b in B):
        raise ValueError("invalid budget ratio")
    return np.concatenate([[0], np.cumsum(B)]).astype(np.int32)


def stlite_budget(L: int, beta_num: int, beta_den: int) -> int:
    return load().stlite_budget(L, beta_num, beta_den)


def stlite_validate(p: Problem) -> None:
    _check(load().stlite_validate(p.ref), "stlite_validate")


def stlite_score_window(p: Problem, q_win, k, a_base, workspace, stream=None) -> None:
    _check(load().stlite_score_window(p.ref, _ptr(q_win), _ptr(k), _ptr(a_base), _ptr(workspace),
                                      _nbytes(workspace), _stream(stream)), "stlite_score_window")


def stlite_css_saliency(p: Problem, k, phi, gate=None, stream=None) -> None:
    _check(load().stlite_css_saliency(p.ref, _ptr(k), _ptr(gate), _ptr(phi), _stream(stream)),
           "stlite_css_saliency")


def stlite_css_saliency_nbhd(p: Problem, nbhd: int, k, phi, stream=None) -> None:
    _check(load().stlite_css_saliency_nbhd(p.ref, int(nbhd), _ptr(k), _ptr(phi), _stream(stream)),
           "stlite_css_saliency_nbhd")


def stlite_tsg_gate(p: Problem, k, rho, tau, gate, workspace, stream=None) -> None:
    _check(load().stlite_tsg_gate(p.ref, _ptr(k), _ptr(rho), _ptr(tau), _ptr(gate), _ptr(workspace),
                                  _nbytes(workspace), _stream(stream)), "stlite_tsg_gate")


def stlite_tsg_rho(p: Problem, k, rho, workspace, stream=None) -> None:
    _check(load().stlite_tsg_rho(p.ref, _ptr(k), _ptr(rho), _ptr(workspace), _nbytes(workspace), _stream(stream)),
           "stlite_tsg_rho")


def stlite_tsg_similarity(p: Problem, sim: int, k, rho, workspace, stream=None) -> None:
    _check(load().stlite_tsg_similarity(p.ref, int(sim), _ptr(k), _ptr(rho), _ptr(workspace), _nbytes(workspace),
                                        _stream(stream)), "stlite_tsg_similarity")


def stlite_tsg_fixed_gate(p: Problem, rho, tau: float, gate, stream=None) -> None:
    _check(load().stlite_tsg_fixed_gate(p.ref, _ptr(rho), float(tau), _ptr(gate), _stream(stream)),
           "stlite_tsg_fixed_gate")


def stlite_tsg_threshold(p: Problem, rho, tau, gate, workspace, stream=None) -> None:
    _check(load().stlite_tsg_threshold(p.ref, _ptr(rho), _ptr(tau), _ptr(gate), _ptr(workspace),
                                       _nbytes(workspace), _stream(stream)), "stlite_tsg_threshold")


def stlite_select_topk(p: Problem, a_base, phi, gate, alpha: float, kept, score, workspace,
                       stream=None) -> None:
    _check(load().stlite_select_topk(p.ref, _ptr(a_base), _ptr(phi), _ptr(gate), float(alpha), _ptr(kept),
                                     _ptr(score), _ptr(workspace), _nbytes(workspace), _stream(stream)),
           "stlite_select_topk")


def stlite_select_topk_noalloc(p: Problem, a_base, phi, gate, alpha: float, kept, score, stream=None) -> None:
    _check(load().stlite_select_topk_noalloc(p.ref, _ptr(a_base), _ptr(phi), _ptr(gate), float(alpha), _ptr(kept),
                                             _ptr(score), _stream(stream)), "stlite_select_topk_noalloc")


NOALLOC_SCRATCH_BYTES = 32 << 20   # STLITE_NOALLOC_SCRATCH_BYTES


def stlite_compact_kv(p: Problem, k, v, kept, k_out, v_out, stream=None) -> None:
    _check(load().stlite_compact_kv(p.ref, _ptr(k), _ptr(v), _ptr(kept), _ptr(k_out), _ptr(v_out),
                                    _stream(stream)), "stlite_compact_kv")


def stlite_kept_overlap(p: Problem, kept_a, kept_b, hits, stream=None) -> None:
    _check(load().stlite_kept_overlap(p.ref, _ptr(kept_a), _ptr(kept_b), _ptr(hits), _stream(stream)),
           "stlite_kept_overlap")


def stlite_decode_attention(p: Problem, cache: int, q_dec, k, v, out, workspace, stream=None) -> None:
    _check(load().stlite_decode_attention(p.ref, int(cache), _ptr(q_dec), _ptr(k), _ptr(v), _ptr(out),
                                          _ptr(workspace), _nbytes(workspace), _stream(stream)),
           "stlite_decode_attention")


def decode(p: Problem, q_dec, k, v, cache: int, out=None, workspace=None, stream=None):
    """Decode attention over the full (CACHE_FULL: k, v) or compacted
    (CACHE_COMPACT: k_out, v_out) cache; returns out [layers, seqs, Hq, 128] fp32."""
    import torch
    if out is None:
        out = torch.empty((p.n_layers, p.n_seqs, p.n_q_heads, 128), dtype=torch.float32, device=q_dec.device)
    if workspace is None:
        n = p.workspace_size(CALL_DECODE_COMPACT if cache == CACHE_COMPACT else CALL_DECODE_FULL)
        workspace = torch.empty(max(n, 256), dtype=torch.uint8, device=q_dec.device)
    stlite_decode_attention(p, cache, q_dec, k, v, out, workspace, stream)
    return out


class Buffers:
    """Device outputs and workspaces for one problem (allocated once, reused).

    ``ws`` serves the calls on the main stream; ``ws_tsg`` is a second
    workspace for the TSG calls, so that they can run on a side stream while
    the window scoring uses ``ws``.
    """

    def __init__(self, p: Problem, device="cuda", keep_stages: bool = True):
        import torch
        U, L, Bt = p.units, p.total_tokens, p.total_budget
        f32 = dict(dtype=torch.float32, device=device)
        self.a_base = torch.empty((U, L), **f32)
        self.phi = torch.empty((U, L), **f32)
        self.rho = torch.empty((U, L), **f32) if keep_stages else None
        self.tau = torch.empty((U, p.n_seqs), **f32) if keep_stages else None
        self.score = torch.empty((U, L), **f32) if keep_stages else None
        self.gate = torch.empty((U, L), dtype=torch.uint8, device=device)
        self.kept = torch.empty((U, max(Bt, 1)), dtype=torch.int32, device=device)
        self.k_out = torch.empty((U, max(Bt, 1), 128), dtype=torch.int16, device=device)
        self.v_out = torch.empty((U, max(Bt, 1), 128), dtype=torch.int16, device=device)
        ws = max(p.workspace_size(c) for c in (CALL_SCORE_WINDOW, CALL_CSS_SALIENCY, CALL_SELECT_TOPK,
                                               CALL_COMPACT_KV))
        ws_tsg = max(p.workspace_size(c) for c in (CALL_TSG_GATE, CALL_TSG_RHO, CALL_TSG_THRESHOLD))
        self.ws = torch.empty(max(ws, 256), dtype=torch.uint8, device=device)
        self.ws_tsg = torch.empty(max(ws_tsg, 256), dtype=torch.uint8, device=device)
        # side streams at the default priority
        self.side = (torch.cuda.Stream(device=device), torch.cuda.Stream(device=device))


PROBE_MFMA_16X16X32, PROBE_MFMA_32X32X16, PROBE_MFMA_32X32X16_EXP2, PROBE_MFMA_16X16X32_EXP2 = 0, 1, 2, 3
PROBE_FLOPS = {PROBE_MFMA_16X16X32: 16 * 16 * 32 * 2, PROBE_MFMA_32X32X16: 32 * 32 * 16 * 2,
               PROBE_MFMA_32X32X16_EXP2: 32 * 32 * 16 * 2, PROBE_MFMA_16X16X32_EXP2: 16 * 16 * 32 * 2}
PROBE_MFMAS_PER_ITER = {PROBE_MFMA_16X16X32: 8, PROBE_MFMA_32X32X16: 8, PROBE_MFMA_32X32X16_EXP2: 8,
                        PROBE_MFMA_16X16X32_EXP2: 16}


def stlite_probe_mfma(shape: int, operands, sink, n_groups: int, iters: int, stream=None) -> None:
    _check(load().stlite_probe_mfma(int(shape), _ptr(operands), _ptr(sink), int(n_groups), int(iters),
                                    _stream(stream)), "stlite_probe_mfma")


def stlite_probe_read(src, nbytes: int, sink, n_groups: int, nontemporal: bool, stream=None) -> None:
    _check(load().stlite_probe_read(_ptr(src), int(nbytes), _ptr(sink), int(n_groups), 1 if nontemporal else 0,
                                    _stream(stream)), "stlite_probe_read")


def stlite_mean_attention(p: Problem, a_base, width: int, a_mean, stream=None) -> None:
    _check(load().stlite_mean_attention(p.ref, _ptr(a_base), int(width), _ptr(a_mean), _stream(stream)),
           "stlite_mean_attention")


def stlite_layer_mean(p: Problem, a_base, a_layer, stream=None) -> None:
    _check(load().stlite_layer_mean(p.ref, _ptr(a_base), _ptr(a_layer), _stream(stream)), "stlite_layer_mean")


def stlite_tsg_rho_concat(p: Problem, k, rho_layer, workspace, stream=None) -> None:
    _check(load().stlite_tsg_rho_concat(p.ref, _ptr(k), _ptr(rho_layer), _ptr(workspace), _nbytes(workspace),
                                        _stream(stream)), "stlite_tsg_rho_concat")


def stlite_css_saliency_concat(p: Problem, k, phi_layer, stream=None) -> None:
    _check(load().stlite_css_saliency_concat(p.ref, _ptr(k), _ptr(phi_layer), _stream(stream)),
           "stlite_css_saliency_concat")


def stlite_compact_kv_layer(p: Problem, k, v, kept_layer, k_out, v_out, stream=None) -> None:
    _check(load().stlite_compact_kv_layer(p.ref, _ptr(k), _ptr(v), _ptr(kept_layer), _ptr(k_out), _ptr(v_out),
                                          _stream(stream)), "stlite_compact_kv_layer")


def layer_problem(p: Problem) -> Problem:
    """The layer-level view of p for the concatenated key space: the same layout
    and budgets, one unit per layer (n_kv_heads = n_q_heads = 1)."""
    h = p.h
    return Problem(p.n_layers, 1, 1, 1, h["cu_seqlens"], h["cu_frames"], h["frame_meta"], h["cu_budget"],
                   device=p.d["cu_seqlens"].device)


def compress_concat(p: Problem, pl: Problem, q_win, k, v, alpha: float = 1.0, stream=None) -> dict:
    """The procedure over the concatenated key space, one kept set per layer
    (pl = layer_problem(p)): window score per kv head, its layer mean, rho and
    Phi over the concatenated keys, the rank gate and the top-B on the layer
    view, and the compaction of every head with its layer's kept set.  Returns
    the device tensors of every stage."""
    import torch
    dev = k.device
    U, Lyr, L, Bt = p.units, p.n_layers, p.total_tokens, p.total_budget
    f32 = dict(dtype=torch.float32, device=dev)
    r = {"a_base": torch.empty((U, L), **f32), "a_layer": torch.empty((Lyr, L), **f32),
         "rho": torch.empty((Lyr, L), **f32), "phi": torch.empty((Lyr, L), **f32),
         "tau": torch.empty((Lyr, p.n_seqs), **f32), "gate": torch.empty((Lyr, L), dtype=torch.uint8, device=dev),
         "kept": torch.empty((Lyr, max(Bt, 1)), dtype=torch.int32, device=dev),
         "k_out": torch.empty((U, max(Bt, 1), 128), dtype=k.dtype, device=dev),
         "v_out": torch.empty((U, max(Bt, 1), 128), dtype=v.dtype, device=dev)}
    n = max(p.workspace_size(CALL_SCORE_WINDOW), p.workspace_size(CALL_TSG_RHO_CONCAT),
            pl.workspace_size(CALL_TSG_THRESHOLD), pl.workspace_size(CALL_SELECT_TOPK), 256)
    ws = torch.empty(n, dtype=torch.uint8, device=dev)
    stlite_score_window(p, q_win, k, r["a_base"], ws, stream)
    stlite_layer_mean(p, r["a_base"], r["a_layer"], stream)
    stlite_tsg_rho_concat(p, k, r["rho"], ws, stream)
    stlite_tsg_threshold(pl, r["rho"], r["tau"], r["gate"], ws, stream)
    stlite_css_saliency_concat(p, k, r["phi"], stream)
    stlite_select_topk(pl, r["a_layer"], r["phi"], r["gate"], alpha, r["kept"], None, ws, stream)
    stlite_compact_kv_layer(p, k, v, r["kept"], r["k_out"], r["v_out"], stream)
    return r


def decode_problem(p: Problem) -> Problem:
    """The same layout and budgets with a one-query window: the problem on which
    stlite_score_window scores the first decode query over the full cache."""
    h = p.h
    return Problem(p.n_layers, p.n_q_heads, p.n_kv_heads, 1, h["cu_seqlens"], h["cu_frames"], h["frame_meta"],
                   h["cu_budget"], device=p.d["cu_seqlens"].device)


def oracle_set(p1: Problem, q_dec, k, kept=None, a_dec=None, stream=None):
    """I* of the cache hit rate (Eq. chr) for every unit and sequence: the top-B_s
    of the first decode query's attention over the full cache.  p1 is
    decode_problem(p); q_dec [n_layers][n_seqs][n_q_heads][d] bf16 (the one-query
    window).  Two C calls: stlite_score_window, then stlite_select_topk with no
    phi and no gate.  Returns (kept [units][total_budget] int32, a_dec)."""
    import torch
    dev = q_dec.device
    if a_dec is None:
        a_dec = torch.empty((p1.units, p1.total_tokens), dtype=torch.float32, device=dev)
    if kept is None:
        kept = torch.empty((p1.units, max(p1.total_budget, 1)), dtype=torch.int32, device=dev)
    n = max(p1.workspace_size(CALL_SCORE_WINDOW), p1.workspace_size(CALL_SELECT_TOPK), 256)
    ws = torch.empty(n, dtype=torch.uint8, device=dev)
    stlite_score_window(p1, q_dec, k, a_dec, ws, stream)
    stlite_select_topk(p1, a_dec, None, None, 0.0, kept, None, ws, stream)
    return kept, a_dec


def kept_overlap(p: Problem, kept_a, kept_b, hits=None, stream=None):
    """hits [units][n_seqs] int32 = |kept_a cap kept_b| per unit and sequence."""
    import torch
    if hits is None:
        hits = torch.empty((p.units, p.n_seqs), dtype=torch.int32, device=kept_a.device)
    stlite_kept_overlap(p, kept_a, kept_b, hits, stream)
    return hits


def compress(p: Problem, q_win, k, v, out: Buffers, alpha: float = 1.0, css: bool = True,
             tsg: bool = True, stream=None, overlap: bool = False, mean_width: int = 0) -> Buffers:
    """The whole pass: score, gate, saliency, select, compact (five C calls).

    mean_width > 0 ranks on the Mean-Attention prior (stlite_mean_attention of
    that width, written to out.a_mean) instead of A_base.

    The TSG gate runs before CSS, which skips the tokens the gate leaves out
    (their Phi is 0; Eq. modal_scoring multiplies it by M = 0 anyway).  With
    ``overlap`` the window scoring runs on ``stream`` while TSG and then CSS
    run on a side stream of ``out``; the top-B selection waits for both.
    Otherwise everything runs in order on ``stream``.
    """
    import torch
    main = stream if stream is not None else torch.cuda.current_stream()
    gate = out.gate if tsg else None
    if not overlap:
        stlite_score_window(p, q_win, k, out.a_base, out.ws, main)
        if tsg:
            stlite_tsg_gate(p, k, out.rho, out.tau, out.gate, out.ws_tsg, main)
        if css:
            stlite_css_saliency(p, k, out.phi, gate, main)
    else:
        side = out.side[0]
        start = torch.cuda.Event()
        start.record(main)
        side.wait_event(start)
        k.record_stream(side)
        stlite_score_window(p, q_win, k, out.a_base, out.ws, main)
        if tsg:
            stlite_tsg_gate(p, k, out.rho, out.tau, out.gate, out.ws_tsg, side)
        if css:
            stlite_css_saliency(p, k, out.phi, gate, side)
        done = torch.cuda.Event()
        done.record(side)
        main.wait_event(done)
    prior = out.a_base
    if mean_width:
        if getattr(out, "a_mean", None) is None:
            out.a_mean = torch.empty_like(out.a_base)
        stlite_mean_attention(p, out.a_base, mean_width, out.a_mean, main)
        prior = out.a_mean
    stlite_select_topk(p, prior, out.phi if css else None, out.gate if tsg else None, alpha,
                       out.kept, out.score, out.ws, main)
    stlite_compact_kv(p, k, v, out.kept, out.k_out, out.v_out, main)
    return out


def capture_compress(p: Problem, q_win, k, v, out: Buffers, alpha: float = 1.0, css: bool = True,
                     tsg: bool = True, mean_width: int = 0):
    """The whole pass (compress() on one stream) captured once into a HIP graph
    (torch.cuda.CUDAGraph); ``graph.replay()`` then runs every kernel of the pass
    with one launch.  Every call of the pass only enqueues kernels on its stream
    (no allocation, copy, memset or synchronisation), and ``out`` holds every
    buffer, so the graph stays valid while p, the inputs and ``out`` live; a
    replay recomputes from whatever the input tensors hold."""
    import torch
    if mean_width and getattr(out, "a_mean", None) is None:
        out.a_mean = torch.empty_like(out.a_base)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # one eager pass first, as torch asks before a capture
        compress(p, q_win, k, v, out, alpha, css, tsg, stream=side, mean_width=mean_width)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        compress(p, q_win, k, v, out, alpha, css, tsg, stream=torch.cuda.current_stream(), mean_width=mean_width)
    return graph

