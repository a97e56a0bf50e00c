"""Seeded synthetic GUI-trajectory inputs for the ST-Lite compression pass.

This module only *draws inputs*: packed KV caches, observation-window queries and
the frame/sequence layout.  It holds none of the method's arithmetic (no
softmax, cosine, gate, selection or gather), so both the fp64 oracle and the
HIP path can consume the very same bytes.

Shapes and statistics follow the paper's workloads:

* a trajectory H_t interleaves screenshots and text (problem setup, Eq.
  history_context); every screenshot is a row-major patch grid of visual tokens
  followed by a run of text tokens, and the observation window is the last
  ``window`` tokens of the sequence;
* consecutive frames are highly redundant (inter-frame redundancy appendix:
  median 82.7% of pixels unchanged), modelled by copying the previous frame's
  patch embeddings and resampling a few rectangles (or nothing, for an exact
  duplicate frame);
* decision-relevant UI elements are small (UI element size appendix: median
  1.7% x 1.6% of the screen), modelled by window queries aimed at one small
  element rectangle of the current frame.

Recipe (all draws in float32, rounded once to bf16 with round-to-nearest-even):

* per-patch embeddings e ~ N(0,1)/sqrt(d), shared by every layer;
* visual keys of (layer l, kv head h) are W_{l,h} e with W_{l,h} ~ N(0, 1/d),
  an independent random projection per layer and head;
* text keys are i.i.d. N(0,1)/sqrt(d); values are i.i.d. N(0,1);
* the query of (q head g, window position w) is the sum of the current-frame
  keys of kv head g//G over the sequence's element rectangle, plus N(0, 0.1^2)
  noise per component.

Two screen models (``Workload.screen``):

* ``"iid"`` (every named workload): each freshly drawn patch embedding is
  independent of its neighbours;
* ``"gui"``: a screen is a few flat panels (a top bar, a side bar and the main
  area, one colour embedding each, drawn once per trajectory) with UI elements
  drawn over about a quarter of the area.  A background patch is its panel's
  colour plus a texture of 1/3 of its scale (neighbouring background patches
  have cosine about 0.9); an element patch is an independent embedding.  A
  frame transition repaints each resampled rectangle the same way.  The
  element rectangle the queries aim at is centred on an element patch.

Random streams: ``numpy.random.SeedSequence(seed).spawn(n_layers + 1)``; stream 0
draws the layout, the frame evolution and the element rectangles, stream l+1
draws everything that belongs to layer l, so any single layer can be
regenerated on its own.
"""
from __future__ import annotations

import dataclasses
import math
from typing import List, Optional, Sequence, Tuple

import numpy as np

HEAD_DIM = 128

# Segment kinds in a trajectory description.
FRAME = "frame"
TEXT = "text"

# Screen models (module docstring).
SCREENS = ("iid", "gui")
GUI_TEXTURE = 1.0 / 3.0   # background texture scale, relative to a panel colour's
GUI_COVER = 0.25          # element area drawn per painted region, as a fraction of it


@dataclasses.dataclass(frozen=True)
class Redundancy:
    """How frame t+1 is derived from frame t (patch-embedding level).

    ``rects``: fixed list of (h, w) rectangles resampled per transition, or None.
    ``frac``: (lo, hi) fraction of the grid resampled, spread over ``n_rects``
    (lo, hi) rectangles, used when ``rects`` is None.
    ``dup_frac``: fraction of the frames (frame 1 onwards) that are exact copies
    of their predecessor.
    """

    rects: Optional[Tuple[Tuple[int, int], ...]] = None
    frac: Tuple[float, float] = (0.05, 0.15)
    n_rects: Tuple[int, int] = (1, 4)
    dup_frac: float = 0.0


@dataclasses.dataclass(frozen=True)
class Workload:
    """A packed batch of GUI trajectories plus model shape and method knobs."""

    name: str
    n_layers: int
    n_q_heads: int
    n_kv_heads: int
    window: int
    beta: Tuple[int, int]                 # budget ratio as a rational num/den
    seqs: Tuple[Tuple[Tuple, ...], ...]   # per sequence: segments (FRAME, rows, cols) | (TEXT, n)
    redundancy: Redundancy = Redundancy()
    element: Tuple[Tuple[int, int], Tuple[int, int]] = ((2, 2), (2, 2))  # (h lo,hi), (w lo,hi)
    seed: int = 0
    alpha: float = 1.0
    head_dim: int = HEAD_DIM
    screen: str = "iid"                   # "iid" | "gui" (module docstring)

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def seq_lengths(self) -> List[int]:
        out = []
        for segs in self.seqs:
            n = 0
            for s in segs:
                n += s[1] * s[2] if s[0] == FRAME else s[1]
            out.append(n)
        return out

    @property
    def total_tokens(self) -> int:
        return sum(self.seq_lengths())

    def with_beta(self, num: int, den: int) -> "Workload":
        return dataclasses.replace(self, beta=(num, den))

    def with_layers(self, n_layers: int) -> "Workload":
        return dataclasses.replace(self, n_layers=n_layers)

    def with_screen(self, screen: str) -> "Workload":
        if screen not in SCREENS:
            raise ValueError(f"screen must be one of {SCREENS}")
        name = self.name if screen == "iid" else f"{self.name}_{screen}"
        return dataclasses.replace(self, screen=screen, name=name)


def _interleaved(n_frames: int, rows: int, cols: int, text) -> Tuple[Tuple, ...]:
    segs = []
    for f in range(n_frames):
        segs.append((FRAME, rows, cols))
        segs.append((TEXT, text[f] if isinstance(text, (list, tuple)) else text))
    return tuple(segs)


def config(idx: int, beta: Optional[Tuple[int, int]] = None) -> Workload:
    """The five benchmark configurations of the compression pass.

    0 tiny: 1 layer, 3 frames of 16x16 patches, each followed by 48 text tokens;
    1 single agent step: one 36x80 screenshot plus 512 text tokens, 28 layers;
    2 long horizon: 20 frames x (2880 visual + 256 text), window 64;
    3 fifty-step trajectory: 48 frames x (2880 + 256), 30% exact duplicates;
    4 ragged batch: 8 trajectories of 6-24 frames, 128-512 text tokens per frame.
    """
    if idx == 0:
        return Workload("tiny", 1, 28, 4, 32, beta or (1, 5),
                        (_interleaved(3, 16, 16, 48),),
                        Redundancy(rects=((2, 3), (2, 3))), ((2, 2), (2, 2)), seed=0)
    if idx == 1:
        return Workload("single_step", 28, 28, 4, 32, beta or (1, 5),
                        (((FRAME, 36, 80), (TEXT, 512)),),
                        Redundancy(), ((2, 2), (2, 2)), seed=1)
    if idx == 2:
        return Workload("long_horizon", 28, 28, 4, 64, beta or (1, 5),
                        (_interleaved(20, 36, 80, 256),),
                        Redundancy(frac=(0.05, 0.15), n_rects=(1, 4)),
                        ((1, 3), (2, 4)), seed=2)
    if idx == 3:
        return Workload("trajectory_50step", 28, 28, 4, 64, beta or (1, 5),
                        (_interleaved(48, 36, 80, 256),),
                        Redundancy(frac=(0.05, 0.20), n_rects=(1, 4), dup_frac=0.30),
                        ((1, 3), (2, 4)), seed=3)
    if idx == 4:
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([4, 0xB47C4])))
        seqs = []
        for _ in range(8):
            nf = int(rng.integers(6, 25))
            text = [int(t) for t in rng.integers(128, 513, size=nf)]
            seqs.append(_interleaved(nf, 36, 80, text))
        return Workload("ragged_batch", 28, 28, 4, 32, beta or (1, 10), tuple(seqs),
                        Redundancy(frac=(0.05, 0.15), n_rects=(1, 4)),
                        ((1, 3), (2, 4)), seed=4)
    raise ValueError(f"unknown config {idx}")


# ---------------------------------------------------------------------------
# Layout
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class Layout:
    """Packed varlen layout shared by both sides.

    cu_seqlens[n_seqs+1], cu_frames[n_seqs+1]: prefix sums of tokens / frames.
    frame_meta[n_frames][3]: absolute token offset, rows, cols of each frame
    (frames of one sequence are listed in temporal order; the last one is the
    current frame).  Every token that is not inside a frame is text.
    """

    cu_seqlens: np.ndarray
    cu_frames: np.ndarray
    frame_meta: np.ndarray

    @property
    def n_seqs(self) -> int:
        return len(self.cu_seqlens) - 1

    @property
    def total_tokens(self) -> int:
        return int(self.cu_seqlens[-1])

    def seq_frames(self, s: int) -> np.ndarray:
        return self.frame_meta[self.cu_frames[s]:self.cu_frames[s + 1]]


def make_layout(w: Workload) -> Layout:
    cu_s = [0]
    cu_f = [0]
    meta = []
    pos = 0
    for segs in w.seqs:
        for seg in segs:
            if seg[0] == FRAME:
                r, c = int(seg[1]), int(seg[2])
                meta.append((pos, r, c))
                pos += r * c
            elif seg[0] == TEXT:
                pos += int(seg[1])
            else:
                raise ValueError(seg)
        cu_s.append(pos)
        cu_f.append(len(meta))
    return Layout(np.asarray(cu_s, np.int32), np.asarray(cu_f, np.int32),
                  np.asarray(meta, np.int32).reshape(-1, 3))


# ---------------------------------------------------------------------------
# bf16 storage helpers (storage conversion only)
# ---------------------------------------------------------------------------

def to_bf16_bits_reference(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round-to-nearest-even (finite inputs)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    b = b + (np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1)))
    return (b >> np.uint32(16)).astype(np.uint16)


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Same rounding as ``to_bf16_bits_reference``, multithreaded through torch's CPU cast."""
    try:
        import torch
    except ImportError:  # pragma: no cover
        return to_bf16_bits_reference(x)
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


# ---------------------------------------------------------------------------
# Drawing
# ---------------------------------------------------------------------------

def _rng(ss: np.random.SeedSequence) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(ss))


def _streams(w: Workload):
    return np.random.SeedSequence(w.seed).spawn(w.n_layers + 1)


def _random_rect(rng, rows, cols, h, ww):
    h = min(h, rows)
    ww = min(ww, cols)
    u0 = int(rng.integers(0, rows - h + 1))
    v0 = int(rng.integers(0, cols - ww + 1))
    return u0, v0, h, ww


@dataclasses.dataclass
class Scene:
    """Layer-independent part of a workload: patch embeddings and targets."""

    layout: Layout
    frame_emb: List[np.ndarray]            # per frame: [rows*cols, d] float32
    element: List[Tuple[int, int, int, int]]  # per sequence: (u0, v0, h, w) in its current frame
    duplicate: List[bool]                  # per frame: exact copy of its predecessor
    content: Optional[List[np.ndarray]] = None  # gui screens, per frame: [rows*cols] bool, element patch


def gui_panels(rows: int, cols: int) -> np.ndarray:
    """Panel of every cell of a rows x cols gui screen: 0 top bar (the first
    ~rows/12 rows), 1 side bar (the first ~cols/6 columns below it), 2 main area."""
    tb = max(1, round(rows / 12))
    sb = max(1, round(cols / 6))
    p = np.full((rows, cols), 2, np.int8)
    p[:tb, :] = 0
    p[tb:, :sb] = 1
    return p


def _gui_paint(rng, e, content, panels, colours, rect, element, d):
    """Repaint rect = (u0, v0, h, w) of a gui screen e [rows, cols, d]: textured
    panel background, then elements over about GUI_COVER of its area (at least
    one), each of a size drawn from ``element`` and clipped to the rectangle."""
    u0, v0, h, ww = rect
    inv = np.float32(1.0 / math.sqrt(d))
    e[u0:u0 + h, v0:v0 + ww] = (colours[panels[u0:u0 + h, v0:v0 + ww]]
                                + np.float32(GUI_TEXTURE) * inv * rng.standard_normal((h, ww, d), dtype=np.float32))
    content[u0:u0 + h, v0:v0 + ww] = False
    (hlo, hhi), (wlo, whi) = element
    mean_area = 0.25 * (hlo + hhi) * (wlo + whi)
    for _ in range(max(1, int(math.ceil(GUI_COVER * h * ww / mean_area)))):
        eh = min(int(rng.integers(hlo, hhi + 1)), h)
        ew = min(int(rng.integers(wlo, whi + 1)), ww)
        a = u0 + int(rng.integers(0, h - eh + 1))
        b = v0 + int(rng.integers(0, ww - ew + 1))
        e[a:a + eh, b:b + ew] = rng.standard_normal((eh, ew, d), dtype=np.float32) * inv
        content[a:a + eh, b:b + ew] = True


def _centred_rect(p, rows, cols, h, ww):
    """Rectangle of size h x w (clipped to the grid) centred on cell p."""
    h = min(h, rows)
    ww = min(ww, cols)
    u0 = min(max(p // cols - h // 2, 0), rows - h)
    v0 = min(max(p % cols - ww // 2, 0), cols - ww)
    return u0, v0, h, ww


def make_scene(w: Workload) -> Scene:
    lay = make_layout(w)
    d = w.head_dim
    rng = _rng(_streams(w)[0])
    red = w.redundancy
    gui = w.screen == "gui"
    if w.screen not in SCREENS:
        raise ValueError(f"unknown screen model {w.screen!r}")
    embs: List[np.ndarray] = []
    dups: List[bool] = []
    conts: List[np.ndarray] = []
    elems = []
    for s in range(lay.n_seqs):
        fm = lay.seq_frames(s)
        nf = len(fm)
        dup_set = set()
        if red.dup_frac > 0 and nf > 1:
            n_dup = int(round(red.dup_frac * nf))
            n_dup = min(n_dup, nf - 1)
            dup_set = set(int(x) for x in rng.choice(np.arange(1, nf), size=n_dup, replace=False))
        prev = None
        cont = None
        colours = None
        for f in range(nf):
            r, c = int(fm[f, 1]), int(fm[f, 2])
            fresh = prev is None or prev.shape[0] != r * c
            if fresh and gui:
                if colours is None:
                    colours = rng.standard_normal((3, d), dtype=np.float32) / np.float32(math.sqrt(d))
                e = np.empty((r, c, d), np.float32)
                cont = np.zeros((r, c), bool)
                _gui_paint(rng, e, cont, gui_panels(r, c), colours, (0, 0, r, c), w.element, d)
                e = e.reshape(r * c, d)
                dups.append(False)
            elif fresh:
                e = (rng.standard_normal((r * c, d), dtype=np.float32) / np.float32(math.sqrt(d)))
                dups.append(False)
            elif f in dup_set:
                e = prev.copy()
                dups.append(True)
            else:
                e = prev.copy().reshape(r, c, d)
                if red.rects is not None:
                    rects = [_random_rect(rng, r, c, h, ww) for (h, ww) in red.rects]
                else:
                    frac = float(rng.uniform(*red.frac))
                    nr = int(rng.integers(red.n_rects[0], red.n_rects[1] + 1))
                    area = frac * r * c / nr
                    rects = []
                    for _ in range(nr):
                        aspect = float(rng.uniform(0.5, 2.0))
                        h = int(np.clip(round(math.sqrt(area * aspect)), 1, r))
                        ww = int(np.clip(round(area / h), 1, c))
                        rects.append(_random_rect(rng, r, c, h, ww))
                if gui:
                    cont = cont.copy()
                    for rect in rects:
                        _gui_paint(rng, e, cont, gui_panels(r, c), colours, rect, w.element, d)
                else:
                    for (u0, v0, h, ww) in rects:
                        e[u0:u0 + h, v0:v0 + ww] = (
                            rng.standard_normal((h, ww, d), dtype=np.float32) / np.float32(math.sqrt(d)))
                e = e.reshape(r * c, d)
                dups.append(False)
            embs.append(e)
            if gui:
                conts.append(cont.reshape(-1))
            prev = e
        if nf:
            r, c = int(fm[-1, 1]), int(fm[-1, 2])
            (hlo, hhi), (wlo, whi) = w.element
            h = int(rng.integers(hlo, hhi + 1))
            ww = int(rng.integers(wlo, whi + 1))
            if gui:  # centred on an element patch of the current frame
                cells = np.flatnonzero(conts[-1])
                elems.append(_centred_rect(int(cells[int(rng.integers(0, len(cells)))]), r, c, h, ww))
            else:
                elems.append(_random_rect(rng, r, c, h, ww))
        else:
            elems.append((0, 0, 0, 0))
    return Scene(lay, embs, elems, dups, conts if gui else None)


def text_positions(lay: Layout) -> np.ndarray:
    """Absolute indices of the tokens that lie in no frame."""
    is_text = np.ones(lay.total_tokens, bool)
    for off, r, c in lay.frame_meta:
        is_text[off:off + r * c] = False
    return np.flatnonzero(is_text)


@dataclasses.dataclass
class LayerInputs:
    k: np.ndarray   # uint16 bf16 bits [n_kv_heads, L_total, d]
    v: np.ndarray   # uint16 bf16 bits [n_kv_heads, L_total, d]
    q: np.ndarray   # uint16 bf16 bits [n_seqs, n_q_heads, window, d]


def make_layer(w: Workload, scene: Scene, layer: int) -> LayerInputs:
    """Draw the keys, values and window queries of one layer."""
    lay = scene.layout
    d = w.head_dim
    L = lay.total_tokens
    hk = w.n_kv_heads
    G = w.group
    rng = _rng(_streams(w)[layer + 1])
    inv = np.float32(1.0 / math.sqrt(d))
    k32 = np.empty((hk, L, d), np.float32)
    text = text_positions(lay)
    for h in range(hk):
        k32[h, text] = rng.standard_normal((len(text), d), dtype=np.float32) * inv
    W = rng.standard_normal((hk, d, d), dtype=np.float32) * inv
    for f, (off, r, c) in enumerate(lay.frame_meta):
        e = scene.frame_emb[f]
        for h in range(hk):
            k32[h, off:off + r * c] = e @ W[h].T
    q32 = np.empty((lay.n_seqs, w.n_q_heads, w.window, d), np.float32)
    for s in range(lay.n_seqs):
        fm = lay.seq_frames(s)
        noise = rng.standard_normal((w.n_q_heads, w.window, d), dtype=np.float32) * np.float32(0.1)
        if len(fm):
            off, r, c = (int(x) for x in fm[-1])
            u0, v0, h, ww = scene.element[s]
            idx = np.array([off + (u0 + a) * c + (v0 + b) for a in range(h) for b in range(ww)])
            for g in range(w.n_q_heads):
                q32[s, g] = k32[g // G, idx].sum(axis=0)[None, :] + noise[g]
        else:
            q32[s] = noise
    v = to_bf16_bits(rng.standard_normal((hk, L, d), dtype=np.float32))
    return LayerInputs(to_bf16_bits(k32), v, to_bf16_bits(q32))


def make_inputs(w: Workload, layers: Optional[Sequence[int]] = None, workers: int = 8):
    """All layers (or the listed ones) stacked: K, V [nl, Hkv, L, d], Q [nl, S, Hq, win, d].

    Layers are drawn in parallel threads; every layer has its own random stream,
    so the result does not depend on ``workers``."""
    scene = make_scene(w)
    layers = list(range(w.n_layers)) if layers is None else list(layers)
    L = scene.layout.total_tokens
    k = np.empty((len(layers), w.n_kv_heads, L, w.head_dim), np.uint16)
    v = np.empty_like(k)
    q = np.empty((len(layers), scene.layout.n_seqs, w.n_q_heads, w.window, w.head_dim), np.uint16)

    def one(i):
        p = make_layer(w, scene, layers[i])
        k[i], v[i], q[i] = p.k, p.v, p.q

    if workers > 1 and len(layers) > 1:
        from concurrent.futures import ThreadPoolExecutor
        with ThreadPoolExecutor(min(workers, len(layers))) as ex:
            list(ex.map(one, range(len(layers))))
    else:
        for i in range(len(layers)):
            one(i)
    return scene, k, v, q


def decode_queries(q: np.ndarray) -> np.ndarray:
    """Decode queries [layers, seqs, Hq, d] (bf16 bits) for the decoding phase
    that follows the compression: each head's window query at the last window
    position, i.e. the query the model formed at the end of prefill, which the
    first decode step's query resembles."""
    return np.ascontiguousarray(q[:, :, :, -1, :])


# ---------------------------------------------------------------------------
# Recompression at every step of one trajectory
# ---------------------------------------------------------------------------

STEP_STREAM = 0x57E95   # spawn key of the per-step draws (elements, anchors, query noise)


@dataclasses.dataclass
class StepInputs:
    """The caches of the steps of one trajectory, packed one sequence per step.

    Step t's context is the trajectory's prefix up to and including the text
    that follows frame t (problem setup, Eq. history_context: the earlier
    screenshots and actions, then the current screenshot); frame t is that
    step's current frame.  Keys and values of a prefix are the trajectory's own
    rows (causal attention leaves a prefix's cache unchanged), so sequence t of
    the packed batch is a copy of rows 0 .. L_t - 1.

    Window queries of step t aim at an element rectangle of frame t.  The
    decode query of step t (first action token) is not one of the window
    queries: it sums the keys of the same element and of an anchor rectangle of
    an earlier frame whose content has since changed (a distant token the
    current screen no longer shows), plus noise.
    """

    base: Workload
    steps: List[int]
    workload: Workload        # the packed batch (one sequence per step)
    layout: Layout
    k: Optional[np.ndarray]   # [nl, Hkv, sum L_t, d] bf16 bits (None unless packed)
    v: Optional[np.ndarray]
    q: np.ndarray             # [nl, T, Hq, window, d]
    q_dec: np.ndarray         # [nl, T, Hq, d]
    element: List[Tuple[int, int, int, int]]        # per step, in frame t
    anchor: List[Optional[Tuple[int, int, int, int, int]]]  # per step: (frame, u0, v0, h, w) or None


def step_prefix_segments(w: Workload, t: int) -> Tuple[Tuple, ...]:
    """Segments of step t's context: everything before frame t + 1."""
    segs = w.seqs[0]
    frames = [i for i, s in enumerate(segs) if s[0] == FRAME]
    end = frames[t + 1] if t + 1 < len(frames) else len(segs)
    return tuple(segs[:end])


def make_step_inputs(w: Workload, steps: Optional[Sequence[int]] = None,
                     layers: Optional[Sequence[int]] = None, base=None, pack: bool = True) -> StepInputs:
    """Inputs of the recompression at the listed steps (default: every frame)
    of the single trajectory of ``w``.  ``base`` = make_inputs(w, layers) may be
    passed to reuse already drawn caches.  With pack=False the packed k and v
    are not built (None): the caller slices each step's rows from the
    trajectory's own arrays."""
    if len(w.seqs) != 1:
        raise ValueError("make_step_inputs takes a single-trajectory workload")
    scene, kb, vb, _ = make_inputs(w, layers) if base is None else base
    lay0 = scene.layout
    fm = lay0.seq_frames(0)
    nf = len(fm)
    steps = list(range(nf)) if steps is None else [int(t) for t in steps]
    if not steps or min(steps) < 0 or max(steps) >= nf:
        raise ValueError("steps must index frames of the trajectory")
    packed = dataclasses.replace(w, seqs=tuple(step_prefix_segments(w, t) for t in steps))
    lay = make_layout(packed)
    lens = np.diff(lay.cu_seqlens)
    if (lens < w.window).any():
        raise ValueError("every step's context must hold the observation window")
    layers = list(range(w.n_layers)) if layers is None else list(layers)
    nl, hk, d, G = len(layers), w.n_kv_heads, w.head_dim, w.group
    L = lay.total_tokens
    k = v = None
    if pack:
        k = np.empty((nl, hk, L, d), np.uint16)
        v = np.empty_like(k)
        for i, t in enumerate(steps):
            a, n = int(lay.cu_seqlens[i]), int(lens[i])
            k[:, :, a:a + n] = kb[:, :, :n]
            v[:, :, a:a + n] = vb[:, :, :n]

    # per-step element and anchor rectangles (layer independent); every step,
    # and every (step, layer), has a stream of its own, so a step regenerates
    # alone whatever other steps are listed
    (hlo, hhi), (wlo, whi) = w.element
    elems, anchors = [], []
    gui = scene.content is not None
    for t in steps:
        rng = _rng(np.random.SeedSequence([w.seed, STEP_STREAM, t]))
        r, c = int(fm[t, 1]), int(fm[t, 2])
        h = int(rng.integers(hlo, hhi + 1))
        ww = int(rng.integers(wlo, whi + 1))
        if gui:  # centred on an element patch of frame t
            cells = np.flatnonzero(scene.content[t])
            elems.append(_centred_rect(int(cells[int(rng.integers(0, len(cells)))]), r, c, h, ww))
        else:
            elems.append(_random_rect(rng, r, c, h, ww))
        anchor = None
        if t > 0:
            f = int(rng.integers(0, t))
            ef, et = scene.frame_emb[f], scene.frame_emb[t]
            if ef.shape == et.shape:
                changed = (ef != et).any(axis=1)
                if gui and (changed & scene.content[f]).any():  # a changed element patch
                    changed &= scene.content[f]
                changed = np.flatnonzero(changed)
                rf, cf = int(fm[f, 1]), int(fm[f, 2])
                if len(changed):
                    p = int(changed[int(rng.integers(0, len(changed)))])
                    h = int(rng.integers(hlo, hhi + 1))
                    ww = int(rng.integers(wlo, whi + 1))
                    anchor = (f,) + _centred_rect(p, rf, cf, h, ww)
        anchors.append(anchor)

    def cells(frame, u0, v0, h, ww):
        off, _, c = (int(x) for x in fm[frame])
        return np.array([off + (u0 + i) * c + (v0 + j) for i in range(h) for j in range(ww)])

    q = np.empty((nl, len(steps), w.n_q_heads, w.window, d), np.uint16)
    q_dec = np.empty((nl, len(steps), w.n_q_heads, d), np.uint16)
    k32 = lambda li, h, idx: bf16_bits_to_f32(kb[li, h, idx])
    for li in range(nl):
        for i, t in enumerate(steps):
            lrng = _rng(np.random.SeedSequence([w.seed, STEP_STREAM, t, layers[li] + 1]))
            el = cells(t, *elems[i])
            an = cells(*anchors[i]) if anchors[i] is not None else None
            noise = lrng.standard_normal((w.n_q_heads, w.window + 1, d), dtype=np.float32) * np.float32(0.1)
            qs = np.empty((w.n_q_heads, w.window, d), np.float32)
            qd = np.empty((w.n_q_heads, d), np.float32)
            for g in range(w.n_q_heads):
                target = k32(li, g // G, el).sum(axis=0)
                qs[g] = target[None, :] + noise[g, :w.window]
                extra = k32(li, g // G, an).sum(axis=0) if an is not None else 0.0
                qd[g] = target + extra + noise[g, w.window]
            q[li, i] = to_bf16_bits(qs)
            q_dec[li, i] = to_bf16_bits(qd)
    return StepInputs(w, steps, packed, lay, k, v, q, q_dec, elems, anchors)
