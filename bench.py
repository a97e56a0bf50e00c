"""Benchmark of the ST-Lite KV-cache compression pass on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 3]

One step is the whole pass -- stlite_score_window, stlite_tsg_gate,
stlite_css_saliency, stlite_select_topk, stlite_compact_kv -- over every layer
and kv head of one synthetic batch that is resident in HBM before timing
starts.  The default workload is the 50-step GUI trajectory: 48 frames of
36 x 80 patches, each followed by 256 text tokens (150,528 tokens), 28 layers,
28 query / 4 kv heads, head_dim 128, window 64, beta = 1/5.

Prints ONE JSON line on stdout.  ``value`` is cached tokens compressed per
second over all layers (tokens / step time).  ``roofline`` describes the call
that takes the largest share of the step, timed with HIP events recorded on
the stream the calls are launched on, inside the timed loop.  ``cpu_baseline``
times the fp64 oracle on a bounded sample of the same workload on the host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "cached KV tokens compressed/sec (all layers) at β=20%; % MFMA peak, HBM GB/s"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def log(msg):
    sys.stderr.write(f"[bench {time.strftime('%H:%M:%S')}] {msg}\n")
    sys.stderr.flush()


def work_model(w, lay, cu_budget):
    """Algorithmic work per call of one step (all units): FLOPs and HBM bytes."""
    units = w.n_layers * w.n_kv_heads
    d = w.head_dim
    rows = w.group * w.window
    L_tot = lay.total_tokens
    n_hist = n_cur = n_vis = 0
    for s in range(lay.n_seqs):
        fm = lay.seq_frames(s)
        sizes = [int(r) * int(c) for _, r, c in fm]
        n_vis += sum(sizes)
        if sizes:
            n_cur_s = sizes[-1]
            n_hist_s = sum(sizes[:-1])
            n_hist += n_hist_s
            n_cur += n_cur_s * (1 if n_hist_s else 0)
    hist_cur = 0
    for s in range(lay.n_seqs):
        sizes = [int(r) * int(c) for _, r, c in lay.seq_frames(s)]
        if len(sizes) > 1:
            hist_cur += sum(sizes[:-1]) * sizes[-1]
    B_tot = int(cu_budget[-1])
    return {
        # QK^T of the window rows against every key, once (the pass forms it twice)
        "score_window": {"bound": "mfma", "flops": units * 2.0 * rows * L_tot * d,
                         "bytes": units * (2.0 * L_tot * d * 2 + 4.0 * L_tot)},
        # N_hist x N_cur x d cosine contraction; K_hist and K_cur read once, rho written
        "tsg_rho": {"bound": "mfma", "flops": units * 2.0 * hist_cur * d,
                    "bytes": units * (2.0 * (n_hist + n_cur) * d + 4.0 * L_tot)},
        # rho of the historical tokens read, the gate written
        "tsg_threshold": {"bound": "hbm", "flops": 0.0, "bytes": units * (4.0 * n_hist + 1.0 * L_tot)},
        "css_saliency": {"bound": "hbm", "flops": units * 2.0 * 5 * n_vis * d,
                         "bytes": units * (2.0 * n_vis * d + 4.0 * L_tot)},
        "select_topk": {"bound": "hbm", "flops": 0.0,
                        "bytes": units * (9.0 * L_tot + 4.0 * B_tot)},
        "compact_kv": {"bound": "hbm", "flops": 0.0,
                       "bytes": units * 4.0 * B_tot * d * 2},
    }


def roofline_entry(model, ms):
    s = ms * 1e-3
    if model["bound"] == "mfma":
        ach = model["flops"] / s / 1e12
        return {"bound": "mfma", "achieved": round(ach, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(ach / PEAK_BF16_TFLOPS, 4), "ms": round(ms, 4)}
    ach = model["bytes"] / s / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(ach / PEAK_HBM_GBS, 4), "ms": round(ms, 4)}


PROFILES = os.path.join(ROOT, "profiles")
KERNEL_SOURCES = {  # the sources a kernel's counters depend on
    "rho_kernel": ["paper_2603_00188_amd/csrc/tsg.hip", "paper_2603_00188_amd/csrc/tile_lds.h",
                   "paper_2603_00188_amd/csrc/stlite_internal.h"],
}


def source_digest(kernel):
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES.get(kernel, []):
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` from the committed counter summary
    profiles/<kernel>_<workload>_traffic.md (FETCH_SIZE + WRITE_SIZE, each scaled
    by the copy-kernel calibration), or None when there is none or the kernel's
    sources changed since the counters were taken."""
    path = os.path.join(PROFILES, f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path) or kernel not in KERNEL_SOURCES:
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and line.startswith("- "):
                k, v = line[2:].split(":", 1)
                fields[k.strip()] = v.strip().strip("`")
    if fields.get("source_digest") != source_digest(kernel):
        return None
    try:
        return float(fields["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def copy_probe(nbytes):
    """A plain device-to-device copy of known size, for scaling the counters."""
    import torch
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes": nbytes, "launches": 3}), flush=True)


def cpu_baseline(w, case_inputs, budget_s=6.0, runs=3, literal=False):
    """The fp64 oracle on the host, timed the way the baseline plan asks: one
    untimed unit, then the median of `runs` timed passes over a sample of whole
    (layer, kv head) units (every sequence) sized to ~budget_s per pass from
    the untimed unit's time, scaled to all units.  literal: time the
    pure-Python loop twin of the oracle instead of the NumPy one (meant for the
    tiny workload)."""
    from oracle import stlite_oracle as O
    from oracle import literal as O1
    scene, k, v, q = case_inputs
    lay = scene.layout
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        cores = max([i.get("num_threads", 1) for i in info] or [1])
    except Exception:  # pragma: no cover
        cores = os.cpu_count()
    units_all = [(l, h) for l in range(w.n_layers) for h in range(w.n_kv_heads)]
    order = [units_all[i] for i in np.random.default_rng(0).permutation(len(units_all))]

    def one(unit):
        l, h = unit
        for s in range(lay.n_seqs):
            if literal:
                a, b = int(lay.cu_seqlens[s]), int(lay.cu_seqlens[s + 1])
                Q = O.bf16_to_f64(q[l, s, h * w.group:(h + 1) * w.group]).tolist()
                K = O.bf16_to_f64(k[l, h, a:b]).tolist()
                frames = O.seq_frames_local(lay.cu_seqlens, lay.cu_frames, lay.frame_meta, s)
                O1.compress(Q, K, frames, O.budget(b - a, *w.beta), w.alpha)
            else:
                O.compress_sequence(q, k, v, lay.cu_seqlens, lay.cu_frames, lay.frame_meta, s, l, h, w.group,
                                    w.beta, w.alpha)

    t0 = time.perf_counter()
    one(order[0])  # untimed
    t_unit = time.perf_counter() - t0
    n = int(min(len(units_all), max(1, round(budget_s / max(t_unit, 1e-9)))))
    sample = order[:n]
    times = []
    for r in range(runs):
        t0 = time.perf_counter()
        for unit in sample:
            one(unit)
        times.append(time.perf_counter() - t0)
        log(f"cpu baseline: timed run {r + 1} of {runs}: {n} units in {times[-1]:.3g} s")
    med = float(np.median(times))
    rate = lay.total_tokens / (med / n * len(units_all))
    what = "pure-Python loop twin of the oracle (one thread)" if literal else "fp64 NumPy oracle"
    return {"value": round(rate, 1), "unit": "tokens/s", "cores": 1 if literal else int(cores),
            "kind": "oracle-literal" if literal else "oracle",
            "sample": f"{n} of {len(units_all)} (layer, kv head) units of the full workload, every sequence, "
                      f"{what}; one untimed unit, then the median of {runs} timed passes "
                      f"({', '.join(f'{t:.3g}' for t in times)} s), rate scaled to all {len(units_all)} units"}


def decode_timing(prob, w, q, dk, dv, out, stream, reps=20):
    """Decode attention (the decoding phase the compression serves) over the
    full cache and over the compacted cache the last step wrote, timed apart
    from the pass: one decode query per head, HIP events on the launch
    stream.  Both are HBM-bound: the bytes are the K and V rows read."""
    import torch
    from paper_2603_00188_amd import stlite as S
    from paper_2603_00188_amd import workload as W
    q_dec = torch.from_numpy(W.decode_queries(q).view(np.int16)).cuda()
    res = torch.empty((prob.n_layers, prob.n_seqs, prob.n_q_heads, 128), dtype=torch.float32, device="cuda")
    units = prob.units
    entry = {}
    for name, cache, kk, vv, call, rows in (
            ("full", S.CACHE_FULL, dk, dv, S.CALL_DECODE_FULL, prob.total_tokens),
            ("compact", S.CACHE_COMPACT, out.k_out, out.v_out, S.CALL_DECODE_COMPACT, prob.total_budget)):
        ws = torch.empty(max(prob.workspace_size(call), 256), dtype=torch.uint8, device="cuda")
        for _ in range(3):
            S.stlite_decode_attention(prob, cache, q_dec, kk, vv, res, ws, stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            S.stlite_decode_attention(prob, cache, q_dec, kk, vv, res, ws, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / reps
        e = roofline_entry({"bound": "hbm", "bytes": units * rows * 128 * 2 * 2.0}, ms)
        e["rows_per_unit"] = int(rows)
        entry[name] = e
    entry["speedup"] = round(entry["full"]["ms"] / entry["compact"]["ms"], 3)
    log(f"decode attention: full cache {entry['full']['ms']:.3f} ms, compacted {entry['compact']['ms']:.3f} ms, "
        f"speedup {entry['speedup']:.2f}x")
    return entry


def variants_timing(prob, w, lay, cu_budget, dk, rho, out, stream, reps=10):
    """The paper's ablation variants on the same workload, each timed apart
    (HIP events on the launch stream) against its own roofline: rho under the
    dot product and the negative L2 distance (the rho contraction's work),
    the fixed-threshold gate (rho of the history read, the gate written), the
    Mean-Attention prior (A_base read, the pooled prior written) and
    CSS over 5x5, 7x7 and 9x9 neighbourhoods (every visual key read once and
    Phi written; the (k^2 - 1)/2 cosines per token are far below the MFMA
    roofline at these sizes)."""
    import torch
    from paper_2603_00188_amd import stlite as S
    model = work_model(w, lay, cu_budget)
    units = prob.units
    n_vis = sum(int(r) * int(c) for _, r, c in lay.frame_meta)

    def timed(fn):
        for _ in range(2):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    tmp = torch.empty_like(rho)
    entry = {}
    for name, sim in (("tsg_rho_dot", S.SIM_DOT), ("tsg_rho_neg_l2", S.SIM_NEG_L2)):
        ms = timed(lambda: S.stlite_tsg_similarity(prob, sim, dk, tmp, out.ws_tsg, stream))
        entry[name] = roofline_entry(model["tsg_rho"], ms)
    S.stlite_tsg_rho(prob, dk, rho, out.ws_tsg, stream)
    ms = timed(lambda: S.stlite_tsg_fixed_gate(prob, rho, 0.85, out.gate, stream))
    entry["tsg_fixed_gate"] = roofline_entry(model["tsg_threshold"], ms)
    ms = timed(lambda: S.stlite_css_saliency(prob, dk, out.phi, None, stream))
    entry["css_saliency_ungated"] = roofline_entry(model["css_saliency"], ms)
    # Mean-Attention prior (pooling width 7): A_base read, A_mean written
    ms = timed(lambda: S.stlite_mean_attention(prob, out.a_base, 7, tmp, stream))
    entry["mean_attention_w7"] = roofline_entry({"bound": "hbm", "bytes": units * 8.0 * lay.total_tokens}, ms)
    for k in (5, 7, 9):
        ms = timed(lambda: S.stlite_css_saliency_nbhd(prob, k, dk, out.phi, stream))
        e = roofline_entry({"bound": "hbm", "bytes": model["css_saliency"]["bytes"]}, ms)
        e["mfma_tflops"] = round(units * 2.0 * ((k * k - 1) // 2 + 1) * n_vis * w.head_dim / (ms * 1e-3) / 1e12, 2)
        entry[f"css_saliency_{k}x{k}"] = e
    # the concatenated key space (one kept set per layer, D = 512)
    if prob.n_kv_heads in (2, 4):
        n_l = prob.n_layers
        rho_l = torch.empty((n_l, prob.total_tokens), dtype=torch.float32, device="cuda")
        phi_l = torch.empty_like(rho_l)
        ws_c = torch.empty(max(prob.workspace_size(S.CALL_TSG_RHO_CONCAT), 256), dtype=torch.uint8, device="cuda")
        ms = timed(lambda: S.stlite_tsg_rho_concat(prob, dk, rho_l, ws_c, stream))
        entry["tsg_rho_concat"] = roofline_entry(model["tsg_rho"], ms)
        ms = timed(lambda: S.stlite_css_saliency_concat(prob, dk, phi_l, stream))
        entry["css_saliency_concat"] = roofline_entry(
            {"bound": "hbm", "bytes": units * 2.0 * n_vis * w.head_dim + 4.0 * n_l * lay.total_tokens}, ms)
        del rho_l, phi_l, ws_c
    log("variants: " + ", ".join(f"{n} {e['ms']:.3f} ms ({e['frac']:.2f})" for n, e in entry.items()))
    return entry


def measured_peaks(stream):
    """Second denominators measured on this GPU (the published peaks stay the
    roofline's `peak`): the matrix cores in the two MFMA shapes the compression
    kernels use, driven by stlite_probe_mfma with random operands that rotate
    per instruction, and the 32x32x16 shape carrying the window score's vector
    work (fma + exp2 + add per logit); a large hipBLASLt bf16 GEMM
    (torch.matmul); a device copy (torch copy_, bytes read + written); and a
    streaming read of 4 GiB through stlite_probe_read with the default and the
    non-temporal cache policy."""
    import torch
    from paper_2603_00188_amd import stlite as S

    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3

    out = {}
    n_groups = 2048  # 8 waves per SIMD on all 256 CUs
    gen = torch.Generator().manual_seed(0)
    ops = (torch.randn(n_groups * 256 * 128, generator=gen) * 0.25).to(torch.bfloat16).cuda().view(torch.int16)
    sink = torch.empty(n_groups * 256, dtype=torch.float32, device="cuda")
    for name, shape, iters in (("mfma_16x16x32_bf16", S.PROBE_MFMA_16X16X32, 200),
                               ("mfma_32x32x16_bf16", S.PROBE_MFMA_32X32X16, 100),
                               ("mfma_32x32x16_bf16_exp2_mix", S.PROBE_MFMA_32X32X16_EXP2, 100),
                               ("mfma_16x16x32_bf16_exp2_mix", S.PROBE_MFMA_16X16X32_EXP2, 100)):
        t = timed(lambda: S.stlite_probe_mfma(shape, ops, sink, n_groups, iters, stream), 5)
        flops = float(S.PROBE_MFMAS_PER_ITER[shape]) * iters * n_groups * 4 * S.PROBE_FLOPS[shape]
        out[name + "_tflops"] = round(flops / t / 1e12, 1)
    n = 8192
    a = torch.randn((n, n), generator=gen).to(torch.bfloat16).cuda()
    b = torch.randn((n, n), generator=gen).to(torch.bfloat16).cuda()
    with torch.cuda.stream(stream):
        t = timed(lambda: torch.matmul(a, b), 10)
    out["hipblaslt_gemm_8192_bf16_tflops"] = round(2.0 * n ** 3 / t / 1e12, 1)
    src = torch.ones(1 << 31, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    with torch.cuda.stream(stream):
        t = timed(lambda: dst.copy_(src), 10)
    out["device_copy_2gib_gbs"] = round(2.0 * src.numel() / t / 1e9, 1)
    # a streaming read of 4 GiB (stlite_probe_read), default and non-temporal cache policy
    rd = torch.empty(1 << 32, dtype=torch.uint8, device="cuda")
    rd_groups = 8192
    rd_sink = torch.empty(rd_groups * 256, dtype=torch.float32, device="cuda")
    for name, nt in (("hbm_stream_read_4gib_gbs", False), ("hbm_stream_read_4gib_nontemporal_gbs", True)):
        t = timed(lambda: S.stlite_probe_read(rd, rd.numel(), rd_sink, rd_groups, nt, stream), 10)
        out[name] = round(rd.numel() / t / 1e9, 1)
    del a, b, src, dst, ops, sink, rd, rd_sink
    log("measured peaks: " + ", ".join(f"{k} {v}" for k, v in out.items()))
    return out


def chr_harness(prob, q, dk, a_base, out, stream):
    """Cache hit rate (Eq. chr) of the pass's kept sets and of SnapKV mode (the
    same window score, flat top-B, no CSS or gate) against I*, the top-B of the
    first decode query's attention over the full cache.  Here the decode query
    is the last window query, so window voting is close to I* by construction:
    these values describe the synthetic inputs, not GUI traces."""
    import torch
    from paper_2603_00188_amd import stlite as S
    from paper_2603_00188_amd import workload as W
    q_dec = torch.from_numpy(np.ascontiguousarray(W.decode_queries(q)).view(np.int16)).cuda()
    p1 = S.decode_problem(prob)
    snap = torch.empty_like(out.kept)
    S.stlite_select_topk(prob, a_base, None, None, 0.0, snap, None, out.ws, stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    star, _ = S.oracle_set(p1, q_dec, dk, stream=stream)  # warm-up and allocation
    torch.cuda.synchronize()
    e0.record(stream)
    S.oracle_set(p1, q_dec, dk, kept=star, stream=stream)
    hits_st = S.kept_overlap(prob, out.kept, star, stream=stream)
    e1.record(stream)
    hits_sn = S.kept_overlap(prob, snap, star, stream=stream)
    torch.cuda.synchronize()
    B = np.diff(prob.h["cu_budget"]).astype(np.float64)
    rate = lambda h: float(np.mean(h[:, B > 0] / B[B > 0])) if (B > 0).any() else float("nan")
    entry = {"st_lite": round(rate(hits_st.cpu().numpy()), 4),
             "snapkv": round(rate(hits_sn.cpu().numpy()), 4),
             "units": prob.units, "ms_oracle_set_and_overlap": round(e0.elapsed_time(e1), 3)}
    log(f"cache hit rate: ST-Lite {entry['st_lite']:.4f}, SnapKV mode {entry['snapkv']:.4f}")
    return entry


def graph_timing(prob, w, dq, dk, dv, out, reps):
    """The whole pass (compress(), five C calls on one stream) eagerly and as a
    HIP graph captured once and replayed, `reps` times each after one warm-up;
    the replay's kept sets must equal the eager ones bit for bit."""
    import torch
    from paper_2603_00188_amd import stlite as S
    st = torch.cuda.current_stream()
    ev = lambda: torch.cuda.Event(enable_timing=True)
    S.compress(prob, dq, dk, dv, out, alpha=w.alpha, stream=st)
    e0, e1 = ev(), ev()
    e0.record(st)
    for _ in range(reps):
        S.compress(prob, dq, dk, dv, out, alpha=w.alpha, stream=st)
    e1.record(st)
    torch.cuda.synchronize()
    kept_eager = out.kept.clone()
    graph = S.capture_compress(prob, dq, dk, dv, out, alpha=w.alpha)
    graph.replay()
    g0, g1 = ev(), ev()
    g0.record(st)
    for _ in range(reps):
        graph.replay()
    g1.record(st)
    torch.cuda.synchronize()
    if not torch.equal(out.kept, kept_eager):
        raise RuntimeError("graph replay kept a different set than the eager pass")
    eager_ms, graph_ms = e0.elapsed_time(e1) / reps, g0.elapsed_time(g1) / reps
    del graph
    log(f"compress(): eager {eager_ms:.3f} ms, graph replay {graph_ms:.3f} ms")
    return {"eager_ms": round(eager_ms, 4), "replay_ms": round(graph_ms, 4),
            "replay_tokens_per_s": round(int(prob.total_tokens) / (graph_ms * 1e-3), 1),
            "note": "compress() with stlite_tsg_gate (rho, threshold and gate in one call); kept sets of the "
                    "replays equal to the eager pass's"}


def multistep_timing(w, inputs, dk, dv, stream, reps=2):
    """Recompression at every step of the trajectory (problem setup, Eq.
    history_context): step t compresses its own context, frames 0..t with the
    text after each (L_t tokens, B_t = floor(beta L_t)), as one problem per step,
    the way a serving loop calls the library after each step's prefill.  Each
    step's cache is a copy of the first L_t rows of the resident trajectory,
    made before its timing starts.  Per step: the whole pass (five calls, HIP
    events on the launch stream, mean of `reps` after one warm-up) and the
    cache hit rates of its kept sets and of SnapKV mode against I*, the top-B_t
    of the step's decode query (not a window query) over its full cache;
    Eq. chr averages them over the steps and units."""
    import dataclasses
    import torch
    from paper_2603_00188_amd import stlite as S
    from paper_2603_00188_amd import workload as W
    si = W.make_step_inputs(w, base=inputs, pack=False)
    toks, ms, ms_graph, chr_st, chr_sn = [], [], [], [], []
    for i, t in enumerate(si.steps):
        wt = dataclasses.replace(w, seqs=(W.step_prefix_segments(w, t),))
        lay = W.make_layout(wt)
        n = lay.total_tokens
        cu_b = S.budgets(lay.cu_seqlens, *w.beta)
        p = S.Problem(w.n_layers, w.n_q_heads, w.n_kv_heads, w.window, lay.cu_seqlens, lay.cu_frames,
                      lay.frame_meta, cu_b)
        kt = dk[:, :, :n].contiguous()
        vt = dv[:, :, :n].contiguous()
        qt = torch.from_numpy(np.ascontiguousarray(si.q[:, i:i + 1]).view(np.int16)).cuda()
        qd = torch.from_numpy(np.ascontiguousarray(si.q_dec[:, i:i + 1]).view(np.int16)).cuda()
        o = S.Buffers(p, keep_stages=False)
        S.compress(p, qt, kt, vt, o, alpha=w.alpha, stream=stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            S.compress(p, qt, kt, vt, o, alpha=w.alpha, stream=stream)
        e1.record(stream)
        # the same pass captured once into a HIP graph and replayed: one launch
        # per pass instead of its kernels one by one (what a serving loop that
        # recompresses a fixed-shape cache would do); its kept sets must be the
        # eager ones, bit for bit
        kept_eager = o.kept.clone()
        graph = S.capture_compress(p, qt, kt, vt, o, alpha=w.alpha)
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        gs = torch.cuda.current_stream()
        graph.replay()
        g0.record(gs)
        for _ in range(reps):
            graph.replay()
        g1.record(gs)
        torch.cuda.synchronize()
        if not torch.equal(o.kept, kept_eager):
            raise RuntimeError(f"step {t}: graph replay kept a different set than the eager pass")
        snap = torch.empty_like(o.kept)
        S.stlite_select_topk(p, o.a_base, None, None, 0.0, snap, None, o.ws, stream)
        star, _ = S.oracle_set(S.decode_problem(p), qd, kt, stream=stream)
        h_st = S.kept_overlap(p, o.kept, star, stream=stream)
        h_sn = S.kept_overlap(p, snap, star, stream=stream)
        torch.cuda.synchronize()
        B = int(cu_b[-1])
        toks.append(n)
        ms.append(e0.elapsed_time(e1) / reps)
        ms_graph.append(g0.elapsed_time(g1) / reps)
        chr_st.append(float(h_st.cpu().numpy().mean()) / B if B else float("nan"))
        chr_sn.append(float(h_sn.cpu().numpy().mean()) / B if B else float("nan"))
        del kt, vt, o, snap, star, graph
    mean = lambda r: float(np.mean([x for x in r if x == x]))
    entry = {
        "workload": f"{w.name} recompressed at each of its {len(si.steps)} steps; step t: frames 0..t "
                    f"and their text, one problem per step, beta {w.beta[0]}/{w.beta[1]}",
        "steps": len(si.steps), "tokens_total": int(sum(toks)), "ms_total": round(float(sum(ms)), 3),
        "tokens_per_s": round(sum(toks) / (sum(ms) * 1e-3), 1),
        "graph": {"ms_total": round(float(sum(ms_graph)), 3),
                  "tokens_per_s": round(sum(toks) / (sum(ms_graph) * 1e-3), 1),
                  "ms_per_step": [round(x, 4) for x in ms_graph],
                  "note": "each step's pass captured into one HIP graph and replayed; kept sets equal "
                          "to the eager pass's"},
        "per_step": {"tokens": toks, "ms": [round(x, 4) for x in ms],
                     "tokens_per_s": [round(n / (m * 1e-3), 1) for n, m in zip(toks, ms)]},
        "chr_st_lite": round(mean(chr_st), 4), "chr_snapkv": round(mean(chr_sn), 4),
        "chr_per_step_st_lite": [round(x, 4) for x in chr_st],
        "chr_per_step_snapkv": [round(x, 4) for x in chr_sn],
        "decode_query": "sum of the step's element keys and of an earlier frame's changed region, plus noise",
    }
    log(f"multi-step: {entry['steps']} steps, {entry['tokens_total']} tokens in {entry['ms_total']:.2f} ms "
        f"({entry['tokens_per_s'] / 1e6:.2f} M tokens/s; graph replay {entry['graph']['ms_total']:.2f} ms); CHR ST-Lite {entry['chr_st_lite']:.4f}, "
        f"SnapKV mode {entry['chr_snapkv']:.4f}")
    return entry


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=3)
    ap.add_argument("--beta", default=None, metavar="NUM/DEN",
                    help="budget ratio as a fraction (default: the workload's own)")
    ap.add_argument("--screen", default="iid", choices=("iid", "gui"),
                    help="screen model of the synthetic frames: independent patches (default) or flat "
                         "textured panels with UI elements")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-baseline-only", action="store_true",
                    help="only time the fp64 oracle on the host for --config (no GPU work) and print it")
    ap.add_argument("--literal", action="store_true",
                    help="with --cpu-baseline-only: time the pure-Python loop twin of the oracle instead "
                         "(the tiny workload, --config 0)")
    ap.add_argument("--pass-only", action="store_true",
                    help="time the pass only: no measured peaks, decode, variants, cache hit rate or "
                         "multi-step timings (for counter runs)")
    ap.add_argument("--overlap", action="store_true",
                    help="run score, TSG and CSS on three concurrent streams")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="BYTES",
                    help="only run a device copy of BYTES bytes three times (counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        sys.stderr.write("bench.py measures one GPU only: the compression pass is per (layer, kv head) and "
                         "this build runs it on a single MI355X; --gpus must be 1\n")
        sys.exit(2)

    from paper_2603_00188_amd import workload as W
    beta = tuple(int(x) for x in args.beta.split("/")) if args.beta else None
    if args.cpu_baseline_only:
        w = W.config(args.config, beta).with_screen(args.screen)
        log(f"generating {w.name}: {w.total_tokens} tokens x {w.n_layers} layers")
        base = cpu_baseline(w, W.make_inputs(w, workers=16), literal=args.literal)
        print(json.dumps({"config": w.name, "tokens": w.total_tokens, "cpu_baseline": base}), flush=True)
        return

    import torch
    from paper_2603_00188_amd import stlite as S

    S.load()  # fails loudly without the HIP library
    torch.cuda.set_device(0)
    if args.copy_probe:
        copy_probe(args.copy_probe)
        return
    w = W.config(args.config, beta).with_screen(args.screen)
    log(f"generating {w.name}: {w.total_tokens} tokens x {w.n_layers} layers")
    inputs = W.make_inputs(w, workers=16)
    scene, k, v, q = inputs
    lay = scene.layout
    cu_budget = S.budgets(lay.cu_seqlens, *w.beta)
    prob = S.Problem(w.n_layers, w.n_q_heads, w.n_kv_heads, w.window, lay.cu_seqlens, lay.cu_frames,
                     lay.frame_meta, cu_budget)
    dk = torch.from_numpy(k.view(np.int16)).cuda()
    dv = torch.from_numpy(v.view(np.int16)).cuda()
    dq = torch.from_numpy(q.view(np.int16)).cuda()
    out = S.Buffers(prob, keep_stages=False)
    rho = torch.empty_like(out.a_base)
    torch.cuda.synchronize()
    log(f"inputs resident: K+V {2 * dk.numel() * 2 / 1e9:.2f} GB")

    stream = torch.cuda.current_stream()
    s_tsg = out.side[0]
    names = ["score_window", "tsg_rho", "tsg_threshold", "css_saliency", "select_topk", "compact_kv"]
    # Concurrent streams gain about 1% here (the two MFMA passes share the
    # matrix cores) and blur the per-kernel times, so the timed step is serial.
    overlap = args.overlap

    def step(ev=None):
        # With --overlap the window score runs on the main stream while TSG
        # and then the gated CSS run on a side stream.  The TSG step runs as
        # its two calls (rho, then threshold and gate), so that the rho GEMM
        # is timed on its own.  Per-call events sit on the stream of their call.
        st = (stream, s_tsg) if overlap else (stream, stream)
        if overlap:
            start = torch.cuda.Event()
            start.record(stream)
            s_tsg.wait_event(start)
        if ev: ev["score_window"][0].record(st[0])
        S.stlite_score_window(prob, dq, dk, out.a_base, out.ws, st[0])
        if ev: ev["score_window"][1].record(st[0])
        if ev: ev["tsg_rho"][0].record(st[1])
        S.stlite_tsg_rho(prob, dk, rho, out.ws_tsg, st[1])
        if ev: ev["tsg_rho"][1].record(st[1])
        if ev: ev["tsg_threshold"][0].record(st[1])
        S.stlite_tsg_threshold(prob, rho, None, out.gate, out.ws_tsg, st[1])
        if ev: ev["tsg_threshold"][1].record(st[1])
        if ev: ev["css_saliency"][0].record(st[1])
        S.stlite_css_saliency(prob, dk, out.phi, out.gate, st[1])
        if ev: ev["css_saliency"][1].record(st[1])
        if overlap:
            done = torch.cuda.Event()
            done.record(s_tsg)
            stream.wait_event(done)
        if ev: ev["select_topk"][0].record(stream)
        S.stlite_select_topk(prob, out.a_base, out.phi, out.gate, w.alpha, out.kept, None, out.ws, stream)
        if ev: ev["select_topk"][1].record(stream)
        if ev: ev["compact_kv"][0].record(stream)
        S.stlite_compact_kv(prob, dk, dv, out.kept, out.k_out, out.v_out, stream)
        if ev: ev["compact_kv"][1].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [{n: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for n in names}
           for _ in range(args.steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(args.steps):
        step(evs[i])
    t_end.record(stream)
    torch.cuda.synchronize()
    ms_step = t_start.elapsed_time(t_end) / args.steps
    per_call = {n: float(np.mean([e[n][0].elapsed_time(e[n][1]) for e in evs])) for n in names}
    log(f"step {ms_step:.3f} ms; calls: " + ", ".join(f"{n} {t:.3f}" for n, t in per_call.items()))

    model = work_model(w, lay, cu_budget)
    stages = {n: roofline_entry(model[n], per_call[n]) for n in names}
    dom = max(names, key=lambda n: per_call[n])
    # Selections: one resident launch when every sequence has at most 32,768
    # tokens (and 1,024 frames), the splitter launches otherwise.
    seqlens = np.diff(np.asarray(lay.cu_seqlens))
    frames = np.diff(np.asarray(lay.cu_frames))
    resident = int(seqlens.max()) <= 32768 and int(frames.max(initial=0)) <= 1024
    kernel_of = {"score_window": "score_pass_kernel<1> + score_pass_kernel<2>",
                 "tsg_rho": "rho_kernel",
                 "tsg_threshold": "gate_resident_kernel" if resident else
                                  "gate_split_sample_kernel + gate_split_classify_kernel + gate_split_resolve_kernel",
                 "css_saliency": "css_kernel<true>",
                 "select_topk": "select_resident_kernel" if resident else
                                "select_split_sample_kernel + select_split_classify_kernel + "
                                "select_split_resolve_kernel + select_split_emit_kernel",
                 "compact_kv": "compact_kernel"}
    roof = dict(stages[dom])
    roof.pop("ms")
    roof["traffic"] = measured_traffic(kernel_of[dom], w.name)
    roof["traffic_source"] = (f"profiles/{kernel_of[dom]}_{w.name}_traffic.md: rocprofv3 FETCH_SIZE + WRITE_SIZE "
                              "per launch, each scaled by a 1 GiB copy; taken in a separate counter run of the "
                              "same sources (null when the kernel's sources have changed since)")
    roof["kernel"] = kernel_of[dom]
    roof["call"] = "stlite_" + dom
    roof["ms_per_launch"] = round(per_call[dom], 4)

    grid = (f"{int(lay.frame_meta[0][1])}x{int(lay.frame_meta[0][2])}" if len(lay.frame_meta) else "no")
    result = {
        "metric": METRIC,
        "value": round(lay.total_tokens / (ms_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{w.name}: {lay.n_seqs} sequence(s), {len(lay.frame_meta)} frames of "
                        f"{grid} patches + text, {lay.total_tokens} tokens, {w.n_layers} layers, "
                        f"{w.n_q_heads}/{w.n_kv_heads} heads, head_dim {w.head_dim}, window {w.window}, "
                        f"beta {w.beta[0]}/{w.beta[1]}, alpha {w.alpha}",
            "tokens": lay.total_tokens, "layers": w.n_layers, "kv_heads": w.n_kv_heads,
            "q_heads": w.n_q_heads, "window": w.window, "beta": f"{w.beta[0]}/{w.beta[1]}",
            "budget_per_unit": int(cu_budget[-1]), "screen": w.screen,
            "streams": "score | tsg_rho+tsg_threshold+css, then select, compact" if overlap else "one stream",
        },
        "roofline": roof,
        "stages": stages,
    }
    if args.pass_only:
        if not args.no_cpu_baseline:
            result["cpu_baseline"] = cpu_baseline(w, inputs)
        print(json.dumps(result), flush=True)
        return
    peaks = measured_peaks(stream)
    result["measured_peaks"] = peaks
    mp = peaks["mfma_16x16x32_bf16_tflops"] if roof["bound"] == "mfma" else peaks["device_copy_2gib_gbs"]
    roof["measured_peak"] = mp
    roof["frac_of_measured_peak"] = round(roof["achieved"] / mp, 4)
    # the score passes execute twice the algorithmic flops; their shape and
    # instruction mix is the exp2 probe's
    sw = stages["score_window"]
    sw["executed_tflops"] = round(2.0 * sw["achieved"], 2)
    sw["measured_peak"] = peaks["mfma_32x32x16_bf16_exp2_mix_tflops"]
    sw["executed_frac_of_measured_peak"] = round(2.0 * sw["achieved"] / sw["measured_peak"], 4)
    result["graph"] = graph_timing(prob, w, dq, dk, dv, out, args.steps)
    result["decode"] = decode_timing(prob, w, q, dk, dv, out, stream)
    result["variants"] = variants_timing(prob, w, lay, cu_budget, dk, rho, out, stream)
    step()  # the pass's kept sets again (the variants overwrote phi and gate)
    result["chr"] = chr_harness(prob, q, dk, out.a_base, out, stream)
    if lay.n_seqs == 1 and len(lay.frame_meta) > 1:
        del out, rho
        result["multistep"] = multistep_timing(w, inputs, dk, dv, stream)
    if not args.no_cpu_baseline:
        log("timing the fp64 oracle on the host (cpu baseline)")
        result["cpu_baseline"] = cpu_baseline(w, inputs)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
