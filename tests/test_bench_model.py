"""The benchmark's host-side model: the algorithmic work each call is priced
at (the numerators of the roofline fractions), the fraction arithmetic, and
the guard that drops a committed traffic figure once its kernel's sources
change.  No GPU work."""
import importlib.util
import os

import numpy as np
import pytest

from paper_2603_00188_amd import workload as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _budgets(lay, beta):
    lens = np.diff(lay.cu_seqlens).astype(np.int64)
    return np.concatenate([[0], np.cumsum(lens * beta[0] // beta[1])])


def test_work_model_trajectory_per_unit_figures(bench):
    """At the 150,528-token trajectory (48 frames of 36 x 80, 256 text tokens
    after each; G = 7, window 64, beta = 1/5) the per-unit work is, written out
    by hand: N_hist = 47 * 2880, N_cur = 2880, N_vis = 48 * 2880, B = 30,105."""
    w = W.config(3)
    lay = W.make_layout(w)
    cu_b = _budgets(lay, w.beta)
    m = bench.work_model(w, lay, cu_b)
    units = 28 * 4
    L, d, rows = 150528, 128, 7 * 64
    n_hist, n_cur, n_vis, B = 47 * 2880, 2880, 48 * 2880, 30105
    assert int(cu_b[-1]) == B
    per = {k: {q: v[q] / units for q in ("flops", "bytes")} for k, v in m.items()}
    assert per["score_window"]["flops"] == 2 * rows * L * d                # 17.26 GFLOP
    assert per["score_window"]["bytes"] == 2 * L * d * 2 + 4 * L
    assert per["tsg_rho"]["flops"] == 2 * n_hist * n_cur * d               # 99.8 GFLOP
    assert per["tsg_rho"]["bytes"] == 2 * (n_hist + n_cur) * d + 4 * L
    assert per["tsg_threshold"]["bytes"] == 4 * n_hist + L                 # 0.69 MB
    assert per["css_saliency"]["bytes"] == 2 * n_vis * d + 4 * L           # 36.0 MB
    assert per["select_topk"]["bytes"] == 9 * L + 4 * B                    # 1.47 MB
    assert per["compact_kv"]["bytes"] == 4 * B * d * 2                     # 30.8 MB
    assert abs(per["score_window"]["flops"] - 17.26e9) < 0.01e9
    assert abs(per["tsg_rho"]["flops"] - 99.8e9) < 0.1e9
    assert abs(per["css_saliency"]["bytes"] - 36.0e6) < 0.05e6


def test_work_model_ragged_batch_sums_sequences(bench):
    """The ragged batch: the rho contraction is summed per sequence (each
    sequence's history against its own current frame), never across them."""
    w = W.config(4)
    lay = W.make_layout(w)
    cu_b = _budgets(lay, w.beta)
    m = bench.work_model(w, lay, cu_b)
    units = w.n_layers * w.n_kv_heads
    want = 0
    for s in range(lay.n_seqs):
        sizes = [int(r) * int(c) for _, r, c in lay.seq_frames(s)]
        want += 2 * sum(sizes[:-1]) * sizes[-1] * w.head_dim
    assert m["tsg_rho"]["flops"] == units * want
    total_hist = sum(sum(int(r) * int(c) for _, r, c in lay.seq_frames(s)[:-1]) for s in range(lay.n_seqs))
    current = sum(int(lay.seq_frames(s)[-1][1]) * int(lay.seq_frames(s)[-1][2]) for s in range(lay.n_seqs))
    all_patches = sum(int(r) * int(c) for _, r, c in lay.frame_meta)
    assert all_patches == total_hist + current      # one current frame per sequence
    assert m["tsg_threshold"]["bytes"] == units * (4 * total_hist + lay.total_tokens)
    assert m["css_saliency"]["bytes"] == units * (2 * all_patches * w.head_dim + 4 * lay.total_tokens)


def test_roofline_entry_fractions(bench):
    e = bench.roofline_entry({"bound": "mfma", "flops": 2.5e15 * 1e-3, "bytes": 0.0}, 2.0)
    assert e["unit"] == "TFLOP/s" and e["achieved"] == 1250.0 and e["frac"] == 0.5 and e["peak"] == 2500.0
    e = bench.roofline_entry({"bound": "hbm", "flops": 0.0, "bytes": 4e9}, 1.0)
    assert e["unit"] == "GB/s" and e["achieved"] == 4000.0 and e["frac"] == 0.5 and e["peak"] == 8000.0


def test_measured_traffic_follows_the_source_digest(bench, tmp_path, monkeypatch):
    """A committed traffic figure is used only while its digest matches the
    kernel's sources; a stale or missing summary gives None."""
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    assert bench.measured_traffic("rho_kernel", "w") is None          # no summary
    good = bench.source_digest("rho_kernel")
    (tmp_path / "rho_kernel_w_traffic.md").write_text(
        f"# t\n\n- source_digest: `{good}`\n- hbm_bytes_per_launch: 4701373011\n")
    assert bench.measured_traffic("rho_kernel", "w") == 4701373011.0
    (tmp_path / "rho_kernel_w_traffic.md").write_text(
        "# t\n\n- source_digest: `0000000000000000`\n- hbm_bytes_per_launch: 4701373011\n")
    assert bench.measured_traffic("rho_kernel", "w") is None          # sources changed
    assert bench.measured_traffic("compact_kernel", "w") is None      # no sources listed


def test_bench_refuses_more_than_one_gpu():
    """The benchmark measures one GPU: --gpus above 1 exits with a message
    before touching any device."""
    import subprocess
    import sys
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr or "single MI355X" in r.stderr
    assert r.stdout == ""
