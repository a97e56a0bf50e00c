"""GPU parity of the cache hit rate harness (Eq. chr) against the fp64 oracle.

For every compared unit and sequence:
  I*    the GPU's oracle set (stlite_score_window on the one-query window of the
        decode query, stlite_select_topk without CSS or gate) against the
        oracle's top-B of the decode attention: exactly B ascending tokens;
        tokens in the symmetric difference must score within 1e-4 |a_B| of
        the oracle's B-th score a_B (the kept-set rule of the pass)
  hits  stlite_kept_overlap bit-exact against a set intersection of the same
        GPU lists on the host (integer work)
  CHR   hits / B against the oracle's CHR of the oracle's own sets, within
        (|kept_gpu xor kept_ref| + |I*_gpu xor I*_ref|) / (2 B): every swapped
        pair inside a tie band moves the count by at most one
"""
import numpy as np
import pytest

from paper_2603_00188_amd import workload as W

pytestmark = pytest.mark.gpu

BAND = 1e-4


@pytest.fixture(scope="module")
def torch_cuda():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch


def _mods():
    from oracle import stlite_oracle as O
    from paper_2603_00188_amd import stlite as S
    from tests import gpu_harness as H
    from tests.test_gpu_parity import SMALL
    return O, S, H, SMALL


def run_chr(case, q_dec_bits=None):
    """Kept sets of ST-Lite and of SnapKV mode, I*, and both hit counts, on the GPU.
    q_dec_bits [layers][seqs][Hq][d]: the decode queries (default: each head's
    last window query)."""
    import torch
    O, S, H, _ = _mods()
    res = case.run()
    out = case.out
    snap = torch.empty_like(out.kept)
    S.stlite_select_topk(case.prob, out.a_base, None, None, 0.0, snap, None, out.ws)
    if q_dec_bits is None:
        q_dec_bits = W.decode_queries(case.q)
    q_dec_bits = np.ascontiguousarray(q_dec_bits)
    q_dec = torch.from_numpy(q_dec_bits.view(np.int16)).cuda()
    p1 = S.decode_problem(case.prob)
    star, _ = S.oracle_set(p1, q_dec, case.dk)
    hits_st = S.kept_overlap(case.prob, out.kept, star)
    hits_sn = S.kept_overlap(case.prob, snap, star)
    torch.cuda.synchronize()
    Bt = case.prob.total_budget
    return dict(res=res, snap=snap[:, :Bt].cpu().numpy(), star=star[:, :Bt].cpu().numpy(),
                hits_st=hits_st.cpu().numpy(), hits_sn=hits_sn.cpu().numpy(), q_dec=q_dec_bits)


def check_chr_unit(case, r, layer, kv, s, ref=None):
    O, S, H, _ = _mods()
    w = case.w
    u = layer * w.n_kv_heads + kv
    a, b = int(case.lay.cu_seqlens[s]), int(case.lay.cu_seqlens[s + 1])
    cb = case.cu_budget
    B = int(cb[s + 1] - cb[s])
    where = f"{w.name} layer {layer} kv {kv} seq {s}"
    if ref is None:
        ref = case.oracle(layer, kv, s)
    kept_st = r["res"]["kept"][u, cb[s]:cb[s + 1]] - a
    kept_sn = r["snap"][u, cb[s]:cb[s + 1]] - a
    star = r["star"][u, cb[s]:cb[s + 1]] - a
    # hits: exact on the GPU's own lists
    assert r["hits_st"][u, s] == len(np.intersect1d(kept_st, star)), f"{where}: ST-Lite hits"
    assert r["hits_sn"][u, s] == len(np.intersect1d(kept_sn, star)), f"{where}: SnapKV hits"
    if B == 0:
        return {}
    # I* against the oracle's top-B of the decode attention
    Qd = O.bf16_to_f64(r["q_dec"][layer, s, kv * w.group:(kv + 1) * w.group])
    K = O.bf16_to_f64(case.k[layer, kv, a:b])
    a_dec = O.decode_attention_scores(Qd, K)
    star_ref = O.chr_oracle_set(a_dec, B)
    assert len(star) == B and (np.diff(star) > 0).all() and star.min() >= 0 and star.max() < b - a, where
    sym_star = np.setxor1d(star, star_ref)
    if len(sym_star):
        aB = np.sort(a_dec.astype(np.float32))[::-1][B - 1]
        far = sym_star[~(np.abs(a_dec[sym_star] - aB) <= BAND * abs(aB))]
        assert len(far) == 0, f"{where}: I* differs away from the B-th attention at {far[:10]}"
    # CHR of the oracle's own sets: ST-Lite and SnapKV mode
    snap_ref = O.select_topk(ref["A"], B)
    out = {}
    for name, kept, kept_ref, hits in (("st_lite", kept_st, ref["kept"], r["hits_st"][u, s]),
                                       ("snapkv", kept_sn, snap_ref, r["hits_sn"][u, s])):
        chr_gpu = hits / B
        chr_ref = O.cache_hit_rate(kept_ref, star_ref)
        slack = (len(np.setxor1d(kept, kept_ref)) + len(sym_star)) / (2 * B)
        assert abs(chr_gpu - chr_ref) <= slack + 1e-12, f"{where}: {name} CHR {chr_gpu} vs {chr_ref}"
        out[name] = chr_gpu
    return out


@pytest.mark.parametrize("name", ["ragged", "tiles", "dups", "beta_tiny", "g8w64"])
def test_chr_small_all_units(torch_cuda, name):
    O, S, H, SMALL = _mods()
    case = H.Case(SMALL[name])
    r = run_chr(case)
    got = []
    for layer in range(case.n_layers):
        for kv in range(case.w.n_kv_heads):
            for s in range(case.lay.n_seqs):
                got.append(check_chr_unit(case, r, layer, kv, s))
    H.log(f"chr {name}: " + ", ".join(f"{k} {np.mean([g[k] for g in got if k in g]):.3f}"
                                      for k in ("st_lite", "snapkv")))


def test_kept_overlap_multi_span_and_orders(torch_cuda):
    """Sequences longer than one 65,536-token span and set pairs with known
    overlaps (equal sets, random sets, an empty budget)."""
    import torch
    O, S, H, _ = _mods()
    cu = np.array([0, 150000, 150010, 220000], np.int32)
    cub = np.array([0, 30000, 30000, 44000], np.int32)
    p = S.Problem(1, 2, 2, 1, cu, [0, 0, 0, 0], np.zeros((0, 3), np.int32), cub)
    rng = np.random.default_rng(7)
    A = np.zeros((2, 44000), np.int32)
    Bl = np.zeros((2, 44000), np.int32)
    want = np.zeros((2, 3), np.int64)
    for u in range(2):
        for s in range(3):
            n = cub[s + 1] - cub[s]
            if n == 0:
                continue
            pool = np.arange(cu[s], cu[s + 1])
            a_set = np.sort(rng.choice(pool, n, replace=False))
            b_set = a_set if u == 0 and s == 0 else np.sort(rng.choice(pool, n, replace=False))
            A[u, cub[s]:cub[s + 1]] = a_set
            Bl[u, cub[s]:cub[s + 1]] = b_set
            want[u, s] = len(np.intersect1d(a_set, b_set))
    da, db = torch.from_numpy(A).cuda(), torch.from_numpy(Bl).cuda()
    hits = S.kept_overlap(p, da, db)
    torch.cuda.synchronize()
    assert np.array_equal(hits.cpu().numpy(), want)
    assert hits.cpu().numpy()[0, 0] == 30000


@pytest.mark.timeout(900)
def test_chr_trajectory_sampled(torch_cuda):
    """The 150,528-token trajectory in the benchmark's launch configuration:
    ST-Lite and SnapKV CHR on sampled units against the oracle."""
    O, S, H, _ = _mods()
    w = W.config(3)
    H.log(f"chr trajectory: generate L={w.total_tokens} x {w.n_layers} layers")
    case = H.Case(w)
    r = run_chr(case)
    for unit in ((0, 0, 0), (13, 2, 0), (27, 3, 0)):
        got = check_chr_unit(case, r, *unit)
        H.log(f"chr trajectory unit {unit}: {got}")
    B = case.prob.total_budget
    H.log(f"chr trajectory mean over all units: ST-Lite {r['hits_st'].mean() / B:.4f}, "
          f"SnapKV {r['hits_sn'].mean() / B:.4f}")


@pytest.mark.timeout(900)
def test_chr_ragged_batch_sampled(torch_cuda):
    """The ragged batch of 8 trajectories (two of its layers): hits of every
    unit and sequence exact, CHR of sampled sequences against the oracle."""
    O, S, H, _ = _mods()
    w = W.config(4)
    H.log(f"chr ragged batch: generate L={w.total_tokens} x 2 layers")
    case = H.Case(w, layers=[0, 27])
    r = run_chr(case)
    cb = case.cu_budget
    for u in range(case.prob.units):
        for s in range(case.lay.n_seqs):
            a = int(case.lay.cu_seqlens[s])
            kept = r["res"]["kept"][u, cb[s]:cb[s + 1]]
            star = r["star"][u, cb[s]:cb[s + 1]]
            assert r["hits_st"][u, s] == len(np.intersect1d(kept, star)), (u, s)
            assert r["hits_sn"][u, s] == len(np.intersect1d(r["snap"][u, cb[s]:cb[s + 1]], star)), (u, s)
            assert (star >= a).all() and (star < case.lay.cu_seqlens[s + 1]).all()
    for unit in ((0, 0, 0), (0, 3, 4), (1, 1, 7), (1, 2, 2)):
        H.log(f"chr ragged batch unit {unit}: {check_chr_unit(case, r, *unit)}")

