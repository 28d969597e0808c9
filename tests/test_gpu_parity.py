"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Inputs come from the seeded generator only; expected values come from the
oracle only.  Every case prints what it runs before touching the GPU.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2609_04852_amd import kvmem as K
from paper_2609_04852_amd import workload as W
from paper_2609_04852_amd.step import LayerState

from parity import (assert_index_bitwise, check_attention, check_scores, check_selection, log, oracle_pool)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    K.lib()  # raises if the library is not built
    yield
    torch.cuda.synchronize()


def oracle_mode(cfg):
    return oracle.MEAN_ALL if cfg.mode == W.MEAN_ALL else oracle.MAX_GROUP


def run_case(cfg, seed, layer=0, budget=None, lpt=None, e2e=True, stats=None):
    """Generate, run the oracle and the GPU path for one layer, and compare."""
    budget = cfg.budget_tokens if budget is None else budget
    log(f"[case] {cfg.name} seed={seed} layer={layer} M={cfg.n_blocks} Hkv={cfg.n_kv_heads} "
        f"Hq={cfg.n_q_heads} d={cfg.head_dim} Bt={cfg.block_tokens} {cfg.kv_dtype} n_q={cfg.n_q} "
        f"S={cfg.sink_blocks} Rr={cfg.n_recent} budget={budget} mode={cfg.mode}")
    w = W.generate(cfg, seed, layers=layer + 1)
    kp, vp_pool, b2p = w.k_pool[layer], w.v_pool[layer], w.block_to_page
    q_l = w.q[0, layer:layer + 1]  # [1][n_q][Hq][d]
    S, Rr = cfg.sink_blocks, cfg.n_recent
    # ---- oracle
    kp_o, vp_o = oracle_pool(cfg, kp), oracle_pool(cfg, vp_pool)
    index_ref = oracle.mean_k(kp_o, b2p)
    rel = oracle.block_relevance(q_l, index_ref[None], S, Rr, oracle_mode(cfg))
    k_eff = oracle.k_eff(budget, budget, cfg.block_tokens, cfg.n_blocks, S, Rr)
    vb_ref, vp_ref = oracle.select(rel, S, Rr, k_eff, b2p)
    last = cfg.block_tokens if lpt is None else lpt
    out_ref, lse_ref = oracle.view_attention(q_l[0], kp_o, vp_o, vp_ref, last_page_tokens=last)
    # ---- GPU
    log("  gpu: build_index")
    st = LayerState(cfg, kp, vp_pool, b2p, budget_tokens=budget)
    st.build_index()
    torch.cuda.synchronize()
    assert_index_bitwise(st.index_rows(), index_ref)
    log("  gpu: select")
    qd = torch.from_numpy(np.ascontiguousarray(q_l)).cuda()
    n_view = st.select(qd)
    torch.cuda.synchronize()
    assert n_view == S + k_eff + Rr
    vb, vpg = st.view_blocks.cpu().numpy(), st.view_pages.cpu().numpy()
    sel_stats = check_selection(vb, vpg, rel, b2p, S, Rr, k_eff, ref_view=vb_ref)
    worst = check_scores(st.scores.cpu().numpy(), rel, S, Rr)
    log(f"  selection ok: {sel_stats}, worst score rel err {worst:.2e}")
    log("  gpu: attention on the oracle's view")
    out, lse = st.attend(qd[0], torch.from_numpy(vp_ref).cuda(), last_page_tokens=last)
    torch.cuda.synchronize()
    err = check_attention(out.cpu().numpy(), lse.cpu().numpy(), out_ref, lse_ref, cfg.kv_dtype)
    log(f"  attention ok: max abs err out {err[0]:.2e} lse {err[1]:.2e}")
    if e2e:
        # end to end: the GPU's attention on the GPU's own view, against the
        # oracle on that same view (it may differ from the oracle's view inside
        # the tie band, where either choice is correct)
        same = np.array_equal(vb, vb_ref)
        log(f"  gpu: attention on its own view ({'equal to' if same else 'in-band different from'} the oracle's)")
        out2, lse2 = st.attend(qd[0], last_page_tokens=last)
        torch.cuda.synchronize()
        if same:
            own_ref, own_lse = out_ref, lse_ref
        else:
            own_ref, own_lse = oracle.view_attention(q_l[0], kp_o, vp_o, vpg, last_page_tokens=last)
        e2 = check_attention(out2.cpu().numpy(), lse2.cpu().numpy(), own_ref, own_lse, cfg.kv_dtype)
        log(f"  end-to-end attention ok: max abs err out {e2[0]:.2e} lse {e2[1]:.2e}")
    if stats is not None:
        stats.update(sel_stats)
    return st, w


@pytest.mark.parametrize("seed", range(6))
def test_tiny(seed):
    run_case(W.CONFIGS["tiny"], seed)


@pytest.mark.parametrize("name", ["64k", "256k"])
def test_mid_configs(name):
    run_case(W.CONFIGS[name], W.CONFIGS[name].seed)


def test_1m():
    run_case(W.CONFIGS["1m"], W.CONFIGS["1m"].seed)


def test_1m_mtp4_layer0():
    run_case(W.CONFIGS["1m_mtp4"], W.CONFIGS["1m_mtp4"].seed, layer=0)


@pytest.mark.parametrize("mode", [W.MEAN_ALL, W.MAX_GROUP])
def test_1m_mixture_4_rows(mode):
    """Clustered (mixture) keys at 4 query rows per KV head: the vector scoring
    kernel's fp32 dot products on the heavy-tailed scores of the 4-layer
    workload's keys (layer 0, one query token), both reductions."""
    cfg = W.CONFIGS["1m_mtp4"].replace(name=f"1m_mix_q1_{mode}", n_q=1, mode=mode)
    run_case(cfg, cfg.seed, layer=0)


SHAPES = [
    # Hkv, Hq, d, Bt, dtype, M, S, Rr, n_q, mode, budget blocks beyond sink+recent
    (2, 8, 128, 32, "f32", 700, 3, 5, 2, W.MEAN_ALL, 100),
    (4, 4, 64, 64, "bf16", 333, 0, 1, 1, W.MAX_GROUP, 41),
    (1, 8, 64, 16, "bf16", 1500, 2, 7, 2, W.MAX_GROUP, 230),
    (8, 16, 128, 16, "bf16", 2000, 0, 33, 4, W.MEAN_ALL, 517),
    (16, 32, 64, 32, "bf16", 900, 1, 9, 1, W.MEAN_ALL, 77),
    (32, 64, 128, 16, "bf16", 300, 0, 4, 1, W.MAX_GROUP, 50),
    (2, 2, 128, 64, "f32", 129, 0, 1, 1, W.MEAN_ALL, 1),
    # 16 query rows per KV head (bf16): the matrix-core attention path
    (2, 16, 128, 16, "bf16", 700, 0, 5, 2, W.MEAN_ALL, 100),
    (4, 16, 64, 32, "bf16", 500, 1, 3, 4, W.MAX_GROUP, 60),
    (2, 8, 128, 64, "bf16", 260, 0, 2, 4, W.MAX_GROUP, 37),
    # fp32 K/V, d128, 64-token pages, 8 rows per KV head (two 4-row workgroups)
    (2, 16, 128, 64, "f32", 150, 0, 2, 1, W.MEAN_ALL, 20),
    # the largest KV head count the library takes (64), no grouping
    (64, 64, 64, 16, "bf16", 200, 1, 2, 1, W.MAX_GROUP, 30),
    (64, 128, 128, 32, "bf16", 150, 0, 3, 2, W.MEAN_ALL, 25),
    # 4 sink blocks, G = 8 (8 rows per KV head on the matrix cores)
    (4, 32, 128, 16, "bf16", 800, 4, 6, 1, W.MEAN_ALL, 90),
    # GQA widths that are not powers of two, and KV head counts that are not
    # either: 3, 5, 6 and 7 rows per KV head (vector scoring), 12 (3 query
    # tokens at G = 4) and 15 (padded 16-row matrix-core scoring), 20 and 21
    # (16-row chunks with a ragged last chunk)
    (8, 24, 128, 16, "bf16", 1200, 0, 9, 1, W.MEAN_ALL, 200),
    (8, 40, 128, 16, "bf16", 900, 1, 7, 1, W.MAX_GROUP, 150),
    (6, 36, 128, 32, "bf16", 700, 0, 5, 1, W.MEAN_ALL, 100),
    (4, 28, 64, 16, "bf16", 800, 2, 6, 1, W.MAX_GROUP, 90),
    (8, 32, 128, 16, "bf16", 1000, 0, 8, 3, W.MEAN_ALL, 160),
    (3, 15, 128, 64, "bf16", 400, 0, 3, 3, W.MAX_GROUP, 60),
    (2, 10, 128, 16, "bf16", 600, 0, 4, 4, W.MAX_GROUP, 80),
    (3, 21, 64, 32, "f32", 400, 1, 3, 3, W.MEAN_ALL, 50),
    (5, 5, 128, 64, "bf16", 300, 0, 2, 1, W.MAX_GROUP, 40),
    (6, 18, 64, 16, "f32", 500, 0, 6, 1, W.MAX_GROUP, 70),
]


def shape_cfg(hkv, hq, d, bt, dt, m, s, rr, nq, mode, extra, planted=3):
    return W.small_config(n_kv_heads=hkv, n_q_heads=hq, head_dim=d, block_tokens=bt, kv_dtype=dt,
                          history_tokens=m * bt, recent_tokens=rr * bt, sink_blocks=s,
                          budget_tokens=(s + rr + extra) * bt, n_q=nq, mode=mode, n_planted=planted)


@pytest.mark.parametrize("shape", SHAPES, ids=[f"s{i}" for i in range(len(SHAPES))])
def test_shapes(shape):
    run_case(shape_cfg(*shape), 11)


@pytest.mark.parametrize("which", ["none", "all"])
def test_budget_extremes(which):
    cfg = shape_cfg(4, 16, 128, 16, "bf16", 600, 2, 6, 1, W.MEAN_ALL, 0)
    budget = (2 + 6) * 16 if which == "none" else 10**9
    run_case(cfg, 3, budget=budget)


@pytest.mark.parametrize("k", [0, 1])
@pytest.mark.parametrize("mode", [W.MEAN_ALL, W.MAX_GROUP])
def test_single_candidate(k, mode):
    """Three blocks: a sink, one candidate and a recent block. The candidate's
    relevance is exactly n_q (a softmax over one block); it is kept when the
    budget leaves room for it and dropped otherwise."""
    run_case(shape_cfg(2, 8, 64, 16, "bf16", 3, 1, 1, 1, mode, k, planted=0), 73)


def test_partial_last_page():
    cfg = shape_cfg(2, 8, 128, 32, "bf16", 400, 0, 3, 2, W.MEAN_ALL, 60)
    run_case(cfg, 5, lpt=7)
    run_case(cfg, 6, lpt=1)


def test_full_selection_is_dense_attention():
    cfg = shape_cfg(2, 8, 64, 16, "f32", 300, 1, 2, 1, W.MEAN_ALL, 0)
    log("[case] full selection vs dense attention")
    w = W.generate(cfg, 8)
    st = LayerState(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page, budget_tokens=10**9)
    st.build_index()
    qd = torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda()
    st.select(qd)
    out, lse = st.attend(qd[0])
    torch.cuda.synchronize()
    assert st.view_blocks.cpu().numpy()[0].tolist() == list(range(cfg.n_blocks))
    all_blocks = np.arange(cfg.n_blocks, dtype=np.int32)[None]
    o_ref, l_ref = oracle.masked_dense_attention(w.q[0, 0], w.k_pool[0], w.v_pool[0], w.block_to_page,
                                                 all_blocks)
    check_attention(out.cpu().numpy(), lse.cpu().numpy(), o_ref, l_ref, "f32")


# (blocks, source pages, budget blocks): ~25 ties per score value (ranked
# pairwise), ~1,300 (radix select in LDS), and a budget that ends inside the
# second-best score's ties
TIE_CASES = [(500, 20, 40), (4000, 3, 40), (4000, 3, 2000)]


@pytest.mark.parametrize("case", TIE_CASES, ids=["t25", "t1300", "t1300_deep"])
def test_exact_ties_take_lower_ids(case):
    """Blocks whose pages hold identical keys score identically; the lower ids win."""
    m, n_src, extra = case
    cfg = shape_cfg(2, 8, 128, 16, "bf16", m, 0, 4, 1, W.MEAN_ALL, extra, planted=0)
    log(f"[case] exact ties {case}")
    w = W.generate(cfg, 9)
    kp = w.k_pool[0].copy()
    # every page gets the keys of one of a few source pages: massive exact ties
    src = np.random.default_rng(0).integers(0, n_src, cfg.n_blocks)
    kp[:] = kp[src]
    index_ref = oracle.mean_k(kp, w.block_to_page)
    rel = oracle.block_relevance(w.q[0, :1], index_ref[None], 0, cfg.n_recent)
    k_eff = oracle.k_eff(cfg.budget_tokens, cfg.budget_tokens, 16, cfg.n_blocks, 0, cfg.n_recent)
    vb_ref, _ = oracle.select(rel, 0, cfg.n_recent, k_eff, w.block_to_page)
    st = LayerState(cfg, kp, w.v_pool[0], w.block_to_page)
    st.build_index()
    st.select(torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(st.view_blocks.cpu().numpy(), vb_ref)


def test_incremental_index_build():
    cfg = W.CONFIGS["64k"]
    log("[case] incremental index build")
    w = W.generate(cfg, 1, with_values=False)
    st = LayerState(cfg, w.k_pool[0], None, w.block_to_page)
    st.index.fill_(-1.0)
    for lo, hi in [(0, 1000), (1000, 1001), (1001, 4096)]:
        st.build_index(lo, hi - lo)
    torch.cuda.synchronize()
    assert_index_bitwise(st.index_rows(), oracle.mean_k(w.k_pool[0], w.block_to_page))


def test_deterministic():
    cfg = W.CONFIGS["256k"]
    log("[case] determinism (two runs)")
    w = W.generate(cfg, 2)
    st = LayerState(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page)
    qd = torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda()
    outs = []
    for _ in range(2):
        st.build_index()
        st.select(qd)
        o, l = st.attend(qd[0])
        torch.cuda.synchronize()
        outs.append([t.cpu().numpy().copy() for t in (st.index, st.scores, st.view_blocks, o, l)])
    for a, b in zip(*outs):
        assert np.array_equal(a.view(np.uint8), b.view(np.uint8))


@pytest.mark.parametrize("bt,lpt", [(16, 16), (32, 5), (64, 33)])
def test_random_views_32_rows(bt, lpt):
    """Attention alone with 32 query rows per KV head (two 16-row groups on the
    matrix cores), arbitrary page lists and a partial last page."""
    cfg = shape_cfg(2, 16, 128, bt, "bf16", 300, 0, 2, 4, W.MAX_GROUP, 10)
    log(f"[case] 32 rows per KV head, Bt={bt}, last page {lpt}")
    w = W.generate(cfg, 21)
    rng = np.random.default_rng(5)
    vp = np.stack([rng.choice(cfg.n_blocks, 97, replace=False) for _ in range(2)]).astype(np.int32)
    q = np.ascontiguousarray(w.q[0, 0])
    o_ref, l_ref = oracle.view_attention(q, w.k_pool[0], w.v_pool[0], vp, last_page_tokens=lpt)
    st = LayerState(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page)
    out, lse = st.attend(torch.from_numpy(q).cuda(), torch.from_numpy(vp).cuda(), last_page_tokens=lpt)
    torch.cuda.synchronize()
    check_attention(out.cpu().numpy(), lse.cpu().numpy(), o_ref, l_ref, "bf16")


def test_random_views_per_head():
    """Attention alone on arbitrary page lists (one per KV head), any order."""
    cfg = shape_cfg(4, 16, 128, 32, "bf16", 800, 0, 2, 2, W.MAX_GROUP, 10)
    log("[case] random per-head views")
    w = W.generate(cfg, 12)
    rng = np.random.default_rng(3)
    vp = np.stack([rng.choice(cfg.n_blocks, 257, replace=False) for _ in range(4)]).astype(np.int32)
    o_ref, l_ref = oracle.view_attention(w.q[0, 0], w.k_pool[0], w.v_pool[0], vp, last_page_tokens=13)
    st = LayerState(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page)
    qd = torch.from_numpy(np.ascontiguousarray(w.q[0, 0])).cuda()
    out, lse = st.attend(qd, torch.from_numpy(vp).cuda(), last_page_tokens=13)
    torch.cuda.synchronize()
    check_attention(out.cpu().numpy(), lse.cpu().numpy(), o_ref, l_ref, "bf16")


def test_out_of_range_pages_give_nan():
    """A page id outside the pool is never read; the outputs that need it are NaN."""
    cfg = shape_cfg(2, 8, 64, 16, "f32", 200, 0, 2, 1, W.MAX_GROUP, 20)
    log("[case] out-of-range page ids")
    w = W.generate(cfg, 13)
    st = LayerState(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page)
    qd = torch.from_numpy(np.ascontiguousarray(w.q[0, 0])).cuda()
    vp = np.stack([np.arange(30), np.arange(30, 60)]).astype(np.int32)
    vp[1, 17] = cfg.n_blocks + 1000  # only KV head 1 sees the bad page
    out, lse = st.attend(qd, torch.from_numpy(vp).cuda())
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    assert np.isnan(o[:, 4:]).all() and np.isfinite(o[:, :4]).all()
    o_ref, _ = oracle.view_attention(w.q[0, 0, :, :4], w.k_pool[0][:, :1], w.v_pool[0][:, :1], vp[:1])
    np.testing.assert_allclose(o[:, :4], o_ref, atol=1e-4, rtol=0)
    # the same on the matrix-core path (16 rows per KV head, bf16)
    cfg16 = shape_cfg(2, 16, 128, 16, "bf16", 200, 0, 2, 2, W.MAX_GROUP, 20)
    w16 = W.generate(cfg16, 13)
    st16 = LayerState(cfg16, w16.k_pool[0], w16.v_pool[0], w16.block_to_page)
    q16 = np.ascontiguousarray(w16.q[0, 0])
    out16, _ = st16.attend(torch.from_numpy(q16).cuda(), torch.from_numpy(vp).cuda())
    torch.cuda.synchronize()
    o16 = out16.cpu().numpy()  # [n_q][Hq][d]; heads 0..7 read KV head 0, 8..15 KV head 1
    assert np.isnan(o16[:, 8:]).all() and np.isfinite(o16[:, :8]).all()
    o16_ref, _ = oracle.view_attention(q16[:, :8], w16.k_pool[0][:, :1], w16.v_pool[0][:, :1], vp[:1])
    np.testing.assert_allclose(o16[:, :8], o16_ref, atol=2e-2, rtol=0)
    b2p = w.block_to_page.copy()
    b2p[7] = -3
    st2 = LayerState(cfg, w.k_pool[0], None, b2p)
    st2.build_index()
    torch.cuda.synchronize()
    idx = st2.index_rows()
    assert np.isnan(idx[7]).all()
    ok = np.ones(cfg.n_blocks, bool)
    ok[7] = False
    ref = oracle.mean_k(w.k_pool[0], w.block_to_page)
    assert_index_bitwise(idx[ok], ref[ok])


def test_all_equal_scores_large():
    """Every page holds the same keys: all scores tie, the pivot bin holds every
    candidate (more than the LDS window), and the lowest ids must win."""
    cfg = shape_cfg(1, 4, 64, 16, "bf16", 20480, 3, 5, 1, W.MEAN_ALL, 7000, planted=0)
    log("[case] all scores equal, 20472 candidates")
    w = W.generate(cfg, 14, with_values=False)
    kp = np.broadcast_to(w.k_pool[0][:1], w.k_pool[0].shape).copy()
    st = LayerState(cfg, kp, kp, w.block_to_page)
    st.build_index()
    st.select(torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda())
    torch.cuda.synchronize()
    vb = st.view_blocks.cpu().numpy()[0]
    expect = list(range(3)) + list(range(3, 3 + 7000)) + list(range(20480 - 5, 20480))
    assert vb.tolist() == expect
    np.testing.assert_array_equal(st.view_pages.cpu().numpy()[0], w.block_to_page[vb])


# ---- FP8 K/V (OCP E4M3 codes, one scale per pool) ------------------------
FP8_SHAPES = [
    # Hkv, Hq, d, Bt, M, S, Rr, n_q, mode, extra, scale
    (8, 32, 128, 16, 2000, 0, 33, 1, W.MEAN_ALL, 517, 8 / 448),     # 4 rows per KV head
    (2, 2, 128, 32, 700, 3, 5, 1, W.MEAN_ALL, 100, 0.0173),          # 1 row: padded MFMA tile
    (4, 8, 64, 64, 333, 0, 1, 1, W.MAX_GROUP, 41, 2.0 ** -5),        # 2 rows, d64, Bt64
    (2, 16, 128, 16, 700, 0, 5, 2, W.MEAN_ALL, 100, 0.011),          # 16 rows
    (4, 16, 64, 32, 500, 1, 3, 4, W.MAX_GROUP, 60, 8 / 448),          # 16 rows, d64
    (1, 8, 64, 16, 1500, 2, 7, 2, W.MAX_GROUP, 230, 0.5),             # saturating scale
    (8, 24, 128, 16, 900, 0, 9, 1, W.MEAN_ALL, 150, 8 / 448),         # G = 3
    (6, 30, 64, 32, 500, 1, 3, 3, W.MAX_GROUP, 60, 8 / 448),          # Hkv = 6, 15 rows
]


def fp8_cfg(hkv, hq, d, bt, m, s, rr, nq, mode, extra, scale, planted=3):
    return shape_cfg(hkv, hq, d, bt, "fp8", m, s, rr, nq, mode, extra, planted).replace(
        kv_scale=float(np.float32(scale)))


@pytest.mark.parametrize("shape", FP8_SHAPES, ids=[f"f{i}" for i in range(len(FP8_SHAPES))])
def test_fp8_shapes(shape):
    run_case(fp8_cfg(*shape), 17)


def test_fp8_partial_last_page():
    cfg = fp8_cfg(2, 8, 128, 32, 400, 0, 3, 2, W.MEAN_ALL, 60, 8 / 448)
    run_case(cfg, 5, lpt=7)
    run_case(cfg, 6, lpt=1)


def test_1m_fp8():
    run_case(W.CONFIGS["1m_fp8"], W.CONFIGS["1m_fp8"].seed)


def test_1m_mtp4_fp8_layer0():
    run_case(W.CONFIGS["1m_mtp4_fp8"], W.CONFIGS["1m_mtp4_fp8"].seed, layer=0)


@pytest.mark.parametrize("bt,lpt", [(16, 16), (32, 5), (64, 33)])
def test_fp8_random_views_32_rows(bt, lpt):
    cfg = fp8_cfg(2, 16, 128, bt, 300, 0, 2, 4, W.MAX_GROUP, 10, 0.0173)
    log(f"[case] fp8, 32 rows per KV head, Bt={bt}, last page {lpt}")
    w = W.generate(cfg, 21)
    rng = np.random.default_rng(5)
    vp = np.stack([rng.choice(cfg.n_blocks, 97, replace=False) for _ in range(2)]).astype(np.int32)
    q = np.ascontiguousarray(w.q[0, 0])
    o_ref, l_ref = oracle.view_attention(q, oracle_pool(cfg, w.k_pool[0]), oracle_pool(cfg, w.v_pool[0]), vp,
                                         last_page_tokens=lpt)
    st = LayerState(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page)
    out, lse = st.attend(torch.from_numpy(q).cuda(), torch.from_numpy(vp).cuda(), last_page_tokens=lpt)
    torch.cuda.synchronize()
    err = check_attention(out.cpu().numpy(), lse.cpu().numpy(), o_ref, l_ref, "fp8")
    log(f"  max abs err out {err[0]:.2e} lse {err[1]:.2e}")


def test_fp8_every_code():
    """Pools drawn uniformly over all 254 finite codes (subnormals, -0, +-448
    included): the index is bitwise and attention within tolerance; a NaN code
    makes its block's index row NaN."""
    cfg = fp8_cfg(2, 8, 128, 16, 300, 0, 2, 1, W.MEAN_ALL, 40, 0.0173, planted=0)
    log("[case] fp8 pools over every finite code")
    w = W.generate(cfg, 23)
    rng = np.random.default_rng(9)
    finite = np.setdiff1d(np.arange(256), [0x7F, 0xFF]).astype(np.uint8)
    kp = rng.choice(finite, w.k_pool[0].shape)
    vp_pool = rng.choice(finite, w.v_pool[0].shape)
    kp_o, vp_o = oracle_pool(cfg, kp), oracle_pool(cfg, vp_pool)
    st = LayerState(cfg, kp, vp_pool, w.block_to_page)
    st.build_index()
    torch.cuda.synchronize()
    assert_index_bitwise(st.index_rows(), oracle.mean_k(kp_o, w.block_to_page))
    # small queries keep the softmax spread over many tokens of these wide-range keys
    q = np.ascontiguousarray(w.q[0, 0] * np.float32(0.01))
    views = np.arange(40, dtype=np.int32)[None]
    o_ref, l_ref = oracle.view_attention(q, kp_o, vp_o, views, last_page_tokens=9)
    out, lse = st.attend(torch.from_numpy(q).cuda(), torch.from_numpy(views).cuda(), last_page_tokens=9)
    torch.cuda.synchronize()
    # values reach 448 * 0.0173 = 7.75: the bound scales with the largest |V|
    err = float(np.abs(out.cpu().numpy().astype(np.float64) - o_ref).max())
    lerr = float(np.abs(lse.cpu().numpy().astype(np.float64) - l_ref).max())
    log(f"  max abs err out {err:.2e} lse {lerr:.2e}")
    assert err <= 2e-2 and lerr <= 2e-2
    kp2 = kp.copy()
    kp2[w.block_to_page[5], 1, 3, 17] = 0x7F
    st2 = LayerState(cfg, kp2, None, w.block_to_page)
    st2.build_index()
    torch.cuda.synchronize()
    idx = st2.index_rows()
    assert np.isnan(idx[5, 1, 17]) and np.isfinite(np.delete(idx[5, 1], 17)).all()
    ok = np.ones(cfg.n_blocks, bool)
    ok[5] = False
    assert_index_bitwise(idx[ok], oracle.mean_k(kp_o, w.block_to_page)[ok])


def test_fp8_out_of_range_pages_give_nan():
    cfg = fp8_cfg(2, 16, 128, 16, 200, 0, 2, 2, W.MAX_GROUP, 20, 0.0173)
    log("[case] fp8 out-of-range page ids")
    w = W.generate(cfg, 13)
    st = LayerState(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page)
    q = np.ascontiguousarray(w.q[0, 0])
    vp = np.stack([np.arange(30), np.arange(30, 60)]).astype(np.int32)
    vp[1, 17] = cfg.n_blocks + 1000
    out, _ = st.attend(torch.from_numpy(q).cuda(), torch.from_numpy(vp).cuda())
    torch.cuda.synchronize()
    o = out.cpu().numpy()
    assert np.isnan(o[:, 8:]).all() and np.isfinite(o[:, :8]).all()
    o_ref, _ = oracle.view_attention(q[:, :8], oracle_pool(cfg, w.k_pool[0])[:, :1],
                                     oracle_pool(cfg, w.v_pool[0])[:, :1], vp[:1])
    np.testing.assert_allclose(o[:, :8], o_ref, atol=2e-2, rtol=0)


# ---- Many query rows per KV head (a prefill replayed over the view): K/V tiles
# shared through LDS by 64-row groups ------------------------------------------
MANY_ROWS = [
    # Hkv, Hq, d, Bt, dtype, n_q, pages in view, last page tokens, n_sel
    (2, 8, 128, 16, "bf16", 128, 70, 16, 1),   # 512 rows
    (2, 8, 128, 32, "bf16", 20, 41, 7, 2),     # 80 rows: a ragged second row group
    (4, 16, 64, 64, "bf16", 12, 23, 33, 4),    # 48 rows, d64
    (2, 8, 128, 16, "fp8", 32, 90, 5, 1),      # 128 rows, FP8
    (1, 4, 64, 32, "fp8", 16, 17, 32, 1),      # 64 rows, FP8 d64
    (2, 8, 64, 32, "fp8", 50, 33, 9, 2),       # 200 rows: 256-row groups, ragged, per-head views
]


@pytest.mark.parametrize("case", MANY_ROWS, ids=[f"m{i}" for i in range(len(MANY_ROWS))])
def test_many_rows_attention(case):
    hkv, hq, d, bt, dt, nq, nv, lpt, n_sel = case
    cfg = W.small_config(n_kv_heads=hkv, n_q_heads=hq, head_dim=d, block_tokens=bt, kv_dtype=dt,
                         kv_scale=float(np.float32(8 / 448)), history_tokens=200 * bt, recent_tokens=2 * bt,
                         budget_tokens=(nv + 2) * bt, n_q=nq, mode=W.MEAN_ALL if n_sel == 1 else W.MAX_GROUP)
    log(f"[case] many rows: Hkv={hkv} Hq={hq} d={d} Bt={bt} {dt} n_q={nq} rows/head={nq * hq // hkv} "
        f"view={nv} last={lpt} n_sel={n_sel}")
    w = W.generate(cfg, 51)
    rng = np.random.default_rng(6)
    vp = np.stack([rng.choice(cfg.n_blocks, nv, replace=False) for _ in range(n_sel)]).astype(np.int32)
    q = np.ascontiguousarray(w.q[0, 0])
    o_ref, l_ref = oracle.view_attention(q, oracle_pool(cfg, w.k_pool[0]), oracle_pool(cfg, w.v_pool[0]), vp,
                                         last_page_tokens=lpt)
    st = LayerState(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page, n_q=nq)
    out, lse = st.attend(torch.from_numpy(q).cuda(), torch.from_numpy(vp).cuda(), last_page_tokens=lpt)
    torch.cuda.synchronize()
    err = check_attention(out.cpu().numpy(), lse.cpu().numpy(), o_ref, l_ref, dt)
    log(f"  max abs err out {err[0]:.2e} lse {err[1]:.2e}")
    # an invalid page in one head's view: that head's rows become NaN, the others do not change
    if n_sel > 1:
        vp2 = vp.copy()
        vp2[1, nv // 2] = cfg.n_blocks + 7
        out2, _ = st.attend(torch.from_numpy(q).cuda(), torch.from_numpy(vp2).cuda(), last_page_tokens=lpt)
        torch.cuda.synchronize()
        o2 = out2.cpu().numpy()
        g_size = hq // hkv
        assert np.isnan(o2[:, g_size:2 * g_size]).all()
        keep = np.ones(hq, bool)
        keep[g_size:2 * g_size] = False
        np.testing.assert_array_equal(o2[:, keep], out.cpu().numpy()[:, keep])


# ---- More than 65,536 candidates (histories beyond 1M tokens in 16-token
# blocks; the Table 4 scalability range) -------------------------------------
def test_4m_history_select():
    cfg = W.small_config(n_kv_heads=8, n_q_heads=32, head_dim=128, block_tokens=32, kv_dtype="bf16",
                         history_tokens=4 * 1048576, recent_tokens=8192, budget_tokens=65536, n_q=1,
                         n_planted=128)
    log(f"[case] 4M-token history: {cfg.n_blocks} blocks, {cfg.n_candidates} candidates")
    w = W.generate(cfg, 61, with_values=False)
    index_ref = oracle.mean_k(w.k_pool[0], w.block_to_page)
    rel = oracle.block_relevance(w.q[0, :1], index_ref[None], 0, cfg.n_recent)
    k_eff = oracle.k_eff(cfg.budget_tokens, cfg.budget_tokens, 32, cfg.n_blocks, 0, cfg.n_recent)
    vb_ref, _ = oracle.select(rel, 0, cfg.n_recent, k_eff, w.block_to_page)
    st = LayerState(cfg, w.k_pool[0], None, w.block_to_page)
    st.build_index()
    torch.cuda.synchronize()
    assert_index_bitwise(st.index_rows(), index_ref)
    st.select(torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda())
    torch.cuda.synchronize()
    stats = check_selection(st.view_blocks.cpu().numpy(), st.view_pages.cpu().numpy(), rel, w.block_to_page, 0,
                            cfg.n_recent, k_eff, ref_view=vb_ref)
    worst = check_scores(st.scores.cpu().numpy(), rel, 0, cfg.n_recent)
    log(f"  selection ok: {stats}, worst score rel err {worst:.2e}")


@pytest.mark.parametrize("mode", [W.MEAN_ALL, W.MAX_GROUP])
def test_max_rows_per_head(mode):
    """The most query rows per KV head the boundary takes: 4,096 (G = 8 and
    512 query tokens), through scoring in 16-row chunks, the row-partitioned
    relevance sum and the many-row attention, end to end."""
    run_case(shape_cfg(2, 16, 64, 16, "bf16", 240, 1, 4, 512, mode, 60), 71)


def test_max_candidates_select():
    """The largest selection row the boundary takes: 2^20 candidates (1,024
    selection chunks; a 16M-token history in 16-token blocks), one KV head
    with d = 64 so that the K pool stays at 2 GiB. Index bitwise, selection
    and scores against the oracle."""
    m = (1 << 20) + 8
    cfg = shape_cfg(1, 4, 64, 16, "bf16", m, 0, 8, 1, W.MEAN_ALL, 1 << 19, planted=64)
    assert cfg.n_candidates == 1 << 20
    log(f"[case] {cfg.n_candidates} candidates (the maximum), k = 2^19")
    w = W.generate(cfg, 67, with_values=False)
    index_ref = oracle.mean_k(w.k_pool[0], w.block_to_page)
    rel = oracle.block_relevance(w.q[0, :1], index_ref[None], 0, cfg.n_recent)
    k_eff = oracle.k_eff(cfg.budget_tokens, cfg.budget_tokens, 16, cfg.n_blocks, 0, cfg.n_recent)
    vb_ref, _ = oracle.select(rel, 0, cfg.n_recent, k_eff, w.block_to_page)
    st = LayerState(cfg, w.k_pool[0], None, w.block_to_page)
    st.build_index()
    torch.cuda.synchronize()
    assert_index_bitwise(st.index_rows(), index_ref)
    st.select(torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda())
    torch.cuda.synchronize()
    stats = check_selection(st.view_blocks.cpu().numpy(), st.view_pages.cpu().numpy(), rel, w.block_to_page, 0,
                            cfg.n_recent, k_eff, ref_view=vb_ref)
    worst = check_scores(st.scores.cpu().numpy(), rel, 0, cfg.n_recent)
    log(f"  selection ok: {stats}, worst score rel err {worst:.2e}")


@pytest.mark.parametrize("k", [40000, 69990])
def test_all_equal_scores_beyond_2_16(k):
    """70,000 candidates with identical scores: the selection is the k lowest ids,
    including ids above 2^16."""
    m = 70000 + 5
    cfg = shape_cfg(1, 4, 64, 16, "bf16", m, 0, 5, 1, W.MEAN_ALL, k, planted=0)
    log(f"[case] all scores equal, {cfg.n_candidates} candidates, k={k}")
    w = W.generate(cfg, 62, with_values=False)
    kp = np.broadcast_to(w.k_pool[0][:1], w.k_pool[0].shape).copy()
    st = LayerState(cfg, kp, None, w.block_to_page)
    st.build_index()
    st.select(torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda())
    torch.cuda.synchronize()
    vb = st.view_blocks.cpu().numpy()[0]
    assert vb.tolist() == list(range(k)) + list(range(m - 5, m))


# ---- Rows of 63 to 16,385 candidates with ties (up to 17 selection chunks) ----
@pytest.mark.parametrize("n_cand,k", [(16384, 1), (16384, 9000), (16384, 16384), (16385, 9000), (1000, 999),
                                      (63, 10)])
def test_all_equal_scores_small_rows(n_cand, k):
    """Identical scores, from one partial chunk to 16 full chunks and one more
    candidate, k from 1 to every candidate: the selection is the k lowest ids,
    in order, after the sinks and before the recent window."""
    m = n_cand + 3 + 5
    cfg = shape_cfg(1, 4, 64, 16, "bf16", m, 3, 5, 1, W.MEAN_ALL, k, planted=0)
    log(f"[case] all scores equal, {cfg.n_candidates} candidates, k={k}")
    w = W.generate(cfg, 65, with_values=False)
    kp = np.broadcast_to(w.k_pool[0][:1], w.k_pool[0].shape).copy()
    st = LayerState(cfg, kp, None, w.block_to_page)
    st.build_index()
    st.select(torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda())
    torch.cuda.synchronize()
    vb = st.view_blocks.cpu().numpy()[0]
    assert vb.tolist() == list(range(3 + k)) + list(range(m - 5, m))
    np.testing.assert_array_equal(st.view_pages.cpu().numpy()[0], w.block_to_page[vb])


@pytest.mark.parametrize("n_cand,mode", [(16384, W.MEAN_ALL), (12000, W.MAX_GROUP), (16385, W.MEAN_ALL)])
def test_exact_ties_small_rows(n_cand, mode):
    """Pages copied from 40 sources: ~400 exact ties per score, and the budget
    ends inside a tie group, with 4 query rows per KV head."""
    m, extra = n_cand + 2 + 4, n_cand // 3 + 7
    cfg = shape_cfg(2, 8, 128, 16, "bf16", m, 2, 4, 1, mode, extra, planted=0)
    log(f"[case] exact ties, {cfg.n_candidates} candidates, mode {mode}")
    w = W.generate(cfg, 66, with_values=False)
    kp = w.k_pool[0]
    kp[:] = kp[np.random.default_rng(2).integers(0, 40, cfg.n_blocks)]
    index_ref = oracle.mean_k(kp, w.block_to_page)
    rel = oracle.block_relevance(w.q[0, :1], index_ref[None], 2, cfg.n_recent, oracle_mode(cfg))
    k_eff = oracle.k_eff(cfg.budget_tokens, cfg.budget_tokens, 16, cfg.n_blocks, 2, cfg.n_recent)
    vb_ref, _ = oracle.select(rel, 2, cfg.n_recent, k_eff, w.block_to_page)
    st = LayerState(cfg, kp, None, w.block_to_page)
    st.build_index()
    st.select(torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(st.view_blocks.cpu().numpy(), vb_ref)


# ---- Exact ties at the threshold in rows beyond 2^17 candidates ------------
def test_exact_ties_140k_candidates():
    """140,000 candidates whose pages copy one of 100 source pages: ~1,400
    exact ties per score (ranked by the radix select in LDS), the budget ends
    inside them."""
    m, n_src, extra = 140000 + 4, 100, 60000
    cfg = shape_cfg(1, 4, 64, 16, "bf16", m, 0, 4, 1, W.MEAN_ALL, extra, planted=0)
    log(f"[case] exact ties, {cfg.n_candidates} candidates")
    w = W.generate(cfg, 63, with_values=False)
    kp = w.k_pool[0]
    kp[:] = kp[np.random.default_rng(1).integers(0, n_src, cfg.n_blocks)]
    index_ref = oracle.mean_k(kp, w.block_to_page)
    rel = oracle.block_relevance(w.q[0, :1], index_ref[None], 0, cfg.n_recent)
    k_eff = oracle.k_eff(cfg.budget_tokens, cfg.budget_tokens, 16, cfg.n_blocks, 0, cfg.n_recent)
    vb_ref, _ = oracle.select(rel, 0, cfg.n_recent, k_eff, w.block_to_page)
    st = LayerState(cfg, kp, None, w.block_to_page)
    st.build_index()
    st.select(torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda())
    torch.cuda.synchronize()
    np.testing.assert_array_equal(st.view_blocks.cpu().numpy(), vb_ref)
    np.testing.assert_array_equal(st.view_pages.cpu().numpy()[0], w.block_to_page[vb_ref[0]])


@pytest.mark.parametrize("m,k", [(131072, 90000), (150000, 100000)])
def test_all_equal_scores_150k(m, k):
    """Up to 150,000 candidates with identical scores (the pivot bin far beyond
    the LDS window): the selection is the k lowest ids."""
    cfg = shape_cfg(1, 4, 64, 16, "bf16", m + 5, 0, 5, 1, W.MEAN_ALL, k, planted=0)
    log(f"[case] all scores equal, {cfg.n_candidates} candidates, k={k}")
    w = W.generate(cfg, 64, with_values=False)
    kp = np.broadcast_to(w.k_pool[0][:1], w.k_pool[0].shape).copy()
    st = LayerState(cfg, kp, None, w.block_to_page)
    st.build_index()
    st.select(torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda())
    torch.cuda.synchronize()
    vb = st.view_blocks.cpu().numpy()[0]
    assert vb.tolist() == list(range(k)) + list(range(m, m + 5))


@pytest.mark.parametrize("copies", [500, 586])
def test_over_a_thousand_splits(copies):
    """A view of 512 distinct pages, each listed `copies` times, gives the same
    output as the distinct pages alone and a log-sum-exp larger by ln(copies)
    (every token's weight appears `copies` times in both sums of the softmax).
    500 and 586 copies make 1,000 and 1,172 splits of 256 pages, so the merge
    walks far more splits than it preloads."""
    cfg = shape_cfg(1, 4, 64, 16, "bf16", 512, 0, 2, 1, W.MAX_GROUP, 10)
    log(f"[case] 512 pages x {copies} copies, 1 KV head, 4 rows")
    w = W.generate(cfg, 29)
    distinct = np.random.default_rng(7).permutation(cfg.n_blocks).astype(np.int32)[None]
    o_ref, l_ref = oracle.view_attention(w.q[0, 0], w.k_pool[0], w.v_pool[0], distinct)
    vp = torch.from_numpy(np.tile(distinct, (1, copies))).cuda()
    st = LayerState(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page)
    qd = torch.from_numpy(np.ascontiguousarray(w.q[0, 0])).cuda()
    out, lse = st.attend(qd, vp)
    torch.cuda.synchronize()
    o1, l1 = out.cpu().numpy().copy(), lse.cpu().numpy().copy()
    check_attention(o1, l1, o_ref, l_ref + math.log(copies), "bf16")
    # a second call through the same workspace gives the same bits
    out, lse = st.attend(qd, vp)
    torch.cuda.synchronize()
    assert np.array_equal(o1, out.cpu().numpy()) and np.array_equal(l1, lse.cpu().numpy())
