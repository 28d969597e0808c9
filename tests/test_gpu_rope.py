"""GPU parity of the position handling (Sec. 4.3 index construction, Sec. 4.4
execution view, Sec. 5.3 copy-free assembly): the Mean-K index from RoPE-encoded
keys, materialisation of selected blocks at compact positions, and in-place
delta re-encoding, each through the C ABI against the oracle on the same inputs.

Every input that carries an encoding is made by the oracle (never by the HIP
path).  Tolerances: the index within 2e-6 (fp32 rotation against the fp64
definition, about one fp32 ulp of the mean); re-encoded bf16 keys within one
bf16 ulp of the rounded fp64 value; copied V bitwise; attention as in
tests/parity.py.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_04852_amd import kvmem as K
from paper_2609_04852_amd import workload as W
from paper_2609_04852_amd.step import LayerState, geom_of, pool_to_device
from parity import check_attention, log

pytestmark = pytest.mark.gpu

BASE = 1e6  # Qwen3's RoPE base


def encode_pool(raw, block_to_page, positions_of_block, base, bf16):
    """Oracle encoding of a raw pool: the page of block b holds its tokens at
    positions_of_block[b] + t.  Returns the stored pool (bf16 bits or fp32)."""
    n_pages, hkv, bt, d = raw.shape
    x = oracle.from_bf16_bits(raw).astype(np.float64) if raw.dtype == np.uint16 else raw.astype(np.float64)
    pos = np.zeros((n_pages, hkv, bt), np.int64)
    pos[block_to_page] = positions_of_block[:, None, None] + np.arange(bt)[None, None, :]
    enc = oracle.rope(x, pos, base)
    return oracle.to_bf16_bits(enc) if bf16 else enc.astype(np.float32)


def pair_norm(x):
    """|(x_j, x_{j+d/2})| for every element: the scale of a rotation's fp32 error."""
    h = x.shape[-1] // 2
    n = np.hypot(x[..., :h], x[..., h:])
    return np.concatenate([n, n], axis=-1)


def bf16_close(gpu_bits, ref64):
    """|gpu - ref| within one bf16 ulp of ref, plus the fp32 rotation error
    (a few fp32 ulps of the pair's norm)."""
    g = oracle.from_bf16_bits(gpu_bits).astype(np.float64)
    tol = np.abs(ref64) * 2.0 ** -7 + pair_norm(ref64) * 2.0 ** -20
    bad = np.abs(g - ref64) > tol
    assert not bad.any(), f"{bad.sum()} of {bad.size} elements beyond one bf16 ulp"
    # fraction of elements whose bits differ from the oracle's own bf16 rounding
    return float((np.asarray(gpu_bits, np.uint16) != oracle.to_bf16_bits(ref64)).mean())


# Workloads of the index-from-encoded-keys cases beyond the named ones: 64-token
# blocks (the 4-layer workload's geometry) and fp32 keys at d = 128.
ROPE_CFGS = {
    "bt64": W.CONFIGS["64k"].replace(block_tokens=64, history_tokens=1024 * 64),
    "f32_d128": W.small_config(n_kv_heads=4, n_q_heads=16, head_dim=128, block_tokens=32, kv_dtype="f32",
                               history_tokens=600 * 32, recent_tokens=4 * 32, budget_tokens=64 * 32),
}


@pytest.mark.parametrize("name,baked", [("tiny", "orig"), ("64k", "orig"), ("64k", "random"), ("64k", "huge"),
                                        ("bt64", "orig"), ("bt64", "random"), ("f32_d128", "orig"),
                                        ("f32_d128", "random")])
def test_index_from_encoded_keys(name, baked):
    cfg = ROPE_CFGS[name] if name in ROPE_CFGS else W.CONFIGS[name]
    log(f"[case] index from encoded keys {name} positions={baked}")
    w = W.generate(cfg, cfg.seed, with_values=False)
    m = cfg.n_blocks
    if baked == "orig":
        p0, bp = np.arange(m, dtype=np.int64) * cfg.block_tokens, None
    elif baked == "random":  # baked positions far beyond the window, e.g. after many delta moves
        p0 = np.random.default_rng(7).integers(0, 2 ** 40, m).astype(np.int64)
        bp = p0
    else:  # positions from 2^41 to 2^50 (both sides of the switch to per-token cos/sin at 2^42)
        p0 = np.random.default_rng(7).integers(2 ** 41, 2 ** 50, m).astype(np.int64)
        p0[::7] = 2 ** 42 - cfg.block_tokens - np.arange(p0[::7].size) % 3  # ends just below the switch
        bp = p0
    enc = encode_pool(w.k_pool[0], w.block_to_page, p0, BASE, cfg.kv_dtype == "bf16")
    ref = oracle.mean_k_rope(enc, w.block_to_page, BASE, block_pos=bp)
    st = LayerState(cfg, enc, None, w.block_to_page)
    K.kvmem_build_index_rope(st.geom, st.k_pool, st.block_to_page, 0, m, st.index, BASE,
                             None if bp is None else torch.from_numpy(bp).cuda())
    torch.cuda.synchronize()
    got = st.index_rows()
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    log(f"  max abs err {err.max():.2e}, exact {np.mean(err == 0):.3f}")
    np.testing.assert_allclose(got, ref, atol=2e-6, rtol=2e-6)
    # the encoding really was removed: the plain Mean-K of the encoded keys is far off
    plain = oracle.mean_k(enc, w.block_to_page)
    assert np.abs(plain - ref).max() > 1e-2


@pytest.mark.parametrize("d,bt,explicit", [(128, 16, True), (64, 32, True), (128, 16, False), (64, 64, False),
                                            (128, 64, True)])
def test_index_from_encoded_fp8_keys(d, bt, explicit):
    """FP8 pools whose codes hold RoPE-encoded keys (encoded by the oracle in
    fp64, then quantised like every FP8 pool), at explicit positions (the kernel
    with the rounding correction) or at the original frame b * Bt below 2^26
    (block_pos NULL: the kernel without it)."""
    cfg = W.CONFIGS["64k"].replace(kv_dtype="fp8", kv_scale=float(np.float32(8 / 448)), head_dim=d,
                                   block_tokens=bt, history_tokens=2048 * bt, n_kv_heads=4, n_q_heads=16)
    log(f"[case] index from encoded FP8 keys d={d} Bt={bt} explicit positions={explicit}")
    w = W.generate(cfg, 5, with_values=False)
    m = cfg.n_blocks
    if explicit:
        p0 = np.random.default_rng(8).integers(0, 2 ** 30, m).astype(np.int64)
    else:
        p0 = np.arange(m, dtype=np.int64) * bt
    raw = oracle.decode_fp8(w.k_pool[0], cfg.kv_scale)
    pos = np.zeros(raw.shape[:3], np.int64)
    pos[w.block_to_page] = p0[:, None, None] + np.arange(bt)[None, None, :]
    codes = W.fp8_codes(oracle.rope(raw, pos, BASE).astype(np.float32), cfg.kv_scale)
    ref = oracle.mean_k_rope(oracle.decode_fp8(codes, cfg.kv_scale), w.block_to_page, BASE,
                             block_pos=p0 if explicit else None)
    st = LayerState(cfg, codes, None, w.block_to_page)
    K.kvmem_build_index_rope(st.geom, st.k_pool, st.block_to_page, 0, m, st.index, BASE,
                             torch.from_numpy(p0).cuda() if explicit else None)
    torch.cuda.synchronize()
    got = st.index_rows()
    err = np.abs(got.astype(np.float64) - ref.astype(np.float64))
    log(f"  max abs err {err.max():.2e}, exact {np.mean(err == 0):.3f}")
    np.testing.assert_allclose(got, ref, atol=2e-6, rtol=2e-6)


@pytest.mark.parametrize("dt,d,bt", [("bf16", 128, 16), ("bf16", 64, 64), ("f32", 128, 32)])
def test_materialize(dt, d, bt):
    cfg = W.small_config(n_kv_heads=4, n_q_heads=16, head_dim=d, block_tokens=bt, kv_dtype=dt,
                         history_tokens=300 * bt, recent_tokens=4 * bt, budget_tokens=64 * bt)
    log(f"[case] materialize {dt} d={d} Bt={bt}")
    w = W.generate(cfg, 3)
    r = np.random.default_rng(11)
    n_blocks, n_dst = 57, 80
    src = r.choice(cfg.n_blocks, n_blocks, replace=False).astype(np.int32)
    dst = r.choice(n_dst, n_blocks, replace=False).astype(np.int32)
    pos = (np.arange(n_blocks, dtype=np.int64) * bt + 12345)  # contiguous compact slots
    k_ref, v_ref = oracle.materialize(w.k_pool[0], w.v_pool[0], src, pos, BASE)
    dev = torch.device("cuda")
    raw = pool_to_device(w.k_pool[0], dev)
    v = pool_to_device(w.v_pool[0], dev)
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    kd = torch.full((n_dst,) + raw.shape[1:], -7.0, dtype=tdt, device=dev)  # sentinel
    vd = torch.full_like(kd, -7.0)
    g = geom_of(cfg)
    K.kvmem_materialize(g, BASE, raw, v, torch.from_numpy(src).cuda(), torch.from_numpy(pos).cuda(),
                        torch.from_numpy(dst).cuda(), kd, vd)
    torch.cuda.synchronize()
    kh, vh = kd.cpu(), vd.cpu()
    if dt == "bf16":
        kb = kh.view(torch.int16).numpy().view(np.uint16)
        frac = bf16_close(kb[dst], k_ref)
        np.testing.assert_array_equal(vh.view(torch.int16).numpy().view(np.uint16)[dst], v_ref)
    else:
        assert (np.abs(kh.numpy()[dst] - k_ref) <= 1e-6 * pair_norm(k_ref)).all()
        np.testing.assert_array_equal(vh.numpy()[dst], v_ref)
        frac = 0.0
    log(f"  K within one bf16 ulp ({frac:.2e} of elements differ from the oracle's rounding), V bitwise")
    untouched = np.setdiff1d(np.arange(n_dst), dst)
    assert (kh[untouched] == -7.0).all() and (vh[untouched] == -7.0).all()


def test_materialize_invalid_pages():
    cfg = W.small_config(n_kv_heads=2, n_q_heads=8, head_dim=128, block_tokens=16, kv_dtype="bf16",
                         history_tokens=40 * 16, recent_tokens=2 * 16, budget_tokens=10 * 16)
    log("[case] materialize with invalid page ids")
    w = W.generate(cfg, 4)
    dev = torch.device("cuda")
    raw = pool_to_device(w.k_pool[0], dev)
    v = pool_to_device(w.v_pool[0], dev)
    kd = torch.zeros((6,) + raw.shape[1:], dtype=torch.bfloat16, device=dev)
    vd = torch.zeros_like(kd)
    src = torch.tensor([3, 10**6, 5, 7], dtype=torch.int32, device=dev)   # second source is not in the pool
    dst = torch.tensor([0, 1, 10**6, 4], dtype=torch.int32, device=dev)   # third destination is not in the pool
    pos = torch.tensor([0, 16, 32, 48], dtype=torch.int64, device=dev)
    K.kvmem_materialize(geom_of(cfg), BASE, raw, v, src, pos, dst, kd, vd)
    torch.cuda.synchronize()
    assert torch.isnan(kd[1].float()).all() and torch.isnan(vd[1].float()).all()
    assert (kd[[2, 3, 5]] == 0).all() and (vd[[2, 3, 5]] == 0).all()  # nothing written there
    k_ref, v_ref = oracle.materialize(w.k_pool[0], w.v_pool[0], np.array([3, 7]), np.array([0, 48]), BASE)
    bf16_close(kd[[0, 4]].cpu().view(torch.int16).numpy().view(np.uint16), k_ref)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_rerope_delta(dt):
    cfg = W.small_config(n_kv_heads=4, n_q_heads=16, head_dim=128, block_tokens=32, kv_dtype=dt,
                         history_tokens=100 * 32, recent_tokens=2 * 32, budget_tokens=20 * 32)
    log(f"[case] delta re-encoding {dt}")
    w = W.generate(cfg, 5, with_values=False)
    r = np.random.default_rng(2)
    n_pages = cfg.n_blocks
    baked = r.integers(0, 10**6, n_pages).astype(np.int64)
    enc = encode_pool(w.k_pool[0], np.arange(n_pages, dtype=np.int32), baked, BASE, dt == "bf16")
    pages = r.choice(n_pages, 37, replace=False).astype(np.int32)
    delta = r.integers(-50000, 50000, 37).astype(np.int64)
    x = oracle.from_bf16_bits(enc).astype(np.float64) if dt == "bf16" else enc.astype(np.float64)
    ref = oracle.rope(x[pages], np.broadcast_to(delta[:, None, None], x[pages].shape[:-1]), BASE)
    kp = pool_to_device(enc, torch.device("cuda"))
    K.kvmem_rerope(geom_of(cfg), BASE, kp, torch.from_numpy(pages).cuda(), torch.from_numpy(delta).cuda())
    torch.cuda.synchronize()
    kh = kp.cpu()
    if dt == "bf16":
        bits = kh.view(torch.int16).numpy().view(np.uint16)
        bf16_close(bits[pages], ref)
        others = np.setdiff1d(np.arange(n_pages), pages)
        np.testing.assert_array_equal(bits[others], enc[others])
    else:
        assert (np.abs(kh.numpy()[pages] - ref) <= 1e-6 * pair_norm(ref)).all()
    # moving a block there and back stays within two bf16 ulps of where it started (bounded drift)
    K.kvmem_rerope(geom_of(cfg), BASE, kp, torch.from_numpy(pages).cuda(), torch.from_numpy(-delta).cuda())
    torch.cuda.synchronize()
    back = kp.cpu()
    start = x[pages]
    now = (oracle.from_bf16_bits(back.view(torch.int16).numpy().view(np.uint16)[pages]).astype(np.float64)
           if dt == "bf16" else back.numpy()[pages].astype(np.float64))
    tol = (2.0 ** -6 if dt == "bf16" else 4e-6) * pair_norm(start)
    assert (np.abs(now - start) <= tol).all()


def test_position_consistent_view_end_to_end():
    """Index from encoded keys -> selection with position-independent queries ->
    materialisation of the view at compact positions -> attention with the query
    encoded at its own position: equals the oracle's run of the same steps."""
    cfg = W.CONFIGS["64k"]
    log("[case] position-consistent view, 64k")
    w = W.generate(cfg, cfg.seed)
    m, bt = cfg.n_blocks, cfg.block_tokens
    p0 = np.arange(m, dtype=np.int64) * bt
    enc = encode_pool(w.k_pool[0], w.block_to_page, p0, BASE, True)  # stored keys carry RoPE
    q = w.q[0, 0:1]  # [1][n_q][Hq][d], position independent (the model's pre-RoPE projection)
    # ---- oracle
    index_ref = oracle.mean_k_rope(enc, w.block_to_page, BASE)
    rel = oracle.block_relevance(q, index_ref[None], cfg.sink_blocks, cfg.n_recent)
    k_eff = oracle.k_eff(cfg.budget_tokens, cfg.budget_tokens, bt, m, cfg.sink_blocks, cfg.n_recent)
    vb_ref, _ = oracle.select(rel, cfg.sink_blocks, cfg.n_recent, k_eff, w.block_to_page)
    n_view = vb_ref.shape[1]
    # the view's blocks, in order, take compact slots 0 .. n_view-1 of the execution pool
    src = w.block_to_page[vb_ref[0]].astype(np.int32)
    dst = np.arange(n_view, dtype=np.int32)
    cpos = dst.astype(np.int64) * bt
    k_exec, v_exec = oracle.materialize(w.k_pool[0], w.v_pool[0], src, cpos, BASE)
    k_exec_bits = oracle.to_bf16_bits(k_exec)
    q_pos = n_view * bt  # the query follows the view
    q_enc = oracle.rope(q[0], q_pos, BASE).astype(np.float32)
    out_ref, lse_ref = oracle.view_attention(q_enc, k_exec_bits, v_exec, dst[None], last_page_tokens=bt)
    # ---- GPU (raw K is the materialisation source; the stored pool carries RoPE)
    st = LayerState(cfg, enc, w.v_pool[0], w.block_to_page)
    K.kvmem_build_index_rope(st.geom, st.k_pool, st.block_to_page, 0, m, st.index, BASE)
    st.select(torch.from_numpy(np.ascontiguousarray(q)).cuda())
    torch.cuda.synchronize()
    np.testing.assert_allclose(st.index_rows(), index_ref, atol=2e-6, rtol=2e-6)
    vb = st.view_blocks.cpu().numpy()
    assert np.array_equal(vb, vb_ref), "selection differs from the oracle's on this seed"
    dev = torch.device("cuda")
    raw = pool_to_device(w.k_pool[0], dev)
    vpool = pool_to_device(w.v_pool[0], dev)
    kx = torch.empty((n_view,) + raw.shape[1:], dtype=torch.bfloat16, device=dev)
    vx = torch.empty_like(kx)
    src_d = st.view_pages[0].contiguous()  # the GPU's own view tables drive the materialisation
    K.kvmem_materialize(st.geom, BASE, raw, vpool, src_d, torch.from_numpy(cpos).cuda(),
                        torch.from_numpy(dst).cuda(), kx, vx)
    geom = st.geom
    n_sel = 1
    ws = torch.empty(K.kvmem_sparse_attn_workspace_bytes(geom, cfg.n_q, n_sel, n_view), dtype=torch.uint8,
                     device=dev)
    out = torch.empty((cfg.n_q, cfg.n_q_heads, cfg.head_dim), dtype=torch.float32, device=dev)
    lse = torch.empty((cfg.n_q, cfg.n_q_heads), dtype=torch.float32, device=dev)
    K.kvmem_sparse_attn(geom, torch.from_numpy(q_enc).cuda(), kx, vx, torch.from_numpy(dst[None]).cuda(),
                        n_sel, n_view, bt, 0.0, out, ws, lse)
    torch.cuda.synchronize()
    frac = bf16_close(kx.cpu().view(torch.int16).numpy().view(np.uint16), k_exec)
    err = check_attention(out.cpu().numpy(), lse.cpu().numpy(), out_ref, lse_ref, "bf16")
    log(f"  view keys within one bf16 ulp ({frac:.2e} differ from the oracle's rounding); "
        f"attention max abs err {err[0]:.2e}")
