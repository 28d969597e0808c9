"""kvmem_select_noalloc (the selection with the library's own device scratch)
against kvmem_select with a caller workspace, through the C ABI: two calls in a
row on one GPU, the second with a smaller input, each bitwise equal to
kvmem_select on the same inputs (view tables and scores)."""
import numpy as np
import pytest
import torch

from paper_2609_04852_amd import kvmem as K
from paper_2609_04852_amd import workload as W
from paper_2609_04852_amd.step import LayerState

pytestmark = pytest.mark.gpu


def _case(cfg, seed):
    print(f"[case] no-alloc select vs select: {cfg.name} M={cfg.n_blocks} Hkv={cfg.n_kv_heads} "
          f"Hq={cfg.n_q_heads} n_q={cfg.n_q} mode={cfg.mode}", flush=True)
    w = W.generate(cfg, seed, with_values=False)
    st = LayerState(cfg, w.k_pool[0], None, w.block_to_page)
    st.build_index()
    q = torch.from_numpy(np.ascontiguousarray(w.q[0, :1])).cuda()
    return st, q


def _noalloc(st, q):
    vb = torch.full_like(st.view_blocks, -5)
    vp = torch.full_like(st.view_pages, -5)
    sc = torch.full_like(st.scores, -5.0)
    n = K.kvmem_select_noalloc(st.geom, q, st.index, st.n_blocks, st.n_sink, st.n_recent, st.budget, st.budget,
                               st.mode, 0.0, st.block_to_page, vb, vp, sc)
    return n, vb, vp, sc


def test_noalloc_matches_select_twice():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    big = W.CONFIGS["256k"]
    small = W.small_config(n_kv_heads=2, n_q_heads=16, head_dim=128, block_tokens=32, kv_dtype="bf16",
                           history_tokens=900 * 32, recent_tokens=5 * 32, sink_blocks=1,
                           budget_tokens=(1 + 5 + 120) * 32, n_q=2, mode=W.MAX_GROUP, n_planted=3)
    for cfg, seed in ((big, 2), (small, 7)):  # the second call is smaller and leaves stale scratch behind it
        st, q = _case(cfg, seed)
        ws_bytes = K.kvmem_select_workspace_bytes(st.geom, 1, st.n_q, st.n_blocks, st.n_sink, st.n_recent, st.mode)
        assert ws_bytes <= K.SELECT_NOALLOC_MAX_BYTES
        n_ref = st.select(q)
        torch.cuda.synchronize()
        ref = [t.cpu().numpy().copy() for t in (st.view_blocks, st.view_pages, st.scores)]
        n, vb, vp, sc = _noalloc(st, q)
        torch.cuda.synchronize()
        assert n == n_ref
        got = [t.cpu().numpy() for t in (vb, vp, sc)]
        for a, b, name in zip(got, ref, ("view_blocks", "view_pages", "scores")):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"{cfg.name}: {name} differs from kvmem_select"
        print(f"  bitwise equal to kvmem_select (workspace {ws_bytes} bytes)", flush=True)


def test_noalloc_rejects_oversized_selection():
    """A selection whose scratch exceeds the library's array is refused on the host."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = W.CONFIGS["64k"]
    g = K.Geom(cfg.n_kv_heads, cfg.n_q_heads, cfg.head_dim, cfg.block_tokens, K.KVMEM_BF16)
    n_q = 64  # 2,048 logit rows of 4,032 candidates: about 33 MB of workspace
    assert K.kvmem_select_workspace_bytes(g, 1, n_q, cfg.n_blocks, 0, cfg.n_recent, 0) > K.SELECT_NOALLOC_MAX_BYTES
    dev = torch.device("cuda")
    q = torch.zeros((1, n_q, cfg.n_q_heads, cfg.head_dim), dtype=torch.float32, device=dev)
    index = torch.zeros(K.kvmem_index_bytes(g, cfg.n_blocks) // 4, dtype=torch.float32, device=dev)
    b2p = torch.arange(cfg.n_blocks, dtype=torch.int32, device=dev)
    vb = torch.empty((1, cfg.n_view), dtype=torch.int32, device=dev)
    with pytest.raises(K.KvmemError) as e:
        K.kvmem_select_noalloc(g, q, index, cfg.n_blocks, 0, cfg.n_recent, cfg.budget_tokens, cfg.budget_tokens,
                               0, 0.0, b2p, vb, torch.empty_like(vb))
    assert e.value.status == -6 and "kvmem_select with a workspace" in str(e.value)
