"""GPU parity of the recall point (Sec. 4.2 step-level scheduling, Eq. 10 as
printed): after a step's prefill, all of its query tokens -- through every
layer and query head -- select one working set.  Scores and selection through
the C ABI against the oracle, as in tests/parity.py."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_04852_amd import kvmem as K
from paper_2609_04852_amd import workload as W
from paper_2609_04852_amd.step import RecallState
from parity import assert_index_bitwise, check_scores, check_selection, log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    K.lib()
    yield
    torch.cuda.synchronize()


def run_recall(cfg, seed, check_index=True):
    log(f"[case] recall {cfg.name} seed={seed} L={cfg.n_layers} M={cfg.n_blocks} n_q={cfg.n_q} "
        f"Hkv={cfg.n_kv_heads} Hq={cfg.n_q_heads} d={cfg.head_dim} Bt={cfg.block_tokens} mode={cfg.mode}")
    w = W.generate(cfg, seed, with_values=False)
    b2p = w.block_to_page
    S, Rr = cfg.sink_blocks, cfg.n_recent
    index_ref = np.stack([oracle.mean_k(oracle_pool(cfg, k), b2p) for k in w.k_pool])
    mode = oracle.MEAN_ALL if cfg.mode == W.MEAN_ALL else oracle.MAX_GROUP
    rel = oracle.block_relevance(w.q[0], index_ref, S, Rr, mode)
    k_eff = oracle.k_eff(cfg.budget_tokens, cfg.budget_tokens, cfg.block_tokens, cfg.n_blocks, S, Rr)
    vb_ref, _ = oracle.select(rel, S, Rr, k_eff, b2p)
    log("  gpu: index + select")
    st = RecallState(cfg, w.k_pool, b2p)
    st.build_index()
    torch.cuda.synchronize()
    if check_index:
        for l in range(cfg.n_layers):
            assert_index_bitwise(st.index_rows(l), index_ref[l])
    n_view = st.select(torch.from_numpy(np.ascontiguousarray(w.q[0])).cuda())
    torch.cuda.synchronize()
    assert n_view == S + k_eff + Rr
    vb, vpg = st.view_blocks.cpu().numpy(), st.view_pages.cpu().numpy()
    stats = check_selection(vb, vpg, rel, b2p, S, Rr, k_eff, ref_view=vb_ref)
    worst = check_scores(st.scores.cpu().numpy(), rel, S, Rr)
    log(f"  selection ok: {stats}, worst score rel err {worst:.2e}")
    return st, w


def oracle_pool(cfg, pool):
    return oracle.decode_fp8(pool, cfg.kv_scale) if cfg.kv_dtype == "fp8" else pool


RECALL_SHAPES = [
    # L, Hkv, Hq, d, Bt, M, S, Rr, n_q, mode, extra blocks
    (2, 2, 8, 128, 32, 700, 0, 8, 32, W.MEAN_ALL, 90),    # 128 rows per KV head and layer
    (3, 1, 4, 64, 16, 1500, 2, 16, 16, W.MEAN_ALL, 200),  # 64 rows, d64, a ragged last tile
    (1, 4, 16, 128, 64, 333, 0, 2, 8, W.MAX_GROUP, 40),    # 32 rows, one selection per KV head
    (2, 8, 32, 128, 16, 2100, 1, 40, 128, W.MEAN_ALL, 300),  # 512 rows: row partitions of the sum
    (1, 2, 8, 64, 16, 400, 0, 4, 256, W.MAX_GROUP, 50),      # 1,024 rows per selection: partitions of the max
]


@pytest.mark.parametrize("shape", RECALL_SHAPES, ids=[f"r{i}" for i in range(len(RECALL_SHAPES))])
def test_recall_shapes(shape):
    L, hkv, hq, d, bt, m, s, rr, nq, mode, extra = shape
    cfg = W.small_config(n_layers=L, n_kv_heads=hkv, n_q_heads=hq, head_dim=d, block_tokens=bt, kv_dtype="bf16",
                         history_tokens=m * bt, recent_tokens=rr * bt, sink_blocks=s,
                         budget_tokens=(s + rr + extra) * bt, n_q=nq, mode=mode, n_planted=3)
    run_recall(cfg, 31)


def test_recall_fp8():
    cfg = W.small_config(n_layers=2, n_kv_heads=4, n_q_heads=16, head_dim=128, block_tokens=32, kv_dtype="fp8",
                         kv_scale=float(np.float32(8 / 448)), history_tokens=900 * 32, recent_tokens=8 * 32,
                         budget_tokens=120 * 32, n_q=64, n_planted=3)
    run_recall(cfg, 32)


def test_recall_1m():
    run_recall(W.CONFIGS["1m_recall"], W.CONFIGS["1m_recall"].seed)
