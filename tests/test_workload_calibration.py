"""The 4-layer mixture workload is calibrated to the attention sparsity the paper
reports (Sec. 4.3: the top-8 of ~103 blocks hold 66.5 % of historical attention,
the top-16 77.0 %).  This checks the generator's recipe at full shape (one layer,
keys only); it is a property of the synthetic inputs, not a parity test."""
import numpy as np

import oracle
from paper_2609_04852_amd import workload as W


def test_mixture_workload_sparsity():
    cfg = W.CONFIGS["1m_mtp4"]
    w = W.generate(cfg, cfg.seed, layers=1, with_values=False)
    index = oracle.mean_k(w.k_pool[0], w.block_to_page)
    cand = index[: cfg.n_blocks - cfg.n_recent].astype(np.float64)
    q = w.q[0, 0].astype(np.float64)
    top8, top16 = [], []
    for m in range(cfg.n_q):
        for h in range(cfg.n_q_heads):
            s = cand[:, h // cfg.group, :] @ q[m, h] / np.sqrt(cfg.head_dim)
            p = np.exp(s - s.max())
            p = np.sort(p / p.sum())[::-1]
            top8.append(p[: int(0.078 * p.size)].sum())
            top16.append(p[: int(0.155 * p.size)].sum())
    assert 0.60 <= np.mean(top8) <= 0.75, np.mean(top8)
    assert 0.72 <= np.mean(top16) <= 0.88, np.mean(top16)
