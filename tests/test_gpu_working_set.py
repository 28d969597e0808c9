"""GPU parity of the working-set update at a recall point (Sec. 4.4, Eq. 11,
Eq. 12): a sequence of recalls over a bounded execution pool, through the C ABI,
against the oracle's WorkingSet on the same views.

Integer results (page table, counts, every state array) must be bitwise equal.
The execution pool's V pages must equal the history's V bitwise; its K pages
must equal RoPE(raw K, compact position) within one bf16 ulp of the element
plus, per delta re-encoding since the page was built from raw K, one bf16
rounding of the pair's norm (fp32 pools: a few fp32 ulps of the pair's norm
per re-encoding).  Views and positions come from a seeded generator or
from the oracle's own selection, never from the HIP path."""
import numpy as np
import pytest
import torch

import oracle
from oracle.working_set import WorkingSet
from paper_2609_04852_amd import kvmem as K
from paper_2609_04852_amd import workload as W
from paper_2609_04852_amd.step import geom_of, pool_to_device
from parity import log

pytestmark = pytest.mark.gpu

BASE = 1e6


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    K.lib()
    yield
    torch.cuda.synchronize()


def pair_norm(x):
    h = x.shape[-1] // 2
    n = np.hypot(x[..., :h], x[..., h:])
    return np.concatenate([n, n], axis=-1)


def random_views(seed, m, steps, lo, hi):
    r = np.random.default_rng(seed)
    out, prev = [], None
    for _ in range(steps):
        n = int(r.integers(lo, hi + 1))
        if prev is not None and r.random() < 0.7:
            keep = r.choice(prev, size=min(len(prev), (3 * n) // 4), replace=False)
            rest = r.choice(np.setdiff1d(np.arange(m), keep), size=n - len(keep), replace=False)
            v = np.sort(np.concatenate([keep, rest]))
        else:
            v = np.sort(r.choice(m, size=n, replace=False))
        out.append(v.astype(np.int32))
        prev = v
    return out


class Runner:
    """GPU execution pool + state, stepped beside the oracle's WorkingSet."""

    def __init__(self, cfg, raw_k, v, block_to_page, n_pages, max_view):
        self.cfg, self.geom = cfg, geom_of(cfg)
        dev = torch.device("cuda")
        self.raw_k, self.v = raw_k, v
        self.raw_d, self.v_d = pool_to_device(raw_k, dev), pool_to_device(v, dev)
        self.b2p = block_to_page
        self.b2p_d = torch.from_numpy(block_to_page.astype(np.int32)).to(dev)
        self.ws = K.WorkingSetArrays(cfg.n_blocks, n_pages)
        self.ws.reset()
        shape = (n_pages,) + tuple(self.raw_d.shape[1:])
        self.k_exec = torch.zeros(shape, dtype=self.raw_d.dtype, device=dev)
        self.v_exec = torch.zeros_like(self.k_exec)
        self.exec_pages = torch.empty(max_view, dtype=torch.int32, device=dev)
        self.counts = torch.zeros(16, dtype=torch.int32, device=dev)
        self.wsp = torch.empty(K.kvmem_working_set_workspace_bytes(max_view, n_pages), dtype=torch.uint8, device=dev)
        self.oracle = WorkingSet(cfg.n_blocks, n_pages)
        self.deltas_since_build = np.zeros(n_pages, np.int64)  # for the K tolerance only

    def step(self, t, view, first, max_deltas):
        vd = torch.from_numpy(view).cuda()
        K.kvmem_working_set_update(self.geom, BASE, self.ws, t, vd, first, max_deltas, self.b2p_d, self.raw_d,
                                   self.v_d, self.k_exec, self.v_exec, self.exec_pages, self.counts, self.wsp)
        torch.cuda.synchronize()
        ref = self.oracle.update(t, view, first, self.cfg.block_tokens, max_deltas)
        n = len(view)
        got_pages = self.exec_pages[:n].cpu().numpy()
        np.testing.assert_array_equal(got_pages, ref["exec_pages"])
        np.testing.assert_array_equal(self.counts[:8].cpu().numpy(), ref["counts"])
        o = self.oracle
        for name in ("block_page", "block_last_step", "page_block", "page_pos", "page_deltas"):
            np.testing.assert_array_equal(getattr(self.ws, name).cpu().numpy(), getattr(o, name), err_msg=name)
        hdr = self.ws.header.cpu().numpy()
        assert (hdr[0], hdr[1], hdr[2]) == (o.prev_step, o.n_prev, o.hand)
        for (_, _, p, _) in ref["build"]:
            self.deltas_since_build[p] = 0
        for (_, p, _) in ref["delta"]:
            self.deltas_since_build[p] += 1
        return ref

    def check_pool(self, view, first):
        bt = self.cfg.block_tokens
        pages = self.exec_pages[:len(view)].cpu().numpy()
        kx, vx = self.k_exec.cpu(), self.v_exec.cpu()
        bf16 = self.cfg.kv_dtype == "bf16"
        if bf16:
            kx = oracle.from_bf16_bits(kx.view(torch.int16).numpy().view(np.uint16)[pages]).astype(np.float64)
            vx = vx.view(torch.int16).numpy().view(np.uint16)[pages]
            raw = oracle.from_bf16_bits(self.raw_k[self.b2p[view]]).astype(np.float64)
        else:
            kx, vx = kx.numpy()[pages].astype(np.float64), vx.numpy()[pages]
            raw = self.raw_k[self.b2p[view]].astype(np.float64)
        np.testing.assert_array_equal(vx, self.v[self.b2p[view]])
        pos = (first + np.arange(len(view)) * bt)[:, None, None] + np.arange(bt)[None, None, :]
        want = oracle.rope(raw, np.broadcast_to(pos, raw.shape[:-1]), BASE)
        # each bf16 rounding errs by at most 2^-8 of the element; a later rotation
        # turns that error vector (norm <= 2^-8 of the pair's norm) into both
        # elements of the pair.  So after k delta steps: one ulp of the element
        # for the last rounding plus k * 2^-8 of the pair norm, plus the fp32
        # rotations (a few ulps of the pair norm each).
        k = self.deltas_since_build[pages][:, None, None, None]
        pn = pair_norm(want)
        tol = np.abs(want) * 2.0 ** -7 + pn * (k * 2.0 ** -8 + (k + 1) * 2.0 ** -18) if bf16 else \
            pn * 2.0 ** -20 * (k + 1)
        err = np.abs(kx - want)
        bad = err > tol
        assert not bad.any(), f"{bad.sum()} K elements off (max deltas {k.max()}, worst err/pair norm " \
                              f"{(err / np.maximum(pn, 1e-30)).max():.2e})"


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_recall_sequence(dt):
    cfg = W.small_config(n_kv_heads=2, n_q_heads=8, head_dim=128, block_tokens=16, kv_dtype=dt,
                         history_tokens=300 * 16, recent_tokens=4 * 16, budget_tokens=80 * 16)
    log(f"[case] working-set sequence {dt}")
    w = W.generate(cfg, 41)
    run = Runner(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page, n_pages=90, max_view=70)
    r = np.random.default_rng(3)
    totals = np.zeros(8, np.int64)
    for t, view in enumerate(random_views(7, cfg.n_blocks, 14, 10, 70)):
        first = int(r.choice([0, 16, 4096, int(r.integers(0, 1 << 20)) * 16]))
        ref = run.step(t * 3 + 1, view, first, 2)  # step ids need only increase
        run.check_pool(view, first)
        totals += ref["counts"]
    log(f"  totals |W| |R| |L| |E| |Lphys| delta rebuild evicted: {totals.tolist()}")
    assert totals[5] > 0 and totals[6] > 0 and totals[7] > 0  # every path ran


def test_repeat_and_shift():
    cfg = W.small_config(n_kv_heads=4, n_q_heads=16, head_dim=64, block_tokens=32, kv_dtype="bf16",
                         history_tokens=200 * 32, recent_tokens=2 * 32, budget_tokens=40 * 32)
    log("[case] working-set repeat / shift / full pool")
    w = W.generate(cfg, 42)
    view = np.sort(np.random.default_rng(1).choice(cfg.n_blocks, 40, replace=False)).astype(np.int32)
    run = Runner(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page, n_pages=40, max_view=40)  # P = n_view
    assert run.step(0, view, 0, 1)["counts"].tolist() == [40, 0, 40, 0, 40, 0, 0, 0]
    assert run.step(1, view, 0, 1)["counts"].tolist() == [40, 40, 0, 0, 0, 0, 0, 0]
    assert run.step(2, view, 32, 1)["counts"].tolist() == [40, 40, 0, 0, 0, 40, 0, 0]
    assert run.step(3, view, 64, 1)["counts"].tolist() == [40, 40, 0, 0, 0, 0, 40, 0]
    run.check_pool(view, 64)
    other = np.sort(np.setdiff1d(np.arange(cfg.n_blocks), view)[:40]).astype(np.int32)
    assert run.step(4, other, 64, 1)["counts"].tolist() == [40, 0, 40, 40, 40, 0, 0, 40]
    run.check_pool(other, 64)


def test_recall_points_on_oracle_selections():
    """Two consecutive recall points of a 4-layer workload: the oracle selects
    the working sets from two query sets; GPU and oracle place them."""
    cfg = W.small_config(n_layers=2, n_kv_heads=2, n_q_heads=8, head_dim=128, block_tokens=32, kv_dtype="bf16",
                         history_tokens=1200 * 32, recent_tokens=16 * 32, budget_tokens=200 * 32, n_q=32,
                         n_planted=8)
    log("[case] working sets of two recall points")
    w = W.generate(cfg, 43, n_query_sets=2)
    b2p = w.block_to_page
    index = np.stack([oracle.mean_k(k, b2p) for k in w.k_pool])
    k_eff = oracle.k_eff(cfg.budget_tokens, cfg.budget_tokens, cfg.block_tokens, cfg.n_blocks, 0, cfg.n_recent)
    run = Runner(cfg, w.k_pool[0], w.v_pool[0], b2p, n_pages=2 * cfg.budget_tokens // 32,
                 max_view=cfg.budget_tokens // 32)
    for t in range(2):
        rel = oracle.block_relevance(w.q[t], index, 0, cfg.n_recent)
        vb, _ = oracle.select(rel, 0, cfg.n_recent, k_eff, b2p)
        ref = run.step(t, vb[0].astype(np.int32), 0, 4)
        run.check_pool(vb[0], 0)
        log(f"  recall {t}: counts {ref['counts'].tolist()}")
