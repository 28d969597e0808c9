"""Pins for the CPU oracle: every check here comes from something other than the
oracle itself -- a closed form, an exact rational computation, brute force over
all subsets, a stated configuration number, or an independent library routine
(torch's scaled_dot_product_attention in float64).  Each group names the
passage of the paper it pins.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from paper_2609_04852_amd import workload as W


def round_to_f32(fr: Fraction) -> np.float32:
    """Correctly rounded (nearest, ties to even) fp32 value of an exact rational."""
    f = np.float32(float(fr))
    cands = [np.nextafter(f, np.float32(-np.inf)), f, np.nextafter(f, np.float32(np.inf))]
    return min(cands, key=lambda c: (abs(Fraction(float(c)) - fr),
                                     int(np.array(c, np.float32).view(np.uint32)) & 1))


def rng(seed=0):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- Eq. 9 ---
class TestMeanK:
    def test_single_token_block_is_identity(self):
        k = rng(1).standard_normal((5, 2, 1, 8)).astype(np.float32)
        b2p = np.array([3, 0, 4, 1, 2], np.int32)
        idx = oracle.mean_k(k, b2p)
        np.testing.assert_array_equal(idx, k[b2p, :, 0, :])

    def test_constant_block(self):
        vals = rng(2).standard_normal((4, 3)).astype(np.float32)
        k = np.broadcast_to(vals[:, :, None, None], (4, 3, 16, 8)).copy()
        idx = oracle.mean_k(k, np.arange(4, dtype=np.int32))
        np.testing.assert_array_equal(idx, np.broadcast_to(vals[:, :, None], (4, 3, 8)))

    @pytest.mark.parametrize("bt", [3, 5, 16])
    def test_exact_rational_mean_fp32(self, bt):
        k = (rng(bt).standard_normal((3, 2, bt, 4)) * 10.0 ** rng(bt + 1).integers(-3, 3, (3, 2, bt, 4))
             ).astype(np.float32)
        b2p = np.array([2, 0, 1], np.int32)
        idx = oracle.mean_k(k, b2p)
        for b in range(3):
            for g in range(2):
                for j in range(4):
                    exact = sum(Fraction(float(x)) for x in k[b2p[b], g, :, j]) / bt
                    assert idx[b, g, j] == round_to_f32(exact)

    def test_exact_rational_mean_bf16(self):
        x = rng(7).standard_normal((3, 2, 16, 8)).astype(np.float32)
        bits = W.bf16_bits(x)
        vals = W.bf16_to_f32(bits)
        b2p = np.array([1, 2, 0], np.int32)
        idx = oracle.mean_k(bits, b2p)
        for b in range(3):
            for g in range(2):
                for j in range(8):
                    exact = sum(Fraction(float(v)) for v in vals[b2p[b], g, :, j]) / 16
                    assert idx[b, g, j] == round_to_f32(exact)

    def test_block_reads_its_page(self):
        # page p holds the constant 100*p + g in head g
        p, hkv = 6, 2
        k = np.zeros((p, hkv, 4, 4), np.float32)
        for pg in range(p):
            for g in range(hkv):
                k[pg, g] = 100 * pg + g
        b2p = np.array([5, 3, 1, 0, 2, 4], np.int32)
        idx = oracle.mean_k(k, b2p)
        for b in range(p):
            for g in range(hkv):
                assert np.all(idx[b, g] == 100 * b2p[b] + g)

    def test_block_range_only(self):
        k = rng(3).standard_normal((8, 1, 4, 4)).astype(np.float32)
        b2p = np.arange(8, dtype=np.int32)
        idx = np.full((8, 1, 4), -7.0, np.float32)
        oracle.mean_k(k, b2p, first_block=2, n_blocks=3, index=idx)
        assert np.all(idx[:2] == -7.0) and np.all(idx[5:] == -7.0)
        np.testing.assert_array_equal(idx[2:5], oracle.mean_k(k, b2p)[2:5])


# ------------------------------------------------------- Eq. 5 / Eq. 7 ---
class TestBudget:
    @pytest.mark.parametrize("name", list(W.CONFIGS))
    def test_stated_configs(self, name):
        c = W.CONFIGS[name]
        k = oracle.k_eff(c.budget_tokens, c.budget_tokens, c.block_tokens, c.n_blocks,
                         c.sink_blocks, c.n_recent)
        assert k == c.top_k

    def test_active_budget_is_the_minimum(self):
        # B_a = min(B_model, B_gpu): the smaller limit decides
        assert oracle.k_eff(262144, 100_000, 16, 65536, 0, 512) == (100_000 - 8192) // 16
        assert oracle.k_eff(50_000, 262144, 16, 65536, 2, 512) == (50_000 - 514 * 16) // 16

    def test_capped_by_candidates(self):
        assert oracle.k_eff(10**9, 10**9, 16, 100, 1, 4) == 95

    def test_budget_below_mandatory(self):
        with pytest.raises(ValueError):
            oracle.k_eff(63, 10**6, 16, 100, 0, 4)
        assert oracle.k_eff(64, 10**6, 16, 100, 0, 4) == 0


# --------------------------------------------------------------- Eq. 10 ---
def sigmoid(x):
    return 1.0 / (1.0 + math.exp(-x))


def idx4(rows):
    """index [L=1][M][Hkv][d=4] from a nested list rows[b][g] = first coordinate."""
    arr = np.zeros((1, len(rows), len(rows[0]), 4), np.float32)
    for b, r in enumerate(rows):
        for g, v in enumerate(r):
            arr[0, b, g, 0] = v
    return arr


class TestRelevance:
    def test_two_candidates_logistic(self):
        q = np.zeros((1, 1, 1, 4), np.float32)
        q[..., 0] = 2.0
        index = idx4([[1.0], [0.5]])
        r = oracle.block_relevance(q, index, 0, 0)
        # logits 2*1/sqrt(4) = 1.0 and 0.5
        assert r[0, 0] == pytest.approx(sigmoid(0.5), abs=1e-15)
        assert r[0, 1] == pytest.approx(sigmoid(-0.5), abs=1e-15)

    def test_gqa_grouping_and_head_mean(self):
        # Hkv=2, Hq=4: heads 0,1 read KV head 0, heads 2,3 read KV head 1
        a = [1.0, 3.0, -2.0, 5.0]
        q = np.zeros((1, 1, 4, 4), np.float32)
        q[0, 0, :, 0] = a
        index = idx4([[0.75, 0.4], [0.25, 0.4]])  # KV head 1 cannot tell the blocks apart
        r = oracle.block_relevance(q, index, 0, 0)
        expect0 = (sigmoid(a[0] * 0.5 / 2) + sigmoid(a[1] * 0.5 / 2) + 0.5 + 0.5) / 4
        assert r[0, 0] == pytest.approx(expect0, abs=1e-15)
        assert r[0, 1] == pytest.approx(1 - expect0, abs=1e-15)

    def test_layers_mean_and_query_token_sum(self):
        # L=2, n_q=2, Hq=Hkv=1: R = sum_m mean_l p
        q = np.zeros((2, 2, 1, 4), np.float32)
        q[0, 0, 0, 0], q[0, 1, 0, 0], q[1, 0, 0, 0], q[1, 1, 0, 0] = 1.0, -4.0, 6.0, 2.0
        index = np.zeros((2, 2, 1, 4), np.float32)
        index[0, :, 0, 0] = [1.0, 0.0]
        index[1, :, 0, 0] = [0.0, 0.5]
        r = oracle.block_relevance(q, index, 0, 0)
        # layer 0 logit gap (b0 - b1) = q/2 ; layer 1 gap = -q*0.5/2
        e = lambda qa, qb: (sigmoid(qa * 1.0 / 2) + sigmoid(-qb * 0.5 / 2)) / 2
        expect0 = e(1.0, 6.0) + e(-4.0, 2.0)
        assert r[0, 0] == pytest.approx(expect0, abs=1e-15)
        assert r[0, 0] + r[0, 1] == pytest.approx(2.0, abs=1e-15)

    def test_group_max(self):
        q = np.zeros((1, 2, 4, 4), np.float32)
        a = np.array([[1.0, -3.0, 2.0, 0.5], [-1.0, 4.0, -2.0, 0.25]])
        q[0, :, :, 0] = a
        index = idx4([[1.0, -1.0], [0.0, 0.0]])
        r = oracle.block_relevance(q, index, 0, 0, mode=oracle.MAX_GROUP)
        assert r.shape == (2, 2)
        for g, sign in ((0, 1.0), (1, -1.0)):
            ps0 = [sigmoid(sign * a[m, h] / 2) for m in range(2) for h in (2 * g, 2 * g + 1)]
            assert r[g, 0] == pytest.approx(max(ps0), abs=1e-15)
            assert r[g, 1] == pytest.approx(max(1 - p for p in ps0), abs=1e-15)

    def test_explicit_scale(self):
        q = np.zeros((1, 1, 1, 4), np.float32)
        q[..., 0] = 2.0
        index = idx4([[1.0], [0.5]])
        r = oracle.block_relevance(q, index, 0, 0, scale=1.0)
        assert r[0, 0] == pytest.approx(sigmoid(1.0), abs=1e-15)

    def test_uniform_keys(self):
        q = rng(4).standard_normal((1, 3, 8, 16)).astype(np.float32)
        index = np.broadcast_to(rng(5).standard_normal((1, 1, 2, 16)).astype(np.float32),
                                (1, 40, 2, 16)).copy()
        r = oracle.block_relevance(q, index, 2, 3)
        np.testing.assert_allclose(r[0, 2:37], 3.0 / 35, rtol=0, atol=1e-15)

    def test_mass_sums_to_query_count(self):
        q = rng(6).standard_normal((2, 3, 8, 32)).astype(np.float32) * 3
        index = rng(7).standard_normal((2, 300, 2, 32)).astype(np.float32)
        r = oracle.block_relevance(q, index, 4, 10)
        assert np.isinf(r[0, :4]).all() and np.isinf(r[0, 290:]).all()
        assert r[0, 4:290].sum() == pytest.approx(3.0, abs=1e-12)

    def test_reserved_blocks_outside_softmax(self):
        q = rng(8).standard_normal((1, 1, 4, 16)).astype(np.float32)
        index = rng(9).standard_normal((1, 50, 2, 16)).astype(np.float32)
        r1 = oracle.block_relevance(q, index, 3, 5)
        index2 = index.copy()
        index2[0, :3] *= 50.0
        index2[0, 45:] *= -30.0
        r2 = oracle.block_relevance(q, index2, 3, 5)
        np.testing.assert_array_equal(r1, r2)

    def test_single_head_rank_follows_logits(self):
        q = rng(10).standard_normal((1, 1, 1, 64)).astype(np.float32)
        index = rng(11).standard_normal((1, 500, 1, 64)).astype(np.float32)
        r = oracle.block_relevance(q, index, 0, 0)[0]
        logits = index[0, :, 0, :].astype(np.float64) @ q[0, 0, 0].astype(np.float64)
        assert list(np.argsort(-r, kind="stable")) == list(np.argsort(-logits, kind="stable"))


# ------------------------------------------------------------ selector ---
def brute_force_select(r32, lo, hi, k):
    """Max-sum k-subset of candidates; among equal sums the lexicographically smallest ids."""
    best = None
    for comb in itertools.combinations(range(lo, hi), k):
        s = sum(Fraction(float(r32[b])) for b in comb)
        key = (-s, comb)
        if best is None or key < best:
            best = key
    return list(best[1]) if best else []


class TestSelect:
    @pytest.mark.parametrize("seed", range(6))
    def test_brute_force_with_ties(self, seed):
        g = rng(100 + seed)
        m, s, rr = 12, int(g.integers(0, 3)), int(g.integers(0, 3))
        r = g.integers(0, 4, m).astype(np.float64)  # many exact ties
        k = int(g.integers(0, m - s - rr + 1))
        b2p = g.permutation(m).astype(np.int32)
        vb, vp = oracle.select(r[None], s, rr, k, b2p)
        chosen = brute_force_select(r.astype(np.float32), s, m - rr, k)
        expect = list(range(s)) + chosen + list(range(m - rr, m))
        assert vb[0].tolist() == expect
        assert vp[0].tolist() == [int(b2p[b]) for b in expect]

    def test_decision_in_fp32(self):
        # differ only below fp32 resolution: a tie, so the lower id wins
        r = np.array([[1.0, 1.0 + 1e-12, 0.5]])
        vb, _ = oracle.select(r, 0, 0, 1, np.arange(3, dtype=np.int32))
        assert vb[0].tolist() == [0]

    def test_all_and_none(self):
        r = rng(12).random((1, 20))
        b2p = np.arange(20, dtype=np.int32)
        assert oracle.select(r, 2, 3, 15, b2p)[0][0].tolist() == list(range(20))
        assert oracle.select(r, 2, 3, 0, b2p)[0][0].tolist() == [0, 1, 17, 18, 19]

    def test_rows_independent(self):
        r = rng(13).random((3, 30))
        b2p = rng(14).permutation(30).astype(np.int32)
        vb, vp = oracle.select(r, 1, 2, 7, b2p)
        for s in range(3):
            vb1, vp1 = oracle.select(r[s:s + 1], 1, 2, 7, b2p)
            assert vb[s].tolist() == vb1[0].tolist() and vp[s].tolist() == vp1[0].tolist()
            top = sorted(range(1, 28), key=lambda b: (-np.float32(r[s, b]), b))[:7]
            assert vb[s].tolist() == [0] + sorted(top) + [28, 29]


# ----------------------------------------------------------- attention ---
def sdpa(q, k, v, scale):
    """torch scaled_dot_product_attention in float64: q [H][d], k/v [H][T][d]."""
    qt = torch.from_numpy(np.asarray(q, np.float64))[None, :, None, :]
    kt = torch.from_numpy(np.asarray(k, np.float64))[None]
    vt = torch.from_numpy(np.asarray(v, np.float64))[None]
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)
    lse = torch.logsumexp(scale * (kt @ qt.transpose(-1, -2))[..., 0], dim=-1)
    return o[0, :, 0, :].numpy(), lse[0].numpy()


def widen(pool):
    return W.bf16_to_f32(pool) if pool.dtype == np.uint16 else pool


def gather(pool, pages, g, last=None):
    """Dense [T][d] keys of KV head g over a page list (last page cut to `last` tokens)."""
    rows = [widen(pool)[p, g] for p in pages]
    if last is not None:
        rows[-1] = rows[-1][:last]
    return np.concatenate(rows, 0).astype(np.float64)


def rand_pools(seed, p, hkv, bt, d, bf16):
    g = rng(seed)
    k = g.standard_normal((p, hkv, bt, d)).astype(np.float32)
    v = g.standard_normal((p, hkv, bt, d)).astype(np.float32)
    if bf16:
        return W.bf16_bits(k), W.bf16_bits(v)
    return k, v


class TestAttention:
    def test_single_token(self):
        k, v = rand_pools(20, 3, 1, 4, 8, False)
        q = rng(21).standard_normal((1, 2, 8)).astype(np.float32)
        out, lse = oracle.view_attention(q, k, v, np.array([[2]], np.int32), last_page_tokens=1)
        for h in range(2):
            np.testing.assert_array_equal(out[0, h], v[2, 0, 0].astype(np.float64))
            a = float(np.dot(q[0, h].astype(np.float64), k[2, 0, 0].astype(np.float64))) / math.sqrt(8)
            assert lse[0, h] == pytest.approx(a, abs=1e-12)

    def test_identical_keys_average_values(self):
        k, v = rand_pools(22, 4, 1, 8, 16, False)
        k[:] = k[0, 0, 0]
        q = rng(23).standard_normal((2, 1, 16)).astype(np.float32)
        pages = np.array([[3, 1, 2]], np.int32)
        out, lse = oracle.view_attention(q, k, v, pages)
        mean_v = np.concatenate([v[p, 0] for p in (3, 1, 2)], 0).astype(np.float64).mean(0)
        for m in range(2):
            np.testing.assert_allclose(out[m, 0], mean_v, rtol=0, atol=1e-14)
            a = float(np.dot(q[m, 0].astype(np.float64), k[0, 0, 0].astype(np.float64))) / 4.0
            assert lse[m, 0] == pytest.approx(a + math.log(24), abs=1e-12)

    @pytest.mark.parametrize("bf16", [False, True])
    @pytest.mark.parametrize("n_sel", [1, 2])
    def test_matches_torch_sdpa(self, bf16, n_sel):
        p, hkv, bt, d, hq, nq = 40, 2, 16, 32, 8, 2
        k, v = rand_pools(24 + bf16, p, hkv, bt, d, bf16)
        q = rng(26).standard_normal((nq, hq, d)).astype(np.float32)
        pages = np.stack([rng(27 + s).choice(p, 9, replace=False) for s in range(n_sel)]).astype(np.int32)
        out, lse = oracle.view_attention(q, k, v, pages, last_page_tokens=5, scale=0.3)
        for m in range(nq):
            for h in range(hq):
                g = h // (hq // hkv)
                s = 0 if n_sel == 1 else g
                o_ref, l_ref = sdpa(q[m, h][None], gather(k, pages[s], g, 5)[None],
                                    gather(v, pages[s], g, 5)[None], 0.3)
                np.testing.assert_allclose(out[m, h], o_ref[0], rtol=0, atol=1e-12)
                assert lse[m, h] == pytest.approx(float(l_ref[0]), abs=1e-12)

    @pytest.mark.parametrize("bf16", [False, True])
    def test_view_equals_masked_dense(self, bf16):
        m_blocks, hkv, bt, d = 30, 2, 8, 16
        k, v = rand_pools(30, m_blocks, hkv, bt, d, bf16)
        q = rng(31).standard_normal((3, 4, d)).astype(np.float32)
        b2p = rng(32).permutation(m_blocks).astype(np.int32)
        for n_sel in (1, 2):
            vb = np.stack([np.sort(rng(33 + s).choice(m_blocks, 11, replace=False))
                           for s in range(n_sel)]).astype(np.int32)
            vp = b2p[vb]
            o1, l1 = oracle.view_attention(q, k, v, vp, last_page_tokens=3)
            o2, l2 = oracle.masked_dense_attention(q, k, v, b2p, vb, last_page_tokens=3)
            np.testing.assert_allclose(o1, o2, rtol=0, atol=1e-12)
            np.testing.assert_allclose(l1, l2, rtol=0, atol=1e-12)

    def test_full_selection_is_full_attention(self):
        c = W.small_config(history_tokens=1024, recent_tokens=64, n_planted=2, top_k=60)
        w = W.generate(c, seed=5)
        index = oracle.mean_k(w.k_pool[0], w.block_to_page)[None]
        r = oracle.block_relevance(w.q[0], index, 0, c.n_recent)
        kk = oracle.k_eff(10**9, 10**9, c.block_tokens, c.n_blocks, 0, c.n_recent)
        assert kk == c.n_candidates
        vb, vp = oracle.select(r, 0, c.n_recent, kk, w.block_to_page)
        assert vb[0].tolist() == list(range(c.n_blocks))
        out, lse = oracle.view_attention(w.q[0, 0], w.k_pool[0], w.v_pool[0], vp)
        chrono = w.block_to_page  # every block in chronological order
        for h in range(c.n_q_heads):
            o_ref, l_ref = sdpa(w.q[0, 0, 0, h][None], gather(w.k_pool[0], chrono, 0)[None],
                                gather(w.v_pool[0], chrono, 0)[None], 1 / math.sqrt(c.head_dim))
            np.testing.assert_allclose(out[0, h], o_ref[0], rtol=0, atol=1e-12)
            assert lse[0, h] == pytest.approx(float(l_ref[0]), abs=1e-12)


# ---------------------------------------------------------- generator ---
class TestWorkload:
    def test_bf16_rne_against_bit_arithmetic(self):
        x = np.concatenate([rng(40).standard_normal(10000).astype(np.float32),
                            # exact ties: low half 0x8000 with even and odd kept lsb
                            np.array([0x3F808000, 0x3F818000, 0xBF808000, 0x3F80FFFF],
                                     np.uint32).view(np.float32)])
        u = x.view(np.uint32).astype(np.uint64)
        expect = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
        np.testing.assert_array_equal(W.bf16_bits(x), expect)
        np.testing.assert_array_equal(W.bf16_to_f32(expect[:4]).view(np.uint32),
                                      expect[:4].astype(np.uint32) << 16)

    def test_deterministic(self):
        a = W.generate("tiny", seed=9)
        b = W.generate("tiny", seed=9)
        np.testing.assert_array_equal(a.k_pool[0], b.k_pool[0])
        np.testing.assert_array_equal(a.v_pool[0], b.v_pool[0])
        np.testing.assert_array_equal(a.q, b.q)
        np.testing.assert_array_equal(a.block_to_page, b.block_to_page)
        c = W.generate("tiny", seed=10)
        assert not np.array_equal(a.k_pool[0], c.k_pool[0])

    def test_planted_keys_are_aligned(self):
        w = W.generate("tiny", seed=0)
        c = w.cfg
        u = w.q[0, 0, :, :, :].reshape(-1, c.head_dim).astype(np.float64).mean(0)
        u /= np.linalg.norm(u)
        assert len(w.planted) == c.n_planted
        assert np.all((w.planted >= 0) & (w.planted < c.n_blocks - c.n_recent))
        for b in w.planted:
            keys = w.k_pool[0][w.block_to_page[b], 0].astype(np.float64)
            cos = keys @ u / np.linalg.norm(keys, axis=1)
            assert np.all(np.abs(cos - 0.9) < 1e-5)
            assert np.allclose(np.linalg.norm(keys, axis=1), math.sqrt(c.head_dim), rtol=1e-5)

    def test_planted_blocks_are_selected(self):
        # sanity of the synthetic recipe, not parity: the planted blocks win the selection
        for seed in range(3):
            w = W.generate("tiny", seed=seed)
            c = w.cfg
            index = oracle.mean_k(w.k_pool[0], w.block_to_page)[None]
            r = oracle.block_relevance(w.q[0], index, 0, c.n_recent)
            vb, _ = oracle.select(r, 0, c.n_recent, c.top_k, w.block_to_page)
            assert set(w.planted.tolist()) <= set(vb[0].tolist())


# ---- Position handling: RoPE removal for the index (Sec. 4.3) and re-encoding
# at compact positions in the execution view (Sec. 4.4, Sec. 5.3) ----------
class TestRope:
    def test_d2_is_multiplication_by_unit_complex(self):
        # with d = 2 the only frequency is base^0 = 1: a plane rotation by p radians
        import cmath
        for p in (0, 1, 5, -3, 1000, 123457):
            z = complex(0.3, -1.7) * cmath.exp(1j * p)
            y = oracle.rope(np.array([[0.3, -1.7]]), [p], 10000.0)[0]
            assert abs(y[0] - z.real) < 1e-12 and abs(y[1] - z.imag) < 1e-12

    def test_pairs_are_half_apart_with_geometric_frequencies(self):
        # unit vectors show which dims pair up and at which rate they turn:
        # e_j mixes only with e_{j+d/2}, at angle p * base^(-2j/d)
        d, base, p = 8, 400.0, 7
        for j in range(d // 2):
            e = np.zeros(d)
            e[j] = 1.0
            y = oracle.rope(e[None], [p], base)[0]
            a = p * base ** (-2.0 * j / d)
            expect = np.zeros(d)
            expect[j], expect[j + d // 2] = math.cos(a), math.sin(a)
            np.testing.assert_allclose(y, expect, atol=1e-14)

    def test_inverse_composition_norm(self):
        x = rng(1).standard_normal((6, 64))
        a = np.array([0, 1, 17, 4096, 262143, 1048575])
        b = np.array([3, -1, 100, -4096, 5, 7])
        np.testing.assert_allclose(oracle.rope(x, 0, 1e6), x, atol=0)
        np.testing.assert_allclose(oracle.rope(oracle.rope(x, a, 1e6), -a, 1e6), x, atol=1e-12)
        np.testing.assert_allclose(oracle.rope(oracle.rope(x, a, 1e6), b, 1e6), oracle.rope(x, a + b, 1e6),
                                   atol=1e-9)
        y = oracle.rope(x, a, 1e6)
        h = 32
        np.testing.assert_allclose(np.hypot(y[:, :h], y[:, h:]), np.hypot(x[:, :h], x[:, h:]), rtol=1e-13)

    def test_dot_products_depend_only_on_relative_position(self):
        q, k = rng(2).standard_normal((2, 128))
        for m, n in ((10, 3), (5000, 4000), (7, 900)):
            base_dot = oracle.rope(q, m, 1e4) @ oracle.rope(k, n, 1e4)
            for s in (1, 333, 100000):
                assert abs(oracle.rope(q, m + s, 1e4) @ oracle.rope(k, n + s, 1e4) - base_dot) < 1e-9

    def test_mean_k_of_encoded_keys_recovers_the_raw_mean(self):
        # keys encoded at their blocks' positions and stored in fp32: removing the
        # encoding before the mean gives the mean of the raw keys (up to fp32 storage)
        r = rng(3)
        n_pages, hkv, bt, d = 40, 2, 16, 64
        raw = r.standard_normal((n_pages, hkv, bt, d)).astype(np.float32)
        b2p = r.permutation(n_pages).astype(np.int32)
        for block_pos in (None, r.integers(0, 10 ** 6, n_pages)):
            p0 = np.arange(n_pages) * bt if block_pos is None else block_pos
            pos = np.empty((n_pages, hkv, bt), np.int64)
            pos[b2p] = (p0[:, None, None] + np.arange(bt)[None, None, :])
            enc = oracle.rope(raw.astype(np.float64), pos, 1e6).astype(np.float32)
            got = oracle.mean_k_rope(enc, b2p, 1e6, block_pos=block_pos)
            want = oracle.mean_k(raw, b2p)
            np.testing.assert_allclose(got, want, atol=2e-6, rtol=0)
        # and the plain index is not what you get from encoded keys (the removal matters)
        assert np.abs(oracle.mean_k(enc, b2p) - want).max() > 0.1

    def test_bf16_rounding_is_nearest_even(self):
        x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 3.140625, 1e-3], np.float32)
        bits = oracle.to_bf16_bits(x)
        back = oracle.from_bf16_bits(bits)
        # 1 + 2^-8 is a tie between 1 and 1 + 2^-7: even mantissa (1.0) wins;
        # 1 + 3*2^-8 ties between 1 + 2^-7 and 1 + 2^-6: the even one is 1 + 2^-6
        np.testing.assert_array_equal(back[:4], np.array([1.0, 1.0, 1.0 + 2 ** -6, -2.5], np.float32))
        assert abs(back[5] - 1e-3) <= 2 ** -9 * 1e-3

    def test_materialize_encodes_each_token_at_its_compact_position(self):
        r = rng(4)
        n_pages, hkv, bt, d = 12, 2, 16, 64
        raw = r.standard_normal((n_pages, hkv, bt, d)).astype(np.float32)
        v = r.standard_normal((n_pages, hkv, bt, d)).astype(np.float32)
        src = np.array([5, 0, 11, 3])
        pos = np.array([0, 16, 32, 48])  # four blocks laid out back to back
        k_out, v_out = oracle.materialize(raw, v, src, pos, 1e6)
        np.testing.assert_array_equal(v_out, v[src])
        for i, p in enumerate(pos):
            for t in (0, 7, 15):
                np.testing.assert_allclose(k_out[i, :, t], oracle.rope(raw[src[i], :, t], p + t, 1e6), atol=0)
        # attention logits against a query at position P only see the offset P - (p + t)
        q = r.standard_normal(d)
        P = 64
        lhs = oracle.rope(q, P, 1e6) @ k_out[2, 1, 9]
        rhs = q @ oracle.rope(raw[src[2], 1, 9], (pos[2] + 9) - P, 1e6)
        assert abs(lhs - rhs) < 1e-9


# ---- FP8 K/V (the KV-cache precision of the evaluation platforms, Sec. 6):
# OCP E4M3 codes with one fp32 scale per pool ------------------------------
def fp8_pools(seed, p, hkv, bt, d, scale):
    """E4M3 codes of two pools (quantised by torch's own float8 cast) and their
    fp64 values decoded by torch."""
    g = rng(seed)
    out = []
    for _ in range(2):
        x = torch.from_numpy((g.standard_normal((p, hkv, bt, d)) * 3.0 / scale).astype(np.float32))
        codes = x.clamp(-448.0, 448.0).to(torch.float8_e4m3fn)
        out.append((codes.view(torch.uint8).numpy(), codes.to(torch.float64).numpy() * float(np.float32(scale))))
    return out


class TestFp8:
    def test_decode_matches_torch_float8_e4m3fn(self):
        codes = np.arange(256, dtype=np.uint8)
        ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
        got = oracle.decode_e4m3(codes)
        np.testing.assert_array_equal(got, ref)
        assert np.array_equal(np.signbit(got[~np.isnan(got)]), np.signbit(ref[~np.isnan(ref)]))

    def test_format_landmarks(self):
        d = oracle.decode_e4m3(np.arange(256, dtype=np.uint8))
        assert d[0x38] == 1.0 and d[0xB8] == -1.0
        assert d[0x7E] == 448.0 and d[0xFE] == -448.0       # largest finite
        assert d[0x08] == 2.0 ** -6                          # smallest normal
        assert d[0x01] == 2.0 ** -9                          # smallest subnormal
        assert d[0x07] == 7 * 2.0 ** -9                      # largest subnormal
        assert d[0x00] == 0.0 and np.signbit(d[0x80])       # +0, -0
        assert np.isnan(d[0x7F]) and np.isnan(d[0xFF])       # the only NaNs, no infinities
        assert np.isfinite(np.delete(d, [0x7F, 0xFF])).all()

    def test_positive_codes_are_ordered_and_sign_is_the_top_bit(self):
        d = oracle.decode_e4m3(np.arange(256, dtype=np.uint8))
        assert (np.diff(d[:0x7F]) > 0).all()
        np.testing.assert_array_equal(d[0x80:0xFF], -d[:0x7F])
        # eight codes per binade, each binade twice as wide as the one below
        for e in range(2, 16):
            assert d[8 * e] == 2 * d[8 * (e - 1)]

    def test_pool_scale_multiplies(self):
        codes = np.arange(256, dtype=np.uint8)
        s = np.float32(0.0173)
        np.testing.assert_array_equal(oracle.decode_fp8(codes, s), oracle.decode_e4m3(codes) * float(s))

    @pytest.mark.parametrize("bt", [16, 5])
    def test_mean_k_of_fp8_pool_is_exact_mean(self, bt):
        s = np.float32(0.0173)
        (codes, vals), _ = fp8_pools(40 + bt, 4, 2, bt, 8, s)
        b2p = np.array([2, 0, 3, 1], np.int32)
        idx = oracle.mean_k(oracle.decode_fp8(codes, s), b2p)
        for b in range(4):
            for g in range(2):
                for j in range(8):
                    exact = sum(Fraction(float(x)) for x in vals[b2p[b], g, :, j]) / bt
                    assert idx[b, g, j] == round_to_f32(exact)

    def test_attention_on_fp8_pool_matches_torch_sdpa(self):
        p, hkv, bt, d, hq = 20, 2, 16, 32, 4
        (kc, kv), (vc, vv) = fp8_pools(50, p, hkv, bt, d, np.float32(2.0 ** -5))
        q = rng(51).standard_normal((1, hq, d)).astype(np.float32)
        pages = rng(52).choice(p, 7, replace=False).astype(np.int32)[None]
        out, lse = oracle.view_attention(q, oracle.decode_fp8(kc, 2.0 ** -5), oracle.decode_fp8(vc, 2.0 ** -5),
                                         pages, last_page_tokens=9, scale=0.2)
        for h in range(hq):
            g = h // (hq // hkv)
            kk = np.concatenate([kv[pg, g] for pg in pages[0]], 0)[:-(bt - 9)]
            vv_ = np.concatenate([vv[pg, g] for pg in pages[0]], 0)[:-(bt - 9)]
            o_ref, l_ref = sdpa(q[0, h][None], kk[None], vv_[None], 0.2)
            np.testing.assert_allclose(out[0, h], o_ref[0], rtol=0, atol=1e-12)
            assert lse[0, h] == pytest.approx(float(l_ref[0]), abs=1e-12)


# ---- Working-set update at a recall point (Sec. 4.4, Eq. 11, Eq. 12) ------
from oracle.working_set import WorkingSet  # noqa: E402


def ws_snapshot(ws):
    return {k: (v.copy() if isinstance(v, np.ndarray) else v) for k, v in vars(ws).items()}


class TestWorkingSet:
    def random_views(self, seed, m, steps, lo, hi):
        r = rng(seed)
        out, prev = [], None
        for _ in range(steps):
            n = int(r.integers(lo, hi + 1))
            if prev is not None and r.random() < 0.6:  # overlap with the previous working set
                keep = r.choice(prev, size=min(len(prev), n // 2), replace=False)
                rest = r.choice(np.setdiff1d(np.arange(m), keep), size=n - len(keep), replace=False)
                v = np.sort(np.concatenate([keep, rest]))
            else:
                v = np.sort(r.choice(m, size=n, replace=False))
            out.append(v)
            prev = v
        return out

    def test_delta_sets_and_physical_loads(self):
        m, p = 60, 25
        ws = WorkingSet(m, p)
        w_prev = set()
        for t, view in enumerate(self.random_views(1, m, 40, 3, 20)):
            before = ws_snapshot(ws)
            g_prev = {b for b in range(m) if before["block_page"][b] >= 0}
            out = ws.update(t, view, 0, 16, 3)
            w = set(view.tolist())
            r_t, l_t, e_t = w & w_prev, w - w_prev, w_prev - w          # Eq. 11
            l_phys = w - g_prev                                        # Eq. 12
            c = out["counts"]
            assert (c[0], c[1], c[2], c[3], c[4]) == (len(w), len(r_t), len(l_t), len(e_t), len(l_phys))
            assert r_t | l_t == w and not (r_t & l_t)
            # every selected block is resident, one page each, and hits kept their pages
            pages = out["exec_pages"]
            assert len(set(pages.tolist())) == len(w) and (pages >= 0).all() and (pages < p).all()
            for b, pg in zip(view, pages):
                assert ws.block_page[b] == pg and ws.page_block[pg] == b
                if b in g_prev:
                    assert pg == before["block_page"][b]
            # the bijection between resident blocks and occupied pages
            res = {b: int(ws.block_page[b]) for b in range(m) if ws.block_page[b] >= 0}
            assert sorted(res.values()) == sorted(int(q) for q in np.nonzero(ws.page_block >= 0)[0])
            assert all(ws.page_block[q] == b for b, q in res.items())
            # loads only for L_phys, into pages that held no block of W_t
            built = {bb for (_, bb, _, _) in out["build"]}
            assert l_phys <= built
            w_prev = w

    def test_pages_taken_in_clock_order(self):
        m, p = 40, 12
        ws = WorkingSet(m, p)
        out = ws.update(0, np.arange(0, 10), 0, 16, 3)          # an empty pool fills from page 0
        assert out["exec_pages"].tolist() == list(range(10)) and ws.hand == 10
        out = ws.update(1, np.array([2, 3, 20, 21, 22, 23]), 0, 16, 3)
        # hits 2, 3 keep pages 2, 3; the four misses take pages 10, 11, 0, 1 (from the hand,
        # skipping nothing: pages 0 and 1 held blocks 0 and 1, which leave the pool)
        assert out["exec_pages"].tolist() == [2, 3, 10, 11, 0, 1]
        assert ws.hand == 2 and out["counts"][7] == 2
        assert ws.block_page[0] == -1 and ws.block_page[1] == -1 and ws.block_page[4] == 4

    def test_unchanged_working_set_moves_nothing(self):
        ws = WorkingSet(100, 50)
        v = np.array([3, 17, 40, 41, 99])
        ws.update(0, v, 128, 32, 2)
        out = ws.update(1, v, 128, 32, 2)
        assert out["counts"].tolist() == [5, 5, 0, 0, 0, 0, 0, 0] and not out["build"] and not out["delta"]

    def test_delta_bound_then_rebuild(self):
        ws = WorkingSet(10, 10)
        v = np.array([1, 5])
        ws.update(0, v, 0, 16, 2)
        kinds = []
        for t in range(1, 8):
            out = ws.update(t, v, 16 * t, 16, 2)                   # the view shifts by one block per step
            kinds.append((len(out["delta"]), out["counts"][6]))
            assert all(s == 16 for (_, _, s) in out["delta"])
        # two delta re-encodings, then a rebuild from raw K, and so on
        assert kinds == [(2, 0), (2, 0), (0, 2), (2, 0), (2, 0), (0, 2), (2, 0)]

    def test_key_contents_follow_positions(self):
        # play the builds and deltas on fp64 pages with the oracle's RoPE: after any
        # sequence the page of view block i holds RoPE(raw K, first_position + i*Bt + t)
        m, p, bt, d = 30, 14, 4, 8
        raw = rng(5).standard_normal((m, 1, bt, d))
        pool = np.zeros((p, 1, bt, d))
        ws = WorkingSet(m, p)
        views = self.random_views(6, m, 25, 2, 10)
        for t, view in enumerate(views):
            first = int(rng(100 + t).integers(0, 500))
            out = ws.update(t, view, first, bt, 3)
            for (i, b, pg, pos) in out["build"]:
                pool[pg] = oracle.rope(raw[b], pos + np.arange(bt)[None, :], 1e4)
            for (i, pg, s) in out["delta"]:
                pool[pg] = oracle.rope(pool[pg], np.full((1, bt), s), 1e4)
            for i, (b, pg) in enumerate(zip(view, out["exec_pages"])):
                want = oracle.rope(raw[b], first + i * bt + np.arange(bt)[None, :], 1e4)
                np.testing.assert_allclose(pool[pg], want, atol=1e-10)
