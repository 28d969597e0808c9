"""Comparison helpers for the GPU-vs-oracle parity tests.

Acceptance rules (the tolerances are written here, once):
  * Mean-K index: bitwise equal to the oracle (both sum exactly in fp64 and
    round once to fp32).
  * Selection: every candidate whose fp32 oracle score lies more than 1e-5
    (relative) above the k-th score must be selected, every one more than 1e-5
    below must not be; only candidates inside that band may differ.  Sink and
    recent blocks must be present, the view must be strictly ascending, and
    view_pages must equal block_to_page[view_blocks] exactly.
  * Scores: within 1e-5 relative of the oracle's fp64 score.
  * Attention: within 2e-2 absolute for bf16 K/V and 1e-4 for fp32 K/V,
    elementwise, on the same view.  FP8 K/V takes the low-precision bound
    (2e-2), against the oracle on the same codes decoded in fp64.
  * Attention, regression bound: the kernels keep q and the softmax weights
    at fp32 accuracy (hi + lo bf16 pairs on the matrix cores) and accumulate
    in fp32, so their measured error is 1e-7 to 2e-6 on the output and about
    1e-5 on the log-sum-exp.  Every case must also stay within 1e-4 of the
    oracle (output and log-sum-exp, every K/V type), so that losing the lo
    halves (about 1e-3 of error) or an fp32 accumulation step fails even
    though it would pass the 2e-2 contract bound.
"""
import numpy as np

BAND = 1e-5
ATOL = {"bf16": 2e-2, "f32": 1e-4, "fp8": 2e-2}
REGRESSION_ATOL = 1e-4
SCORE_RTOL = 1e-5


def oracle_pool(cfg, pool):
    """The pool as the oracle reads it: FP8 codes decoded (times the pool scale)
    by the oracle's own decoder, other types as stored."""
    import oracle
    return oracle.decode_fp8(pool, cfg.kv_scale) if cfg.kv_dtype == "fp8" else pool


def log(*a):
    print(*a, flush=True)


def assert_index_bitwise(gpu_index: np.ndarray, ref_index: np.ndarray):
    assert gpu_index.shape == ref_index.shape
    same = gpu_index.view(np.uint32) == ref_index.view(np.uint32)
    n_bad = int((~same).sum())
    assert n_bad == 0, f"{n_bad} index entries differ from the oracle (bitwise)"


def kth_score(r32_cand: np.ndarray, k: int) -> float:
    """fp32 score of the k-th candidate in (score desc, id asc) order."""
    order = np.lexsort((np.arange(r32_cand.size), -r32_cand.astype(np.float64)))
    return float(r32_cand[order[k - 1]])


def check_selection(view_blocks: np.ndarray, view_pages: np.ndarray, relevance: np.ndarray,
                    block_to_page: np.ndarray, n_sink: int, n_recent: int, k_eff: int,
                    ref_view: np.ndarray | None = None) -> dict:
    """Check each selection row; returns counts of in-band differences."""
    n_sel, m = relevance.shape
    n_view = n_sink + k_eff + n_recent
    assert view_blocks.shape == (n_sel, n_view), (view_blocks.shape, (n_sel, n_view))
    np.testing.assert_array_equal(view_pages, block_to_page[view_blocks])
    stats = {"band_members": 0, "band_diffs": 0, "exact_rows": 0}
    lo, hi = n_sink, m - n_recent
    for s in range(n_sel):
        vb = view_blocks[s]
        assert vb[:n_sink].tolist() == list(range(n_sink))
        assert vb[n_sink + k_eff:].tolist() == list(range(hi, m))
        mid = vb[n_sink:n_sink + k_eff]
        assert np.all(np.diff(vb) > 0), "view is not strictly ascending"
        assert np.all((mid >= lo) & (mid < hi))
        if k_eff == 0 or k_eff == hi - lo:
            stats["exact_rows"] += 1
            continue
        r32 = relevance[s, lo:hi].astype(np.float32)
        rk = kth_score(r32, k_eff)
        assert rk > 1e-30, "k-th score underflows fp32; the band test would be meaningless"
        chosen = np.zeros(hi - lo, bool)
        chosen[mid - lo] = True
        must = r32.astype(np.float64) > rk * (1 + BAND)
        must_not = r32.astype(np.float64) < rk * (1 - BAND)
        missing = np.nonzero(must & ~chosen)[0]
        extra = np.nonzero(must_not & chosen)[0]
        assert missing.size == 0, f"row {s}: {missing.size} blocks above the band not selected, e.g. {missing[:5] + lo}"
        assert extra.size == 0, f"row {s}: {extra.size} blocks below the band selected, e.g. {extra[:5] + lo}"
        band = ~must & ~must_not
        stats["band_members"] += int(band.sum())
        if ref_view is not None:
            ref_chosen = np.zeros(hi - lo, bool)
            ref_chosen[ref_view[s, n_sink:n_sink + k_eff] - lo] = True
            diff = int((ref_chosen != chosen).sum())
            assert np.all((ref_chosen == chosen) | band)
            stats["band_diffs"] += diff
            stats["exact_rows"] += int(diff == 0)
    return stats


def check_scores(gpu_scores: np.ndarray, relevance: np.ndarray, n_sink: int, n_recent: int):
    m = relevance.shape[1]
    lo, hi = n_sink, m - n_recent
    assert np.all(np.isinf(gpu_scores[:, :lo])) and np.all(np.isinf(gpu_scores[:, hi:]))
    ref = relevance[:, lo:hi]
    got = gpu_scores[:, lo:hi].astype(np.float64)
    rel = np.abs(got - ref) / np.maximum(np.abs(ref), 1e-300)
    worst = float(rel.max())
    assert worst <= SCORE_RTOL, f"score relative error {worst:.3g} > {SCORE_RTOL}"
    return worst


def check_attention(out: np.ndarray, lse: np.ndarray, ref_out: np.ndarray, ref_lse: np.ndarray,
                    kv_dtype: str, regression: bool = True):
    """Contract bound, then (unless regression=False, for inputs far outside the
    workloads' value range) the regression bound."""
    atol = ATOL[kv_dtype]
    err = float(np.abs(out.astype(np.float64) - ref_out).max())
    lerr = float(np.abs(lse.astype(np.float64) - ref_lse).max())
    assert np.isfinite(out).all() and np.isfinite(lse).all()
    assert err <= atol, f"attention max abs error {err:.3g} > {atol}"
    assert lerr <= atol, f"lse max abs error {lerr:.3g} > {atol}"
    if regression:
        assert err <= REGRESSION_ATOL, f"attention max abs error {err:.3g} > regression bound {REGRESSION_ATOL}"
        assert lerr <= REGRESSION_ATOL, f"lse max abs error {lerr:.3g} > regression bound {REGRESSION_ATOL}"
    return err, lerr
