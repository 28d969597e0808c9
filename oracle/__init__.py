"""CPU oracle for the KVMem per-decode-step path -- TEST INFRASTRUCTURE ONLY.

A plain fp64 C implementation (kvmem_oracle.c) of what the GPU path computes,
written from the paper (KVMem, arXiv 2609.04852), with this thin ctypes layer
that only marshals numpy arrays.  Only the tests, the smoke check and the
benchmark's CPU-baseline leg may import it; the HIP library never does, and
this package never imports the HIP library.

Entry points and the passages they follow:
  mean_k            Eq. 9  (Sec. 4.3, Mean-K retrieval-index construction)
  k_eff             Eq. 5, Eq. 7 (Sec. 3.1, active budget and view capacity)
  block_relevance   Eq. 10 (Sec. 4.3, query-conditioned block scoring)
  select            Sec. 4.3 selector (sink + recent reserved, top-k, chronological)
  view_attention    Sec. 4.4 / Sec. 5.3: attention through the view's page table
  masked_dense_attention   the same attention as dense attention with the
                    non-view blocks masked out
  working_set.WorkingSet   Eq. 11, Eq. 12 (Sec. 4.4): the working-set delta and
                    the physical loads of a recall point over a bounded page pool
  decode_e4m3, decode_fp8  FP8 K/V (the KV-cache precision of Sec. 6's
                    platforms): OCP E4M3 codes to fp64, times the pool's scale;
                    the entry points above take the decoded pool as float64
"""
import ctypes
import os

import numpy as np

MEAN_ALL = 0
MAX_GROUP = 1

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libkvmem_oracle.so")
_lib = None


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from .build import build_oracle
        build_oracle()
    lib = ctypes.CDLL(_LIB_PATH)
    P = ctypes.c_void_p
    i32, i64, dbl = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    ci = ctypes.c_int
    lib.oracle_mean_k.argtypes = [ci, ci, ci, ci, P, i64, P, i32, i32, P]
    lib.oracle_mean_k.restype = ci
    lib.oracle_k_eff.argtypes = [i64, i64, ci, i32, i32, i32]
    lib.oracle_k_eff.restype = i64
    lib.oracle_block_relevance.argtypes = [ci, ci, ci, ci, ci, P, P, i32, i32, i32, ci, dbl, P]
    lib.oracle_block_relevance.restype = ci
    lib.oracle_select.argtypes = [ci, P, i32, i32, i32, i64, P, P, P]
    lib.oracle_select.restype = ci
    lib.oracle_view_attention.argtypes = [ci, ci, ci, ci, ci, ci, P, P, P, i64, P, ci, i32, i32,
                                          dbl, P, P]
    lib.oracle_view_attention.restype = ci
    lib.oracle_masked_dense_attention.argtypes = [ci, ci, ci, ci, ci, ci, P, P, P, i64, P, i32, P,
                                                  ci, i32, i32, dbl, P, P]
    lib.oracle_masked_dense_attention.restype = ci
    lib.oracle_rope.argtypes = [i64, ci, P, P, dbl, P]
    lib.oracle_rope.restype = ci
    lib.oracle_mean_k_rope.argtypes = [ci, ci, ci, ci, P, i64, P, P, dbl, i32, i32, P]
    lib.oracle_mean_k_rope.restype = ci
    lib.oracle_num_threads.argtypes = []
    lib.oracle_num_threads.restype = ci
    _lib = lib
    return lib


def _c(a, dtype):
    a = np.ascontiguousarray(a)
    if a.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {a.dtype}")
    return a


def _pool(pool):
    """A K/V pool is float32, bf16 stored as raw uint16 bits, or float64 (an
    FP8 pool decoded by decode_fp8)."""
    pool = np.ascontiguousarray(pool)
    if pool.dtype == np.float32:
        return pool, 0
    if pool.dtype == np.uint16:
        return pool, 1
    if pool.dtype == np.float64:
        return pool, 2
    raise TypeError("pool must be float32, uint16 (bf16 bits) or float64")


def decode_e4m3(codes):
    """OCP FP8 E4M3 (the FN variant: 1 sign, 4 exponent bits with bias 7, 3
    mantissa bits, no infinities; S.1111.111 is NaN) to fp64:
      exponent field e > 0: (-1)^s * 2^(e-7) * (1 + m/8)
      exponent field 0:     (-1)^s * 2^(-6) * (m/8)"""
    c = np.asarray(codes, np.uint8).astype(np.int64)
    s = np.where(c >> 7, -1.0, 1.0)
    e = (c >> 3) & 15
    m = (c & 7).astype(np.float64)
    val = np.where(e > 0, np.ldexp(1.0 + m / 8.0, e - 7), np.ldexp(m / 8.0, -6))
    val = s * val
    return np.where((c & 0x7F) == 0x7F, np.nan, val)


def decode_fp8(codes, scale):
    """An FP8 K/V pool (E4M3 codes with one fp32 scale per pool) as fp64 values:
    decode_e4m3(code) * scale."""
    return decode_e4m3(codes) * float(np.float32(scale))


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what}: invalid arguments")


def num_threads() -> int:
    return _load().oracle_num_threads()


def mean_k(k_pool, block_to_page, first_block=0, n_blocks=None, index=None):
    """Eq. 9.  k_pool [P][Hkv][Bt][d]; returns/updates index [M][Hkv][d] float32."""
    k_pool, is_bf16 = _pool(k_pool)
    n_pages, hkv, bt, d = k_pool.shape
    b2p = _c(block_to_page, np.int32)
    m = b2p.shape[0]
    if n_blocks is None:
        n_blocks = m - first_block
    if index is None:
        index = np.zeros((m, hkv, d), np.float32)
    if index.dtype != np.float32 or not index.flags.c_contiguous or index.shape != (m, hkv, d):
        raise TypeError("index must be a C-contiguous float32 [M][Hkv][d] array")
    if first_block < 0 or n_blocks < 0 or first_block + n_blocks > m:
        raise ValueError("block range out of bounds")
    rc = _load().oracle_mean_k(hkv, bt, d, is_bf16, k_pool.ctypes.data, n_pages,
                               b2p.ctypes.data, first_block, n_blocks, index.ctypes.data)
    _check(rc, "mean_k")
    return index


def rope(x, pos, base):
    """RoPE, rotate-half form (Sec. 4.3 / 4.4 position handling): rows of x [..., d]
    rotated to positions pos (broadcast over the leading dims, any sign).  fp64."""
    x = np.asarray(x, np.float64)
    d = x.shape[-1]
    pos = np.broadcast_to(np.asarray(pos, np.int64), x.shape[:-1])
    xr = np.ascontiguousarray(x.reshape(-1, d))
    pr = np.ascontiguousarray(pos.reshape(-1))
    out = np.empty_like(xr)
    rc = _load().oracle_rope(xr.shape[0], d, xr.ctypes.data, pr.ctypes.data, float(base), out.ctypes.data)
    _check(rc, "rope")
    return out.reshape(x.shape)


def mean_k_rope(k_pool, block_to_page, base, block_pos=None, first_block=0, n_blocks=None, index=None):
    """Eq. 9 from keys that carry RoPE: token t of block b sits at block_pos[b] + t
    (None: b * Bt + t) and is rotated back before the mean.  Returns index [M][Hkv][d]."""
    k_pool, is_bf16 = _pool(k_pool)
    n_pages, hkv, bt, d = k_pool.shape
    b2p = _c(block_to_page, np.int32)
    m = b2p.shape[0]
    if n_blocks is None:
        n_blocks = m - first_block
    if index is None:
        index = np.zeros((m, hkv, d), np.float32)
    bp = None if block_pos is None else _c(np.asarray(block_pos, np.int64), np.int64)
    if bp is not None and bp.shape != (m,):
        raise ValueError("block_pos must have one entry per block")
    if first_block < 0 or n_blocks < 0 or first_block + n_blocks > m:
        raise ValueError("block range out of bounds")
    rc = _load().oracle_mean_k_rope(hkv, bt, d, is_bf16, k_pool.ctypes.data, n_pages, b2p.ctypes.data,
                                    None if bp is None else bp.ctypes.data, float(base), first_block,
                                    n_blocks, index.ctypes.data)
    _check(rc, "mean_k_rope")
    return index


def to_bf16_bits(x):
    """Round fp32 (or fp64 via fp32) values to bf16 bits, to nearest even (finite values)."""
    u = np.ascontiguousarray(np.asarray(x, np.float32)).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def from_bf16_bits(b):
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32)


def materialize(raw_k_pool, v_pool, src_pages, positions, base):
    """Execution-view materialisation (Sec. 4.4, Sec. 5.3): block i takes page
    src_pages[i] of the position-independent K pool; its token t is re-encoded at
    positions[i] + t.  Returns (K [n][Hkv][Bt][d] fp64, V [n][Hkv][Bt][d] as stored)."""
    raw, _ = _pool(raw_k_pool)
    vp, _ = _pool(v_pool)
    src = np.asarray(src_pages, np.int64)
    k = raw[src].astype(np.float64) if raw.dtype == np.float32 else from_bf16_bits(raw[src]).astype(np.float64)
    bt = raw.shape[2]
    pos = np.asarray(positions, np.int64)[:, None, None] + np.arange(bt)[None, None, :]
    pos = np.broadcast_to(pos, k.shape[:-1])
    return rope(k, pos, base), vp[src].copy()


def k_eff(model_ctx_tokens, gpu_kv_tokens, block_tokens, n_blocks, n_sink, n_recent):
    """Eq. 5 / Eq. 7.  Returns k_eff, or raises when the budget cannot hold the mandatory context."""
    k = _load().oracle_k_eff(int(model_ctx_tokens), int(gpu_kv_tokens), int(block_tokens),
                             int(n_blocks), int(n_sink), int(n_recent))
    if k < 0:
        raise ValueError("budget below the mandatory sink+recent context, or bad shape")
    return int(k)


def block_relevance(q, index, n_sink, n_recent, mode=MEAN_ALL, scale=0.0):
    """Eq. 10.  q [L][n_q][Hq][d] float32, index [L][M][Hkv][d] float32.

    Returns R float64 [n_sel][M] (n_sel = 1 for MEAN_ALL, L*Hkv for MAX_GROUP);
    reserved blocks hold +inf."""
    q = _c(q, np.float32)
    index = _c(index, np.float32)
    if q.ndim != 4 or index.ndim != 4 or q.shape[0] != index.shape[0] or q.shape[3] != index.shape[3]:
        raise ValueError("q must be [L][n_q][Hq][d] and index [L][M][Hkv][d]")
    L, nq, hq, d = q.shape
    _, m, hkv, _ = index.shape
    n_sel = 1 if mode == MEAN_ALL else L * hkv
    out = np.empty((n_sel, m), np.float64)
    rc = _load().oracle_block_relevance(L, nq, hq, hkv, d, q.ctypes.data, index.ctypes.data, m,
                                        n_sink, n_recent, mode, float(scale), out.ctypes.data)
    _check(rc, "block_relevance")
    return out


def select(relevance, n_sink, n_recent, k, block_to_page):
    """Selector.  relevance [n_sel][M] float64 -> (view_blocks, view_pages) int32 [n_sel][n_view]."""
    r = _c(relevance, np.float64)
    if r.ndim == 1:
        r = r[None, :]
    n_sel, m = r.shape
    b2p = _c(block_to_page, np.int32)
    if b2p.shape[0] != m:
        raise ValueError("block_to_page length must equal the number of blocks")
    n_view = n_sink + k + n_recent
    vb = np.empty((n_sel, n_view), np.int32)
    vp = np.empty((n_sel, n_view), np.int32)
    rc = _load().oracle_select(n_sel, r.ctypes.data, m, n_sink, n_recent, int(k), b2p.ctypes.data,
                               vb.ctypes.data, vp.ctypes.data)
    _check(rc, "select")
    return vb, vp


def view_attention(q, k_pool, v_pool, view_pages, last_page_tokens=None, scale=0.0):
    """Attention through the page table.  q [n_q][Hq][d] float32 (one layer);
    pools [P][Hkv][Bt][d]; view_pages [n_sel][n_view].  Returns (out, lse) float64."""
    q = _c(q, np.float32)
    k_pool, kb = _pool(k_pool)
    v_pool, vb = _pool(v_pool)
    if kb != vb or k_pool.shape != v_pool.shape:
        raise ValueError("K and V pools must match in shape and dtype")
    n_pages, hkv, bt, d = k_pool.shape
    vp = _c(view_pages, np.int32)
    if vp.ndim == 1:
        vp = vp[None, :]
    n_sel, n_view = vp.shape
    nq, hq, dq = q.shape
    if dq != d:
        raise ValueError("head_dim mismatch")
    lpt = bt if last_page_tokens is None else int(last_page_tokens)
    out = np.empty((nq, hq, d), np.float64)
    lse = np.empty((nq, hq), np.float64)
    rc = _load().oracle_view_attention(nq, hq, hkv, d, bt, kb, q.ctypes.data, k_pool.ctypes.data,
                                       v_pool.ctypes.data, n_pages, vp.ctypes.data, n_sel, n_view,
                                       lpt, float(scale), out.ctypes.data, lse.ctypes.data)
    _check(rc, "view_attention")
    return out, lse


def masked_dense_attention(q, k_pool, v_pool, block_to_page, view_blocks, last_page_tokens=None,
                           scale=0.0):
    """Dense attention over all M blocks with non-view blocks masked.  Returns (out, lse) float64."""
    q = _c(q, np.float32)
    k_pool, kb = _pool(k_pool)
    v_pool, vb = _pool(v_pool)
    if kb != vb or k_pool.shape != v_pool.shape:
        raise ValueError("K and V pools must match in shape and dtype")
    n_pages, hkv, bt, d = k_pool.shape
    b2p = _c(block_to_page, np.int32)
    vbl = _c(view_blocks, np.int32)
    if vbl.ndim == 1:
        vbl = vbl[None, :]
    n_sel, n_view = vbl.shape
    nq, hq, _ = q.shape
    lpt = bt if last_page_tokens is None else int(last_page_tokens)
    out = np.empty((nq, hq, d), np.float64)
    lse = np.empty((nq, hq), np.float64)
    rc = _load().oracle_masked_dense_attention(nq, hq, hkv, d, bt, kb, q.ctypes.data,
                                               k_pool.ctypes.data, v_pool.ctypes.data, n_pages,
                                               b2p.ctypes.data, b2p.shape[0], vbl.ctypes.data,
                                               n_sel, n_view, lpt, float(scale), out.ctypes.data,
                                               lse.ctypes.data)
    _check(rc, "masked_dense_attention")
    return out, lse
