"""Python binding of the KVMem C ABI (libkvmem.so): argument marshalling only.

Each function has the name of the C entry point it calls and takes torch
tensors for device buffers; every step of the computation runs in the HIP
kernels behind the C ABI.  The library is loaded on first use and an
ImportError is raised if it has not been built -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import re

import torch

KVMEM_OK = 0
KVMEM_F32, KVMEM_BF16, KVMEM_FP8_E4M3 = 0, 1, 2
KVMEM_REDUCE_MEAN_ALL, KVMEM_REDUCE_MAX_GROUP = 0, 1

STATUS_NAMES = {
    0: "KVMEM_OK", -1: "KVMEM_ERR_NULL", -2: "KVMEM_ERR_SHAPE", -3: "KVMEM_ERR_DTYPE",
    -4: "KVMEM_ERR_UNSUPPORTED", -5: "KVMEM_ERR_BUDGET", -6: "KVMEM_ERR_WORKSPACE",
    -7: "KVMEM_ERR_ALIGN", -8: "KVMEM_ERR_HIP",
}

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkvmem.so")
HEADER_PATH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                           "include", "kvmem.h")


class KvmemError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


class kvmem_geom(ctypes.Structure):
    _fields_ = [("n_kv_heads", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("block_tokens", ctypes.c_int32),
                ("kv_dtype", ctypes.c_int32), ("k_scale", ctypes.c_float), ("v_scale", ctypes.c_float)]


@dataclasses.dataclass(frozen=True)
class Geom:
    n_kv_heads: int
    n_q_heads: int
    head_dim: int
    block_tokens: int
    kv_dtype: int  # KVMEM_F32, KVMEM_BF16 or KVMEM_FP8_E4M3
    k_scale: float = 1.0  # FP8 pools: K = decoded code * k_scale
    v_scale: float = 1.0  # FP8 pools: V = decoded code * v_scale

    def c(self) -> kvmem_geom:
        return kvmem_geom(self.n_kv_heads, self.n_q_heads, self.head_dim, self.block_tokens,
                          self.kv_dtype, self.k_scale, self.v_scale)


class kvmem_working_set(ctypes.Structure):
    _fields_ = [("n_blocks", ctypes.c_int32), ("n_pages", ctypes.c_int32),
                ("block_page", ctypes.c_void_p), ("block_last_step", ctypes.c_void_p),
                ("page_block", ctypes.c_void_p), ("page_pos", ctypes.c_void_p),
                ("page_deltas", ctypes.c_void_p), ("header", ctypes.c_void_p)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libkvmem.so (raises ImportError if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2609_04852_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, G = ctypes.c_void_p, ctypes.POINTER(kvmem_geom)
    i32, i64, f32, sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
    pi32 = ctypes.POINTER(ctypes.c_int32)
    L.kvmem_index_bytes.argtypes = [G, i32]
    L.kvmem_index_bytes.restype = sz
    L.kvmem_build_index.argtypes = [G, P, i64, P, i32, i32, P, P]
    L.kvmem_plan_view.argtypes = [G, i32, i32, i32, i64, i64, pi32, pi32]
    L.kvmem_select_workspace_bytes.argtypes = [G, i32, i32, i32, i32, i32, i32]
    L.kvmem_select_workspace_bytes.restype = sz
    L.kvmem_select.argtypes = [G, i32, P, i32, P, i32, i32, i32, i64, i64, i32, f32, P, P, P, P,
                               pi32, P, sz, P]
    L.kvmem_select_noalloc.argtypes = [G, i32, P, i32, P, i32, i32, i32, i64, i64, i32, f32, P, P, P, P,
                                       pi32, P]
    L.kvmem_sparse_attn_workspace_bytes.argtypes = [G, i32, i32, i32]
    L.kvmem_sparse_attn_workspace_bytes.restype = sz
    L.kvmem_sparse_attn.argtypes = [G, P, i32, P, P, i64, P, i32, i32, i32, f32, P, P, P, sz, P]
    dbl = ctypes.c_double
    L.kvmem_build_index_rope.argtypes = [G, P, i64, P, P, dbl, i32, i32, P, P]
    L.kvmem_materialize.argtypes = [G, dbl, P, P, i64, P, P, P, i32, P, P, i64, P]
    L.kvmem_rerope.argtypes = [G, dbl, P, i64, P, P, i32, P]
    W = ctypes.POINTER(kvmem_working_set)
    L.kvmem_working_set_reset.argtypes = [W, P]
    L.kvmem_working_set_workspace_bytes.argtypes = [i32, i32]
    L.kvmem_working_set_workspace_bytes.restype = sz
    L.kvmem_working_set_update.argtypes = [G, dbl, W, i32, P, i32, i64, i32, P, P, P, i64, P, P, P, P, P, sz, P]
    for name in ("kvmem_build_index", "kvmem_plan_view", "kvmem_select", "kvmem_select_noalloc", "kvmem_sparse_attn",
                 "kvmem_build_index_rope", "kvmem_materialize", "kvmem_rerope", "kvmem_working_set_reset",
                 "kvmem_working_set_update"):
        getattr(L, name).restype = ctypes.c_int
    L.kvmem_last_error.argtypes = []
    L.kvmem_last_error.restype = ctypes.c_char_p
    _lib = L
    return L


def header_functions() -> list[str]:
    """Names of the functions declared in include/kvmem.h."""
    text = open(HEADER_PATH).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(kvmem_\w+)\s*\(", text, re.M)))


def kvmem_last_error() -> str:
    return lib().kvmem_last_error().decode()


def _check(status: int):
    if status != KVMEM_OK:
        raise KvmemError(status, kvmem_last_error())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def kv_dtype_of(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return KVMEM_BF16
    if t.dtype == torch.float32:
        return KVMEM_F32
    if t.dtype in (torch.float8_e4m3fn, torch.uint8):  # FP8 E4M3 codes
        return KVMEM_FP8_E4M3
    raise TypeError(f"K/V pools must be bfloat16, float32 or float8_e4m3fn (or uint8 codes), got {t.dtype}")


def _need(t: torch.Tensor, dtype, name: str):
    if t.dtype != dtype or not t.is_contiguous() or not t.is_cuda:
        raise TypeError(f"{name} must be a contiguous CUDA {dtype} tensor")


INDEX_TILE = 64


def kvmem_index_bytes(geom: Geom, n_blocks: int) -> int:
    n = lib().kvmem_index_bytes(ctypes.byref(geom.c()), n_blocks)
    if n == 0 and n_blocks > 0:
        raise KvmemError(-2, kvmem_last_error())
    return n


def index_rows(index, n_blocks: int, n_kv_heads: int, head_dim: int):
    """One layer of the tiled Mean-K index ([T][Hkv][d/4][64][4], torch or
    numpy) as a [n_blocks][Hkv][d] array (a layout change only)."""
    t = -(-n_blocks // INDEX_TILE)
    x = index.reshape(-1)[: t * INDEX_TILE * n_kv_heads * head_dim]
    x = x.reshape(t, n_kv_heads, head_dim // 4, INDEX_TILE, 4)
    x = x.permute(0, 3, 1, 2, 4) if isinstance(x, torch.Tensor) else x.transpose(0, 3, 1, 2, 4)
    return x.reshape(t * INDEX_TILE, n_kv_heads, head_dim)[:n_blocks]


def kvmem_build_index(geom: Geom, k_pool: torch.Tensor, block_to_page: torch.Tensor,
                      first_block: int, n_blocks: int, index: torch.Tensor, stream=None):
    _need(block_to_page, torch.int32, "block_to_page")
    _need(index, torch.float32, "index")
    if not k_pool.is_cuda or not k_pool.is_contiguous():
        raise TypeError("k_pool must be a contiguous CUDA tensor")
    if block_to_page.numel() < first_block + n_blocks:
        raise ValueError("block_to_page is shorter than the block range")
    if index.numel() * 4 < kvmem_index_bytes(geom, first_block + n_blocks):
        raise ValueError("index is smaller than the block range needs")
    n_pages = k_pool.numel() // (geom.n_kv_heads * geom.block_tokens * geom.head_dim)
    _check(lib().kvmem_build_index(ctypes.byref(geom.c()), _ptr(k_pool), n_pages,
                                   _ptr(block_to_page), first_block, n_blocks, _ptr(index),
                                   _stream(stream)))


def kvmem_plan_view(geom: Geom, n_blocks: int, n_sink: int, n_recent: int,
                    model_ctx_tokens: int, gpu_kv_tokens: int) -> tuple[int, int]:
    k = ctypes.c_int32()
    n = ctypes.c_int32()
    _check(lib().kvmem_plan_view(ctypes.byref(geom.c()), n_blocks, n_sink, n_recent,
                                 model_ctx_tokens, gpu_kv_tokens, ctypes.byref(k), ctypes.byref(n)))
    return k.value, n.value


def kvmem_select_workspace_bytes(geom: Geom, n_layers: int, n_q: int, n_blocks: int, n_sink: int,
                                 n_recent: int, mode: int) -> int:
    n = lib().kvmem_select_workspace_bytes(ctypes.byref(geom.c()), n_layers, n_q, n_blocks, n_sink,
                                           n_recent, mode)
    if n == 0:
        raise KvmemError(-2, kvmem_last_error())
    return n


def kvmem_select(geom: Geom, q: torch.Tensor, index: torch.Tensor, n_blocks: int, n_sink: int,
                 n_recent: int, model_ctx_tokens: int, gpu_kv_tokens: int, mode: int, scale: float,
                 block_to_page: torch.Tensor, view_blocks: torch.Tensor, view_pages: torch.Tensor,
                 workspace: torch.Tensor, scores: torch.Tensor | None = None, stream=None) -> int:
    """q [L][n_q][Hq][d] float32; index: L tiled layers (see kvmem_index_bytes).  Returns n_view."""
    _need(q, torch.float32, "q")
    _need(index, torch.float32, "index")
    _need(block_to_page, torch.int32, "block_to_page")
    _need(view_blocks, torch.int32, "view_blocks")
    _need(view_pages, torch.int32, "view_pages")
    _need(workspace, torch.uint8, "workspace")
    if q.dim() != 4 or tuple(q.shape[2:]) != (geom.n_q_heads, geom.head_dim):
        raise ValueError("q must be [L][n_q][Hq][d]")
    n_layers, n_q = q.shape[0], q.shape[1]
    if index.numel() * 4 < n_layers * kvmem_index_bytes(geom, n_blocks):
        raise ValueError("index is smaller than n_layers tiled layers of n_blocks blocks")
    if block_to_page.numel() != n_blocks:
        raise ValueError("block_to_page must have one entry per block")
    k_eff, n_view = kvmem_plan_view(geom, n_blocks, n_sink, n_recent, model_ctx_tokens, gpu_kv_tokens)
    n_sel = 1 if mode == KVMEM_REDUCE_MEAN_ALL else n_layers * geom.n_kv_heads
    if view_blocks.numel() < n_sel * n_view or view_pages.numel() < n_sel * n_view:
        raise ValueError("view tables are smaller than n_sel * n_view")
    if scores is not None:
        _need(scores, torch.float32, "scores")
        if scores.numel() < n_sel * n_blocks:
            raise ValueError("scores is smaller than n_sel * n_blocks")
    out_n = ctypes.c_int32()
    _check(lib().kvmem_select(ctypes.byref(geom.c()), n_layers, _ptr(q), n_q, _ptr(index), n_blocks,
                              n_sink, n_recent, model_ctx_tokens, gpu_kv_tokens, mode, scale,
                              _ptr(block_to_page), _ptr(view_blocks), _ptr(view_pages), _ptr(scores),
                              ctypes.byref(out_n), _ptr(workspace), workspace.numel(),
                              _stream(stream)))
    return out_n.value


SELECT_NOALLOC_MAX_BYTES = 16 << 20  # KVMEM_SELECT_NOALLOC_MAX_BYTES


def kvmem_select_noalloc(geom: Geom, q: torch.Tensor, index: torch.Tensor, n_blocks: int, n_sink: int,
                         n_recent: int, model_ctx_tokens: int, gpu_kv_tokens: int, mode: int, scale: float,
                         block_to_page: torch.Tensor, view_blocks: torch.Tensor, view_pages: torch.Tensor,
                         scores: torch.Tensor | None = None, stream=None) -> int:
    """kvmem_select with the library's own device scratch instead of a workspace
    (no allocation around the call).  Returns n_view."""
    _need(q, torch.float32, "q")
    _need(index, torch.float32, "index")
    _need(block_to_page, torch.int32, "block_to_page")
    _need(view_blocks, torch.int32, "view_blocks")
    _need(view_pages, torch.int32, "view_pages")
    if q.dim() != 4 or tuple(q.shape[2:]) != (geom.n_q_heads, geom.head_dim):
        raise ValueError("q must be [L][n_q][Hq][d]")
    n_layers, n_q = q.shape[0], q.shape[1]
    if index.numel() * 4 < n_layers * kvmem_index_bytes(geom, n_blocks):
        raise ValueError("index is smaller than n_layers tiled layers of n_blocks blocks")
    if block_to_page.numel() != n_blocks:
        raise ValueError("block_to_page must have one entry per block")
    k_eff, n_view = kvmem_plan_view(geom, n_blocks, n_sink, n_recent, model_ctx_tokens, gpu_kv_tokens)
    n_sel = 1 if mode == KVMEM_REDUCE_MEAN_ALL else n_layers * geom.n_kv_heads
    if view_blocks.numel() < n_sel * n_view or view_pages.numel() < n_sel * n_view:
        raise ValueError("view tables are smaller than n_sel * n_view")
    if scores is not None:
        _need(scores, torch.float32, "scores")
        if scores.numel() < n_sel * n_blocks:
            raise ValueError("scores is smaller than n_sel * n_blocks")
    out_n = ctypes.c_int32()
    _check(lib().kvmem_select_noalloc(ctypes.byref(geom.c()), n_layers, _ptr(q), n_q, _ptr(index), n_blocks,
                                      n_sink, n_recent, model_ctx_tokens, gpu_kv_tokens, mode, scale,
                                      _ptr(block_to_page), _ptr(view_blocks), _ptr(view_pages), _ptr(scores),
                                      ctypes.byref(out_n), _stream(stream)))
    return out_n.value


def kvmem_sparse_attn_workspace_bytes(geom: Geom, n_q: int, n_sel: int, n_view: int) -> int:
    n = lib().kvmem_sparse_attn_workspace_bytes(ctypes.byref(geom.c()), n_q, n_sel, n_view)
    if n == 0:
        raise KvmemError(-2, kvmem_last_error())
    return n


def kvmem_sparse_attn(geom: Geom, q: torch.Tensor, k_pool: torch.Tensor, v_pool: torch.Tensor,
                      view_pages: torch.Tensor, n_sel: int, n_view: int, last_page_tokens: int,
                      scale: float, out: torch.Tensor, workspace: torch.Tensor,
                      lse: torch.Tensor | None = None, stream=None):
    """q [n_q][Hq][d] float32 (one layer); view_pages [n_sel][n_view] int32."""
    _need(q, torch.float32, "q")
    _need(out, torch.float32, "out")
    _need(view_pages, torch.int32, "view_pages")
    _need(workspace, torch.uint8, "workspace")
    if k_pool.dtype != v_pool.dtype or k_pool.shape != v_pool.shape:
        raise ValueError("K and V pools must match in dtype and shape")
    if kv_dtype_of(k_pool) != geom.kv_dtype:
        raise TypeError("pool dtype does not match geom.kv_dtype")
    if not (k_pool.is_cuda and v_pool.is_cuda and k_pool.is_contiguous() and v_pool.is_contiguous()):
        raise TypeError("pools must be contiguous CUDA tensors")
    if q.dim() != 3 or tuple(q.shape[1:]) != (geom.n_q_heads, geom.head_dim):
        raise ValueError("q must be [n_q][Hq][d]")
    n_q = q.shape[0]
    if out.numel() != q.numel():
        raise ValueError("out must have the shape of q")
    if view_pages.numel() < n_sel * n_view:
        raise ValueError("view_pages is smaller than n_sel * n_view")
    if lse is not None:
        _need(lse, torch.float32, "lse")
        if lse.numel() < n_q * geom.n_q_heads:
            raise ValueError("lse is smaller than n_q * Hq")
    n_pages = k_pool.numel() // (geom.n_kv_heads * geom.block_tokens * geom.head_dim)
    _check(lib().kvmem_sparse_attn(ctypes.byref(geom.c()), _ptr(q), n_q, _ptr(k_pool), _ptr(v_pool),
                                   n_pages, _ptr(view_pages), n_sel, n_view, last_page_tokens, scale,
                                   _ptr(out), _ptr(lse), _ptr(workspace), workspace.numel(),
                                   _stream(stream)))


def kvmem_build_index_rope(geom: Geom, k_pool: torch.Tensor, block_to_page: torch.Tensor,
                           first_block: int, n_blocks: int, index: torch.Tensor, rope_base: float,
                           block_pos: torch.Tensor | None = None, stream=None):
    """kvmem_build_index for keys that carry RoPE: token t of block b sits at
    block_pos[b] + t (None: b * Bt + t) and is turned back before the mean."""
    _need(block_to_page, torch.int32, "block_to_page")
    _need(index, torch.float32, "index")
    if block_pos is not None:
        _need(block_pos, torch.int64, "block_pos")
        if block_pos.numel() < first_block + n_blocks:
            raise ValueError("block_pos is shorter than the block range")
    if not k_pool.is_cuda or not k_pool.is_contiguous():
        raise TypeError("k_pool must be a contiguous CUDA tensor")
    if block_to_page.numel() < first_block + n_blocks:
        raise ValueError("block_to_page is shorter than the block range")
    if index.numel() * 4 < kvmem_index_bytes(geom, first_block + n_blocks):
        raise ValueError("index is smaller than the block range needs")
    n_pages = k_pool.numel() // (geom.n_kv_heads * geom.block_tokens * geom.head_dim)
    _check(lib().kvmem_build_index_rope(ctypes.byref(geom.c()), _ptr(k_pool), n_pages, _ptr(block_to_page),
                                        _ptr(block_pos), float(rope_base), first_block, n_blocks, _ptr(index),
                                        _stream(stream)))


def kvmem_materialize(geom: Geom, rope_base: float, raw_k_pool: torch.Tensor, v_pool: torch.Tensor,
                      src_pages: torch.Tensor, positions: torch.Tensor, dst_pages: torch.Tensor,
                      k_dst_pool: torch.Tensor, v_dst_pool: torch.Tensor, stream=None):
    """Re-encode the keys of src_pages at positions[i] + t into dst_pages; copy V."""
    for t, name in ((raw_k_pool, "raw_k_pool"), (v_pool, "v_pool"), (k_dst_pool, "k_dst_pool"),
                    (v_dst_pool, "v_dst_pool")):
        if kv_dtype_of(t) != geom.kv_dtype or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous pool of geom.kv_dtype")
    _need(src_pages, torch.int32, "src_pages")
    _need(dst_pages, torch.int32, "dst_pages")
    _need(positions, torch.int64, "positions")
    n = src_pages.numel()
    if dst_pages.numel() != n or positions.numel() != n:
        raise ValueError("src_pages, dst_pages and positions must have the same length")
    _check(lib().kvmem_materialize(ctypes.byref(geom.c()), float(rope_base), _ptr(raw_k_pool), _ptr(v_pool),
                                   raw_k_pool.shape[0], _ptr(src_pages), _ptr(positions), _ptr(dst_pages), n,
                                   _ptr(k_dst_pool), _ptr(v_dst_pool), k_dst_pool.shape[0], _stream(stream)))


def kvmem_rerope(geom: Geom, rope_base: float, k_pool: torch.Tensor, pages: torch.Tensor,
                 delta_positions: torch.Tensor, stream=None):
    """Turn the keys of `pages` in place by delta_positions[i] positions."""
    if kv_dtype_of(k_pool) != geom.kv_dtype or not k_pool.is_contiguous():
        raise TypeError("k_pool must be a contiguous pool of geom.kv_dtype")
    _need(pages, torch.int32, "pages")
    _need(delta_positions, torch.int64, "delta_positions")
    if delta_positions.numel() != pages.numel():
        raise ValueError("pages and delta_positions must have the same length")
    _check(lib().kvmem_rerope(ctypes.byref(geom.c()), float(rope_base), _ptr(k_pool), k_pool.shape[0],
                              _ptr(pages), _ptr(delta_positions), pages.numel(), _stream(stream)))


class WorkingSetArrays:
    """The repository view of an execution pool of n_pages pages (kvmem_working_set):
    caller-owned device arrays, emptied by reset()."""

    def __init__(self, n_blocks: int, n_pages: int, device="cuda"):
        dev = torch.device(device)
        self.n_blocks, self.n_pages = int(n_blocks), int(n_pages)
        self.block_page = torch.empty(n_blocks, dtype=torch.int32, device=dev)
        self.block_last_step = torch.empty(n_blocks, dtype=torch.int32, device=dev)
        self.page_block = torch.empty(n_pages, dtype=torch.int32, device=dev)
        self.page_pos = torch.empty(n_pages, dtype=torch.int64, device=dev)
        self.page_deltas = torch.empty(n_pages, dtype=torch.int32, device=dev)
        self.header = torch.empty(8, dtype=torch.int32, device=dev)

    def c(self) -> kvmem_working_set:
        return kvmem_working_set(self.n_blocks, self.n_pages, self.block_page.data_ptr(),
                                 self.block_last_step.data_ptr(), self.page_block.data_ptr(),
                                 self.page_pos.data_ptr(), self.page_deltas.data_ptr(), self.header.data_ptr())

    def reset(self, stream=None):
        _check(lib().kvmem_working_set_reset(ctypes.byref(self.c()), _stream(stream)))


def kvmem_working_set_workspace_bytes(n_view: int, n_pages: int) -> int:
    n = lib().kvmem_working_set_workspace_bytes(n_view, n_pages)
    if n == 0:
        raise KvmemError(-2, kvmem_last_error())
    return n


def kvmem_working_set_update(geom: Geom, rope_base: float, ws: WorkingSetArrays, step: int,
                             view_blocks: torch.Tensor, first_position: int, max_deltas: int,
                             block_to_page: torch.Tensor, raw_k_pool: torch.Tensor, v_pool: torch.Tensor,
                             k_exec_pool: torch.Tensor, v_exec_pool: torch.Tensor, exec_pages: torch.Tensor,
                             counts: torch.Tensor, workspace: torch.Tensor, stream=None):
    """One recall point's working-set update (Eq. 11, Eq. 12); see kvmem.h."""
    for t, name in ((view_blocks, "view_blocks"), (block_to_page, "block_to_page"), (exec_pages, "exec_pages"),
                    (counts, "counts")):
        _need(t, torch.int32, name)
    _need(workspace, torch.uint8, "workspace")
    for t, name in ((raw_k_pool, "raw_k_pool"), (v_pool, "v_pool"), (k_exec_pool, "k_exec_pool"),
                    (v_exec_pool, "v_exec_pool")):
        if kv_dtype_of(t) != geom.kv_dtype or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous pool of geom.kv_dtype")
    if k_exec_pool.shape[0] != ws.n_pages or v_exec_pool.shape != k_exec_pool.shape:
        raise ValueError("the execution pools must have ws.n_pages pages")
    n_view = view_blocks.numel()
    if exec_pages.numel() < n_view or counts.numel() < 16:
        raise ValueError("exec_pages needs n_view entries and counts 16")
    _check(lib().kvmem_working_set_update(ctypes.byref(geom.c()), float(rope_base), ctypes.byref(ws.c()), step,
                                          _ptr(view_blocks), n_view, first_position, max_deltas,
                                          _ptr(block_to_page), _ptr(raw_k_pool), _ptr(v_pool), raw_k_pool.shape[0],
                                          _ptr(k_exec_pool), _ptr(v_exec_pool), _ptr(exec_pages), _ptr(counts),
                                          _ptr(workspace), workspace.numel(), _stream(stream)))
