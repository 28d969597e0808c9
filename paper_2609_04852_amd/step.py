"""Device-resident state for the KVMem decode step, driven through the C ABI.

`LayerState` owns one layer's device buffers (K/V page pools, block table,
Mean-K index, view tables, outputs and both workspaces) and runs the three
library calls on a torch stream.  It only allocates and marshals; every
computation happens in libkvmem.so.
"""
from __future__ import annotations

import numpy as np
import torch

from . import kvmem as K
from .workload import MEAN_ALL, Config


def geom_of(cfg: Config) -> K.Geom:
    dt = {"f32": K.KVMEM_F32, "bf16": K.KVMEM_BF16, "fp8": K.KVMEM_FP8_E4M3}[cfg.kv_dtype]
    return K.Geom(cfg.n_kv_heads, cfg.n_q_heads, cfg.head_dim, cfg.block_tokens, dt,
                  cfg.kv_scale, cfg.kv_scale)


def mode_of(cfg: Config) -> int:
    return K.KVMEM_REDUCE_MEAN_ALL if cfg.mode == MEAN_ALL else K.KVMEM_REDUCE_MAX_GROUP


def pool_to_device(pool: np.ndarray, device) -> torch.Tensor:
    """Upload a host pool (float32, bf16 bits as uint16, or E4M3 codes as uint8)
    as float32 / bfloat16 / float8_e4m3fn."""
    if pool.dtype == np.uint8:
        return torch.from_numpy(pool).to(device).view(torch.float8_e4m3fn)
    if pool.dtype == np.uint16:
        return torch.from_numpy(pool.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(pool).to(device)


class LayerState:
    """One layer: pools, block table, index, and the buffers of select + attention."""

    def __init__(self, cfg: Config, k_pool: np.ndarray, v_pool: np.ndarray | None,
                 block_to_page: np.ndarray, device="cuda", n_sink: int | None = None,
                 n_recent: int | None = None, budget_tokens: int | None = None, n_q: int | None = None,
                 mode: int | None = None):
        self.cfg = cfg
        self.device = torch.device(device)
        self.geom = geom_of(cfg)
        self.n_sink = cfg.sink_blocks if n_sink is None else n_sink
        self.n_recent = cfg.n_recent if n_recent is None else n_recent
        self.budget = cfg.budget_tokens if budget_tokens is None else budget_tokens
        self.n_q = cfg.n_q if n_q is None else n_q
        self.mode = mode_of(cfg) if mode is None else mode
        self.k_pool = pool_to_device(k_pool, self.device)
        self.v_pool = pool_to_device(v_pool, self.device) if v_pool is not None else None
        self.block_to_page = torch.from_numpy(np.ascontiguousarray(block_to_page, np.int32)).to(self.device)
        self.n_blocks = int(block_to_page.shape[0])
        g = self.geom
        self.index = torch.empty(K.kvmem_index_bytes(g, self.n_blocks) // 4, dtype=torch.float32,
                                 device=self.device)
        self.k_eff, self.n_view = K.kvmem_plan_view(g, self.n_blocks, self.n_sink, self.n_recent,
                                                    self.budget, self.budget)
        self.n_sel = 1 if self.mode == K.KVMEM_REDUCE_MEAN_ALL else g.n_kv_heads
        self.view_blocks = torch.empty((self.n_sel, self.n_view), dtype=torch.int32, device=self.device)
        self.view_pages = torch.empty_like(self.view_blocks)
        self.scores = torch.empty((self.n_sel, self.n_blocks), dtype=torch.float32, device=self.device)
        try:
            ws = K.kvmem_select_workspace_bytes(g, 1, self.n_q, self.n_blocks, self.n_sink, self.n_recent,
                                                self.mode)
            self.select_ws = torch.empty(ws, dtype=torch.uint8, device=self.device)
        except K.KvmemError as e:  # attention-only use of a shape that selection does not take
            self.select_ws, self.select_error = None, e
        aws = K.kvmem_sparse_attn_workspace_bytes(g, self.n_q, self.n_sel, self.n_view)
        self.attn_ws = torch.empty(aws, dtype=torch.uint8, device=self.device)
        self.out = torch.empty((self.n_q, g.n_q_heads, g.head_dim), dtype=torch.float32, device=self.device)
        self.lse = torch.empty((self.n_q, g.n_q_heads), dtype=torch.float32, device=self.device)

    def index_rows(self) -> np.ndarray:
        """The index as a host [M][Hkv][d] array."""
        g = self.geom
        return K.index_rows(self.index.cpu().numpy(), self.n_blocks, g.n_kv_heads, g.head_dim).copy()

    def build_index(self, first_block: int = 0, n_blocks: int | None = None, stream=None):
        n = self.n_blocks - first_block if n_blocks is None else n_blocks
        K.kvmem_build_index(self.geom, self.k_pool, self.block_to_page, first_block, n, self.index,
                            stream)

    def select(self, q: torch.Tensor, with_scores: bool = True, stream=None) -> int:
        """q [1][n_q][Hq][d] (this layer).  Fills view_blocks/view_pages (and scores)."""
        if self.select_ws is None:
            raise self.select_error
        return K.kvmem_select(self.geom, q, self.index, self.n_blocks, self.n_sink, self.n_recent,
                              self.budget, self.budget, self.mode, 0.0, self.block_to_page,
                              self.view_blocks, self.view_pages, self.select_ws,
                              self.scores if with_scores else None, stream)

    def attend(self, q: torch.Tensor, view_pages: torch.Tensor | None = None,
               last_page_tokens: int | None = None, stream=None):
        """q [n_q][Hq][d].  Attention over view_pages (default: this layer's selection)."""
        vp = self.view_pages if view_pages is None else view_pages
        n_sel, n_view = vp.shape
        lpt = self.geom.block_tokens if last_page_tokens is None else last_page_tokens
        ws = self.attn_ws
        need = K.kvmem_sparse_attn_workspace_bytes(self.geom, q.shape[0], n_sel, n_view)
        if need > ws.numel():
            ws = torch.empty(need, dtype=torch.uint8, device=self.device)
        K.kvmem_sparse_attn(self.geom, q, self.k_pool, self.v_pool, vp, n_sel, n_view, lpt, 0.0,
                            self.out, ws, self.lse, stream)
        return self.out, self.lse

    def step(self, q_layer: torch.Tensor, stream=None):
        """One decode step of this layer: select, then attention over the view."""
        self.select(q_layer, with_scores=False, stream=stream)
        return self.attend(q_layer[0], stream=stream)


class RecallState:
    """A recall point (Sec. 4.2, Eq. 10): the Mean-K indexes of several layers in
    one buffer and one selection over all of them from a multi-token query."""

    def __init__(self, cfg: Config, k_pools: list, block_to_page: np.ndarray, device="cuda",
                 budget_tokens: int | None = None, n_q: int | None = None):
        self.cfg = cfg
        self.device = torch.device(device)
        self.geom = geom_of(cfg)
        g = self.geom
        self.n_layers = len(k_pools)
        self.n_q = cfg.n_q if n_q is None else n_q
        self.budget = cfg.budget_tokens if budget_tokens is None else budget_tokens
        self.mode = mode_of(cfg)
        self.block_to_page = torch.from_numpy(np.ascontiguousarray(block_to_page, np.int32)).to(self.device)
        self.n_blocks = int(block_to_page.shape[0])
        self.layer_floats = K.kvmem_index_bytes(g, self.n_blocks) // 4
        self.index = torch.empty(self.n_layers * self.layer_floats, dtype=torch.float32, device=self.device)
        self.k_pools = [pool_to_device(k, self.device) for k in k_pools]
        self.k_eff, self.n_view = K.kvmem_plan_view(g, self.n_blocks, cfg.sink_blocks, cfg.n_recent,
                                                    self.budget, self.budget)
        self.n_sel = 1 if self.mode == K.KVMEM_REDUCE_MEAN_ALL else self.n_layers * g.n_kv_heads
        self.view_blocks = torch.empty((self.n_sel, self.n_view), dtype=torch.int32, device=self.device)
        self.view_pages = torch.empty_like(self.view_blocks)
        self.scores = torch.empty((self.n_sel, self.n_blocks), dtype=torch.float32, device=self.device)
        ws = K.kvmem_select_workspace_bytes(g, self.n_layers, self.n_q, self.n_blocks, cfg.sink_blocks,
                                            cfg.n_recent, self.mode)
        self.select_ws = torch.empty(ws, dtype=torch.uint8, device=self.device)

    def layer_index(self, l: int) -> torch.Tensor:
        return self.index[l * self.layer_floats:(l + 1) * self.layer_floats]

    def build_index(self, stream=None):
        for l, kp in enumerate(self.k_pools):
            K.kvmem_build_index(self.geom, kp, self.block_to_page, 0, self.n_blocks, self.layer_index(l), stream)

    def index_rows(self, l: int) -> np.ndarray:
        g = self.geom
        return K.index_rows(self.layer_index(l).cpu().numpy(), self.n_blocks, g.n_kv_heads, g.head_dim).copy()

    def select(self, q: torch.Tensor, with_scores: bool = True, stream=None) -> int:
        """q [L][n_q][Hq][d]: the recall point's query over every layer."""
        return K.kvmem_select(self.geom, q, self.index, self.n_blocks, self.cfg.sink_blocks, self.cfg.n_recent,
                              self.budget, self.budget, self.mode, 0.0, self.block_to_page, self.view_blocks,
                              self.view_pages, self.select_ws, self.scores if with_scores else None, stream)
