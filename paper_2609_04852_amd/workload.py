"""Seeded synthetic inputs for the KVMem decode-step path.

This module only draws random inputs; it holds none of the method's
arithmetic (no Mean-K, no scoring, no selection, no attention).  Both the CPU
oracle (tests) and the HIP path read the same arrays produced here.

The paper evaluates on long agent histories (LongMemEval-S ~115K tokens,
MemoryAgentBench 103K-1.44M, AgentLongBench 32K-4M; Sec. 6.1) with bounded
execution views (32K-100K tokens; 64K in the Table 4 scalability study).  No
such data is available here, so synthetic paged K/V of the same shapes stands
in for them:

* offset configs (tiny, 64K, 256K, 1M): every (page, KV head) gets an offset
  o ~ N(0, 0.5^2 I_d); token vectors are z + o with z ~ N(0, I_d); K and V are
  drawn independently.  A few "planted" blocks have keys aligned with the
  group's mean query: key = sqrt(d) * (0.9 u + sqrt(0.19) nu), where u is the
  unit mean of the group's query vectors and nu a random unit vector orthogonal
  to u (cosine 0.9 with u).
* mixture config (4 layers x 1M, 64-token blocks, 4 query tokens): per (layer,
  KV head) 256 centres mu_j ~ N(0, 2^2 I_d); every page draws a centre index
  j ~ Zipf(1.1) truncated to 256 (P(j) proportional to (j+1)^-1.1), and its keys
  are mu_j + N(0, I_d).  This gives heavy-tailed block scores: about 2/3 of a
  head's block-softmax mass lies in the top 7.8 % of blocks, in line with the
  sparsity the paper reports (Sec. 4.3: top-8 of ~103 blocks hold 66.5 %).
* queries: per (layer, KV head) a direction u_g ~ N(0, I_d); query head h of
  group g at token m is u_g + 0.5 eps, eps ~ N(0, I_d); stored fp32.
* the block -> page map is a seeded random permutation of [0, M), so page
  gathers are scattered; pools hold exactly M pages.

bf16 values are produced from fp32 draws by round-to-nearest-even and kept as
raw uint16 bit patterns.  FP8 pools (the KV-cache precision of the paper's
evaluation platforms, Sec. 6) hold OCP E4M3 codes of x / kv_scale, rounded to
nearest even and saturated at +-448, with one static scale per pool:
kv_scale = 8/448 for the offset configs (|x| up to 8, about 7 standard
deviations) and 16/448 for the mixture.  All draws come from numpy's PCG64 with one
SeedSequence child per independent chunk, so results do not depend on the
number of worker threads.
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os

import numpy as np

MEAN_ALL = "mean_all"
MAX_GROUP = "max_group"


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    description: str
    n_layers: int
    n_kv_heads: int
    n_q_heads: int
    head_dim: int
    kv_dtype: str  # "f32", "bf16" or "fp8" (E4M3 codes times kv_scale)
    history_tokens: int
    block_tokens: int
    recent_tokens: int
    sink_blocks: int
    budget_tokens: int
    n_q: int
    mode: str
    n_planted: int
    kind: str  # "offset" or "mixture"
    seed: int
    top_k: int  # the stated number of selectable historical blocks
    kv_scale: float = 1.0  # fp8: the static scale of every K and V pool

    @property
    def n_blocks(self) -> int:
        return self.history_tokens // self.block_tokens

    @property
    def n_recent(self) -> int:
        return self.recent_tokens // self.block_tokens

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def n_candidates(self) -> int:
        return self.n_blocks - self.sink_blocks - self.n_recent

    @property
    def n_view(self) -> int:
        return self.sink_blocks + self.top_k + self.n_recent

    @property
    def n_sel(self) -> int:
        """Selections per call for one layer: 1 shared, or one per KV head."""
        return 1 if self.mode == MEAN_ALL else self.n_kv_heads

    @property
    def elem_bytes(self) -> int:
        return {"f32": 4, "bf16": 2, "fp8": 1}[self.kv_dtype]

    def replace(self, **kw) -> "Config":
        return dataclasses.replace(self, **kw)


CONFIGS = {
    "tiny": Config("tiny", "1 layer, 1x4 GQA, d64, fp32 K/V, 4,096-token history in 16-token "
                   "blocks, top-k 32 + 64 recent tokens, 1 query", 1, 1, 4, 64, "f32", 4096, 16, 64,
                   0, 576, 1, MEAN_ALL, 3, "offset", 0, 32),
    "64k": Config("64k", "1 layer, 8x4 GQA, d128, bf16 K/V, 65,536-token history in 16-token "
                  "blocks, budget 8,192 tokens (top-k 448 + 1,024 recent)", 1, 8, 32, 128, "bf16",
                  65536, 16, 1024, 0, 8192, 1, MEAN_ALL, 16, "offset", 1, 448),
    "256k": Config("256k", "1 layer, 8x4 GQA, d128, bf16 K/V, 262,144-token history in 16-token "
                   "blocks, budget 32,768 tokens (top-k 1,792 + 4,096 recent)", 1, 8, 32, 128,
                   "bf16", 262144, 16, 4096, 0, 32768, 1, MEAN_ALL, 64, "offset", 2, 1792),
    "1m": Config("1m", "1 layer, 8x4 GQA, d128, bf16 K/V, 1,048,576-token history in 16-token "
                 "blocks, budget 262,144 tokens (top-k 15,872 + 8,192 recent)", 1, 8, 32, 128,
                 "bf16", 1048576, 16, 8192, 0, 262144, 1, MEAN_ALL, 256, "offset", 3, 15872),
    "1m_mtp4": Config("1m_mtp4", "4 layers x 1,048,576-token history, 8x4 GQA, d128, bf16 K/V, "
                      "64-token blocks, 4 query tokens, one selection per KV head (max over the 4 "
                      "tokens x 4 heads), top-k 3,968 + 8,192 recent, 256-cluster mixture keys",
                      4, 8, 32, 128, "bf16", 1048576, 64, 8192, 0, 262144, 4, MAX_GROUP, 0,
                      "mixture", 4, 3968),
}
# A recall point (Sec. 4.2, Eq. 10 as printed; the Table 4 setting): after the
# prefill of a new agent step, its 128 query tokens select one working set for
# all layers and heads; the view then stays fixed for the step's decode.
CONFIGS["1m_recall"] = Config(
    "1m_recall", "recall point: 4 layers x 1,048,576-token history, 8x4 GQA, d128, bf16 K/V, 32-token "
    "blocks, 128-token query (the step's prefill), one selection for all layers and heads (Eq. 10), "
    "budget 65,536 tokens (top-k 1,792 + 8,192 recent)", 4, 8, 32, 128, "bf16", 1048576, 32, 8192, 0, 65536,
    128, MEAN_ALL, 256, "offset", 5, 1792)
# The FP8 variants of the 1M-token workloads (same draws, stored as E4M3 codes).
CONFIGS["1m_fp8"] = CONFIGS["1m"].replace(
    name="1m_fp8", kv_dtype="fp8", kv_scale=float(np.float32(8 / 448)),
    description=CONFIGS["1m"].description.replace("bf16 K/V", "FP8 E4M3 K/V (scale 8/448)"))
CONFIGS["1m_mtp4_fp8"] = CONFIGS["1m_mtp4"].replace(
    name="1m_mtp4_fp8", kv_dtype="fp8", kv_scale=float(np.float32(16 / 448)),
    description=CONFIGS["1m_mtp4"].description.replace("bf16 K/V", "FP8 E4M3 K/V (scale 16/448)"))


def fp8_codes(x: np.ndarray, scale: float) -> np.ndarray:
    """fp32 -> OCP E4M3 codes (uint8) of x / scale: fp32 division, then round to
    nearest even, saturating at +-448 (torch's CPU cast after clamping)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32) / np.float32(scale))
    return t.clamp_(-448.0, 448.0).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit pattern (uint16), round to nearest, ties to even (torch's CPU cast)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit pattern -> fp32 (exact)."""
    return (np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(
        np.float32)


@dataclasses.dataclass
class Workload:
    cfg: Config
    seed: int
    q: np.ndarray  # float32 [n_sets][L][n_q][Hq][d]
    k_pool: list  # per layer: [P][Hkv][Bt][d] uint16 (bf16 bits), uint8 (E4M3 codes) or float32
    v_pool: list
    block_to_page: np.ndarray  # int32 [M]
    planted: np.ndarray  # int32 block ids (may be empty)


def _workers() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _store(x: np.ndarray, cfg: Config) -> np.ndarray:
    if cfg.kv_dtype == "fp8":
        return fp8_codes(x, cfg.kv_scale)
    return bf16_bits(x) if cfg.kv_dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def _pool_dtype(cfg: Config):
    return {"f32": np.float32, "bf16": np.uint16, "fp8": np.uint8}[cfg.kv_dtype]


def _offset_pool(ss: np.random.SeedSequence, cfg: Config, chunk: int) -> np.ndarray:
    """[P][Hkv][Bt][d]: per-(page, head) offset N(0, 0.5^2) plus N(0,1) tokens."""
    m, hkv, bt, d = cfg.n_blocks, cfg.n_kv_heads, cfg.block_tokens, cfg.head_dim
    pool = np.empty((m, hkv, bt, d), _pool_dtype(cfg))
    starts = list(range(0, m, chunk))
    children = ss.spawn(len(starts))

    def fill(i):
        lo = starts[i]
        hi = min(m, lo + chunk)
        rng = np.random.Generator(np.random.PCG64(children[i]))
        off = rng.standard_normal((hi - lo, hkv, 1, d), dtype=np.float32) * np.float32(0.5)
        z = rng.standard_normal((hi - lo, hkv, bt, d), dtype=np.float32)
        z += off
        pool[lo:hi] = _store(z, cfg)

    with _cf.ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(fill, range(len(starts))))
    return pool


def _mixture_pool(ss: np.random.SeedSequence, cfg: Config, chunk: int,
                  n_clusters: int = 256, sigma_c: float = 2.0, zipf_s: float = 1.1) -> np.ndarray:
    """[P][Hkv][Bt][d]: keys mu_{j(page)} + N(0,1); centres per KV head, Zipf cluster choice."""
    m, hkv, bt, d = cfg.n_blocks, cfg.n_kv_heads, cfg.block_tokens, cfg.head_dim
    ss_c, ss_j, ss_z = ss.spawn(3)
    rc = np.random.Generator(np.random.PCG64(ss_c))
    centres = rc.standard_normal((hkv, n_clusters, d), dtype=np.float32) * np.float32(sigma_c)
    rj = np.random.Generator(np.random.PCG64(ss_j))
    w = (np.arange(1, n_clusters + 1, dtype=np.float64)) ** (-zipf_s)
    cluster = rj.choice(n_clusters, size=(m, hkv), p=w / w.sum())
    pool = np.empty((m, hkv, bt, d), _pool_dtype(cfg))
    starts = list(range(0, m, chunk))
    children = ss_z.spawn(len(starts))
    heads = np.arange(hkv)[None, :]

    def fill(i):
        lo = starts[i]
        hi = min(m, lo + chunk)
        rng = np.random.Generator(np.random.PCG64(children[i]))
        z = rng.standard_normal((hi - lo, hkv, bt, d), dtype=np.float32)
        z += centres[heads, cluster[lo:hi]][:, :, None, :]
        pool[lo:hi] = _store(z, cfg)

    with _cf.ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(fill, range(len(starts))))
    return pool


def _queries(ss: np.random.SeedSequence, cfg: Config, n_sets: int) -> np.ndarray:
    ss_u, ss_e = ss.spawn(2)
    ru = np.random.Generator(np.random.PCG64(ss_u))
    u = ru.standard_normal((cfg.n_layers, cfg.n_kv_heads, cfg.head_dim))
    re = np.random.Generator(np.random.PCG64(ss_e))
    eps = re.standard_normal((n_sets, cfg.n_layers, cfg.n_q, cfg.n_q_heads, cfg.head_dim))
    head_group = np.arange(cfg.n_q_heads) // cfg.group
    q = u[None, :, None, head_group, :] + 0.5 * eps
    return np.ascontiguousarray(q, dtype=np.float32)


def _plant(ss: np.random.SeedSequence, cfg: Config, pool: np.ndarray, q0: np.ndarray,
           block_to_page: np.ndarray) -> np.ndarray:
    """Overwrite the keys of n_planted candidate blocks with group-aligned keys (cosine 0.9)."""
    rng = np.random.Generator(np.random.PCG64(ss))
    lo, hi = cfg.sink_blocks, cfg.n_blocks - cfg.n_recent
    planted = np.sort(rng.choice(np.arange(lo, hi), size=cfg.n_planted, replace=False))
    d = cfg.head_dim
    for g in range(cfg.n_kv_heads):
        u = q0[:, g * cfg.group:(g + 1) * cfg.group, :].astype(np.float64).reshape(-1, d).mean(0)
        u /= np.linalg.norm(u)
        nu = rng.standard_normal((cfg.n_planted, cfg.block_tokens, d))
        nu -= (nu @ u)[..., None] * u
        nu /= np.linalg.norm(nu, axis=-1, keepdims=True)
        keys = np.sqrt(d) * (0.9 * u + np.sqrt(0.19) * nu)
        pool[block_to_page[planted], g] = _store(keys.astype(np.float32), cfg)
    return planted.astype(np.int32)


def generate(cfg: Config | str, seed: int | None = None, n_query_sets: int = 1,
             layers: int | None = None, with_values: bool = True, chunk_pages: int = 128) -> Workload:
    """Draw one workload.  `layers` limits how many layers' pools are drawn
    (each layer's draws are independent of the others, so a prefix is exact)."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    seed = cfg.seed if seed is None else seed
    n_layers = cfg.n_layers if layers is None else min(layers, cfg.n_layers)
    root = np.random.SeedSequence([int(seed), 0x4B564D])
    ss_q, ss_map, ss_plant, ss_layers = root.spawn(4)
    q = _queries(ss_q, cfg, n_query_sets)
    rmap = np.random.Generator(np.random.PCG64(ss_map))
    block_to_page = rmap.permutation(cfg.n_blocks).astype(np.int32)
    layer_ss = ss_layers.spawn(cfg.n_layers)
    k_pool, v_pool = [], []
    planted = np.zeros(0, np.int32)
    for layer in range(n_layers):
        ss_k, ss_v = layer_ss[layer].spawn(2)
        if cfg.kind == "mixture":
            k = _mixture_pool(ss_k, cfg, chunk_pages)
        else:
            k = _offset_pool(ss_k, cfg, chunk_pages)
            if layer == 0 and cfg.n_planted > 0:
                planted = _plant(ss_plant, cfg, k, q[0, 0], block_to_page)
        k_pool.append(k)
        v_pool.append(_offset_pool(ss_v, cfg, chunk_pages) if with_values else None)
    return Workload(cfg, int(seed), q, k_pool, v_pool, block_to_page, planted)


def small_config(**kw) -> Config:
    """A small offset-kind configuration for parity sweeps; any field may be overridden."""
    base = CONFIGS["tiny"].replace(name="custom", description="custom small shape")
    return base.replace(**kw)
