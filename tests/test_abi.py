"""Host-side tests of the C ABI: the library loads, exports everything the
header declares, and rejects bad arguments before touching HIP.

Every call here fails argument validation, which happens before any HIP call,
so none of them needs (or touches) a GPU.  No call is ever made with fake
pointers that could pass validation.
"""
import ctypes
import subprocess

import pytest
import torch

import oracle
from paper_2609_04852_amd import kvmem as K
from paper_2609_04852_amd import workload as W
from paper_2609_04852_amd.step import geom_of

FAKE = ctypes.c_void_p(0x10000)  # aligned, never dereferenced: validation fails first
MISALIGNED = ctypes.c_void_p(0x10004)


@pytest.fixture(scope="module")
def L():
    return K.lib()


# The validation cases below pass fake device pointers that are rejected on the
# host.  They are host logic, so they are only run where no GPU is visible.
no_gpu = pytest.mark.skipif(torch.cuda.is_available(), reason="host-only validation checks")


def g1(**kw):
    base = dict(n_kv_heads=8, n_q_heads=32, head_dim=128, block_tokens=16, kv_dtype=K.KVMEM_BF16)
    base.update(kw)
    return K.kvmem_geom(**base)


def test_exports_every_declared_function(L):
    names = K.header_functions()
    assert {"kvmem_build_index", "kvmem_select", "kvmem_sparse_attn", "kvmem_plan_view",
            "kvmem_select_workspace_bytes", "kvmem_sparse_attn_workspace_bytes",
            "kvmem_last_error"} <= set(names)
    for n in names:
        assert hasattr(L, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", K.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if " T " in line}
    assert set(names) <= exported


def _status(rc):
    return K.STATUS_NAMES[rc]


def test_geometry_validation(L):
    z = ctypes.c_int32()
    assert _status(L.kvmem_plan_view(None, 100, 0, 4, 10**6, 10**6, None, None)) == "KVMEM_ERR_NULL"
    assert "geom" in K.kvmem_last_error()
    for bad, st in [(dict(n_q_heads=30), "KVMEM_ERR_SHAPE"), (dict(n_kv_heads=65, n_q_heads=130), "KVMEM_ERR_UNSUPPORTED"),
                    (dict(head_dim=96), "KVMEM_ERR_UNSUPPORTED"), (dict(block_tokens=8), "KVMEM_ERR_UNSUPPORTED"),
                    (dict(kv_dtype=7), "KVMEM_ERR_DTYPE")]:
        rc = L.kvmem_plan_view(ctypes.byref(g1(**bad)), 100, 0, 4, 10**6, 10**6, ctypes.byref(z), None)
        assert _status(rc) == st, bad
        assert K.kvmem_last_error() != ""


@pytest.mark.parametrize("name", list(W.CONFIGS))
def test_plan_view_matches_oracle_on_configs(name):
    c = W.CONFIGS[name]
    k, n = K.kvmem_plan_view(geom_of(c), c.n_blocks, c.sink_blocks, c.n_recent, c.budget_tokens,
                             c.budget_tokens)
    assert k == c.top_k == oracle.k_eff(c.budget_tokens, c.budget_tokens, c.block_tokens, c.n_blocks,
                                        c.sink_blocks, c.n_recent)
    assert n == c.n_view


def test_plan_view_budget_cases():
    g = K.Geom(8, 32, 128, 16, K.KVMEM_BF16)
    assert K.kvmem_plan_view(g, 65536, 0, 512, 262144, 100_000)[0] == (100_000 - 8192) // 16
    assert K.kvmem_plan_view(g, 100, 1, 4, 10**9, 10**9) == (95, 100)
    with pytest.raises(K.KvmemError) as e:
        K.kvmem_plan_view(g, 100, 0, 4, 63, 10**6)
    assert e.value.status == -5
    with pytest.raises(K.KvmemError):
        K.kvmem_plan_view(g, 100, 50, 50, 10**6, 10**6)  # no candidate left


def test_any_gqa_width_is_accepted():
    """Every G * n_q up to 4,096 rows per KV head and every KV head count up to 64
    is a valid selection and attention shape (Eq. 10's head map g(h) is general)."""
    for hkv, hq in [(8, 24), (8, 40), (6, 36), (4, 28), (3, 12), (5, 5), (7, 56), (64, 64)]:
        for n_q in (1, 3, 4, 9):
            g = K.Geom(hkv, hq, 128, 16, K.KVMEM_BF16)
            assert K.kvmem_select_workspace_bytes(g, 1, n_q, 4096, 0, 64, K.KVMEM_REDUCE_MEAN_ALL) > 0
            assert K.kvmem_select_workspace_bytes(g, 2, n_q, 4096, 1, 64, K.KVMEM_REDUCE_MAX_GROUP) > 0
            assert K.kvmem_sparse_attn_workspace_bytes(g, n_q, hkv, 512) > 0
    with pytest.raises(K.KvmemError) as e:
        K.kvmem_select_workspace_bytes(K.Geom(8, 32, 128, 16, K.KVMEM_BF16), 1, 1025, 4096, 0, 64, 0)
    assert e.value.status == -2 or "4096" in str(e.value)


def test_workspace_queries():
    c = W.CONFIGS["1m"]
    g = geom_of(c)
    ws = K.kvmem_select_workspace_bytes(g, 1, 1, c.n_blocks, 0, c.n_recent, K.KVMEM_REDUCE_MEAN_ALL)
    assert ws >= 32 * c.n_candidates * 4  # the logits alone
    aws = K.kvmem_sparse_attn_workspace_bytes(g, 1, 1, c.n_view)
    assert aws > 0
    with pytest.raises(K.KvmemError):
        K.kvmem_select_workspace_bytes(g, 1, 1, (1 << 20) + 1024, 0, 512, 0)  # too many candidates
    with pytest.raises(K.KvmemError):
        K.kvmem_sparse_attn_workspace_bytes(g, 1, 3, 10)  # n_sel must be 1 or Hkv


@no_gpu
def test_build_index_validation(L):
    g = ctypes.byref(g1())
    assert _status(L.kvmem_build_index(g, None, 10, FAKE, 0, 4, FAKE, None)) == "KVMEM_ERR_NULL"
    assert _status(L.kvmem_build_index(g, FAKE, 10, FAKE, -1, 4, FAKE, None)) == "KVMEM_ERR_SHAPE"
    assert _status(L.kvmem_build_index(g, FAKE, 0, FAKE, 0, 4, FAKE, None)) == "KVMEM_ERR_SHAPE"
    assert _status(L.kvmem_build_index(g, MISALIGNED, 10, FAKE, 0, 4, FAKE, None)) == "KVMEM_ERR_ALIGN"
    # empty range: a no-op that succeeds without any pointer
    assert _status(L.kvmem_build_index(g, None, 10, None, 0, 0, None, None)) == "KVMEM_OK"


def _select(L, geom, **kw):
    a = dict(n_layers=1, q=FAKE, n_q=1, index=FAKE, n_blocks=4096, n_sink=0, n_recent=64,
             model=8192, gpu=8192, mode=0, scale=0.0, b2p=FAKE, vb=FAKE, vp=FAKE, scores=None,
             n_view=None, ws=FAKE, ws_bytes=0, stream=None)
    a.update(kw)
    return _status(L.kvmem_select(ctypes.byref(geom), a["n_layers"], a["q"], a["n_q"], a["index"],
                                  a["n_blocks"], a["n_sink"], a["n_recent"], a["model"], a["gpu"],
                                  a["mode"], a["scale"], a["b2p"], a["vb"], a["vp"], a["scores"],
                                  a["n_view"], a["ws"], a["ws_bytes"], a["stream"]))


@no_gpu
def test_select_validation(L):
    g = g1()
    big = 1 << 40
    assert _select(L, g, ws_bytes=0) == "KVMEM_ERR_WORKSPACE"
    assert _select(L, g, q=None, ws_bytes=big) == "KVMEM_ERR_NULL"
    assert _select(L, g, vp=None, ws_bytes=big) == "KVMEM_ERR_NULL"
    assert _select(L, g, q=MISALIGNED, ws_bytes=big) == "KVMEM_ERR_ALIGN"
    assert _select(L, g, scores=MISALIGNED, ws_bytes=big) == "KVMEM_ERR_ALIGN"
    assert _select(L, g, model=1000, ws_bytes=big) == "KVMEM_ERR_BUDGET"
    assert _select(L, g, n_recent=4096, ws_bytes=big) == "KVMEM_ERR_SHAPE"
    assert _select(L, g, mode=5, ws_bytes=big) == "KVMEM_ERR_SHAPE"
    assert _select(L, g, n_q=1028, ws_bytes=big) == "KVMEM_ERR_UNSUPPORTED"  # G*n_q = 4112 > 4096
    assert _select(L, g, n_blocks=(1 << 20) + 1024, n_recent=512, model=10**9, gpu=10**9,
                   ws_bytes=big) == "KVMEM_ERR_UNSUPPORTED"
    assert _select(L, g, n_layers=0, ws_bytes=big) == "KVMEM_ERR_SHAPE"


def _attn(L, geom, **kw):
    a = dict(q=FAKE, n_q=1, k=FAKE, v=FAKE, n_pages=100, vp=FAKE, n_sel=1, n_view=10, lpt=16,
             scale=0.0, out=FAKE, lse=None, ws=FAKE, ws_bytes=0, stream=None)
    a.update(kw)
    return _status(L.kvmem_sparse_attn(ctypes.byref(geom), a["q"], a["n_q"], a["k"], a["v"],
                                       a["n_pages"], a["vp"], a["n_sel"], a["n_view"], a["lpt"],
                                       a["scale"], a["out"], a["lse"], a["ws"], a["ws_bytes"],
                                       a["stream"]))


@no_gpu
def test_sparse_attn_validation(L):
    g = g1()
    big = 1 << 40
    assert _attn(L, g) == "KVMEM_ERR_WORKSPACE"
    assert _attn(L, g, ws=None, ws_bytes=big) == "KVMEM_ERR_WORKSPACE"
    assert _attn(L, g, k=None, ws_bytes=big) == "KVMEM_ERR_NULL"
    assert _attn(L, g, v=MISALIGNED, ws_bytes=big) == "KVMEM_ERR_ALIGN"
    assert _attn(L, g, n_sel=3, ws_bytes=big) == "KVMEM_ERR_SHAPE"
    assert _attn(L, g, n_view=0, ws_bytes=big) == "KVMEM_ERR_SHAPE"
    assert _attn(L, g, lpt=0, ws_bytes=big) == "KVMEM_ERR_SHAPE"
    assert _attn(L, g, lpt=17, ws_bytes=big) == "KVMEM_ERR_SHAPE"
    assert _attn(L, g, n_q=0, ws_bytes=big) == "KVMEM_ERR_SHAPE"
    assert _attn(L, g, n_pages=0, ws_bytes=big) == "KVMEM_ERR_SHAPE"
    assert _attn(L, g1(head_dim=80), ws_bytes=big) == "KVMEM_ERR_UNSUPPORTED"


@no_gpu
def test_rope_calls_validation(L):
    g = ctypes.byref(g1())
    # index from encoded keys
    assert _status(L.kvmem_build_index_rope(g, FAKE, 10, FAKE, None, 0.5, 0, 4, FAKE, None)) == "KVMEM_ERR_SHAPE"
    assert _status(L.kvmem_build_index_rope(g, FAKE, 10, FAKE, None, float("inf"), 0, 4, FAKE, None)) \
        == "KVMEM_ERR_SHAPE"
    assert _status(L.kvmem_build_index_rope(g, None, 10, FAKE, None, 1e6, 0, 4, FAKE, None)) == "KVMEM_ERR_NULL"
    assert _status(L.kvmem_build_index_rope(g, FAKE, 10, FAKE, MISALIGNED, 1e6, 0, 4, FAKE, None)) \
        == "KVMEM_ERR_ALIGN"
    assert _status(L.kvmem_build_index_rope(g, None, 10, None, None, 1e6, 0, 0, None, None)) == "KVMEM_OK"
    # materialisation
    m = lambda **kw: _status(L.kvmem_materialize(
        g, kw.get("base", 1e6), kw.get("raw", FAKE), FAKE, kw.get("nsrc", 10), FAKE, kw.get("pos", FAKE), FAKE,
        kw.get("n", 4), FAKE, FAKE, kw.get("ndst", 10), None))
    assert m(base=1.0) == "KVMEM_ERR_SHAPE"
    assert m(raw=None) == "KVMEM_ERR_NULL"
    assert m(pos=None) == "KVMEM_ERR_NULL"
    assert m(nsrc=0) == "KVMEM_ERR_SHAPE"
    assert m(ndst=-1) == "KVMEM_ERR_SHAPE"
    assert m(n=-1) == "KVMEM_ERR_SHAPE"
    assert m(pos=MISALIGNED) == "KVMEM_ERR_ALIGN"
    assert m(n=0, raw=None, pos=None) == "KVMEM_OK"
    # delta re-encoding
    r = lambda **kw: _status(L.kvmem_rerope(g, kw.get("base", 1e6), kw.get("k", FAKE), kw.get("np", 10),
                                            kw.get("pages", FAKE), FAKE, kw.get("n", 4), None))
    assert r(base=float("nan")) == "KVMEM_ERR_SHAPE"
    assert r(k=None) == "KVMEM_ERR_NULL"
    assert r(np=0) == "KVMEM_ERR_SHAPE"
    assert r(pages=MISALIGNED) == "KVMEM_ERR_ALIGN"
    assert r(n=0, k=None, pages=None) == "KVMEM_OK"
    bad = g1(head_dim=96)
    assert _status(L.kvmem_rerope(ctypes.byref(bad), 1e6, FAKE, 10, FAKE, FAKE, 4, None)) == "KVMEM_ERR_UNSUPPORTED"


def test_fp8_geometry_validation(L):
    z = ctypes.c_int32()
    for ks, vs, st in [(0.02, 0.02, "KVMEM_OK"), (0.0, 0.02, "KVMEM_ERR_SHAPE"), (0.02, -1.0, "KVMEM_ERR_SHAPE"),
                       (float("inf"), 0.02, "KVMEM_ERR_SHAPE"), (0.02, float("nan"), "KVMEM_ERR_SHAPE")]:
        g = g1(kv_dtype=K.KVMEM_FP8_E4M3, k_scale=ks, v_scale=vs)
        assert _status(L.kvmem_plan_view(ctypes.byref(g), 100, 0, 4, 10**6, 10**6, ctypes.byref(z), None)) == st
    # the scales are not read for the other types
    assert _status(L.kvmem_plan_view(ctypes.byref(g1(k_scale=0.0, v_scale=float("nan"))), 100, 0, 4, 10**6,
                                     10**6, ctypes.byref(z), None)) == "KVMEM_OK"


@no_gpu
def test_fp8_position_calls_unsupported(L):
    g = ctypes.byref(g1(kv_dtype=K.KVMEM_FP8_E4M3, k_scale=0.02, v_scale=0.02))
    assert _status(L.kvmem_materialize(g, 1e6, FAKE, FAKE, 10, FAKE, FAKE, FAKE, 4, FAKE, FAKE, 10, None)) \
        == "KVMEM_ERR_UNSUPPORTED"
    assert _status(L.kvmem_rerope(g, 1e6, FAKE, 10, FAKE, FAKE, 4, None)) == "KVMEM_ERR_UNSUPPORTED"
    assert "FP8" in K.kvmem_last_error()
    # the index from encoded keys does take FP8 pools (host checks pass down to the NULL check)
    assert _status(L.kvmem_build_index_rope(g, None, 10, FAKE, None, 1e6, 0, 4, FAKE, None)) == "KVMEM_ERR_NULL"


@no_gpu
def test_working_set_validation(L):
    ws = K.kvmem_working_set(100, 50, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)
    assert L.kvmem_working_set_workspace_bytes(60, 50) == 0   # view larger than the pool
    assert L.kvmem_working_set_workspace_bytes(10, 50) > 0
    g = ctypes.byref(g1())
    big = 1 << 30

    def up(**kw):
        w = kw.get("ws", ws)
        return _status(L.kvmem_working_set_update(
            kw.get("g", g), kw.get("base", 1e6), ctypes.byref(w) if w is not None else None, kw.get("step", 1),
            kw.get("view", FAKE), kw.get("n", 10), 0, kw.get("md", 2), FAKE, FAKE, FAKE, 100, FAKE, FAKE, FAKE,
            kw.get("counts", FAKE), FAKE, kw.get("wsb", big), None))

    assert up(ws=None) == "KVMEM_ERR_NULL"
    assert up(base=0.5) == "KVMEM_ERR_SHAPE"
    assert up(step=-1) == "KVMEM_ERR_SHAPE"
    assert up(n=51) == "KVMEM_ERR_SHAPE"
    assert up(md=-1) == "KVMEM_ERR_SHAPE"
    assert up(view=None) == "KVMEM_ERR_NULL"
    assert up(counts=MISALIGNED) == "KVMEM_ERR_ALIGN"
    assert up(wsb=16) == "KVMEM_ERR_WORKSPACE"
    assert up(ws=K.kvmem_working_set(100, 0, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE)) == "KVMEM_ERR_SHAPE"
    assert up(ws=K.kvmem_working_set(100, 50, FAKE, None, FAKE, FAKE, FAKE, FAKE)) == "KVMEM_ERR_NULL"
    fp8 = ctypes.byref(g1(kv_dtype=K.KVMEM_FP8_E4M3, k_scale=0.02, v_scale=0.02))
    assert up(g=fp8) == "KVMEM_ERR_UNSUPPORTED"
    assert _status(L.kvmem_working_set_reset(None, None)) == "KVMEM_ERR_NULL"
