// C ABI of the KVMem HIP library: argument validation (host only, before any
// HIP call), workspace sizing, and kernel dispatch.  See include/kvmem.h for
// the contract of every entry point.
#include "../../include/kvmem.h"

#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <string>

#include "kvmem_internal.h"

// Scratch of kvmem_select_noalloc: a file-scope device array, one copy per GPU
// that loads this library, held until the process ends.  Host code never uses
// its name as an address: each device's address is looked up once with
// hipGetSymbolAddress (with that device current) and kept in g_scratch_ptr.
static __device__ __align__(256) unsigned char scratch[KVMEM_SELECT_NOALLOC_MAX_BYTES];

namespace {

thread_local std::string g_error;

kvmem_status fail(kvmem_status st, const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_error = buf;
    return st;
}

kvmem_status ok() {
    g_error.clear();
    return KVMEM_OK;
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

kvmem_status check_geom(const kvmem_geom *g) {
    if (!g) return fail(KVMEM_ERR_NULL, "geom is NULL");
    if (g->n_kv_heads <= 0 || g->n_q_heads <= 0 || g->n_q_heads % g->n_kv_heads != 0)
        return fail(KVMEM_ERR_SHAPE, "n_q_heads (%d) must be a positive multiple of n_kv_heads (%d)",
                    g->n_q_heads, g->n_kv_heads);
    if (g->n_kv_heads > 64)
        return fail(KVMEM_ERR_UNSUPPORTED, "n_kv_heads %d: at most 64 are supported", g->n_kv_heads);
    if (g->head_dim != 64 && g->head_dim != 128)
        return fail(KVMEM_ERR_UNSUPPORTED, "head_dim %d: 64 or 128 is required", g->head_dim);
    if (g->block_tokens != 16 && g->block_tokens != 32 && g->block_tokens != 64)
        return fail(KVMEM_ERR_UNSUPPORTED, "block_tokens %d: 16, 32 or 64 is required",
                    g->block_tokens);
    if (g->kv_dtype != KVMEM_F32 && g->kv_dtype != KVMEM_BF16 && g->kv_dtype != KVMEM_FP8_E4M3)
        return fail(KVMEM_ERR_DTYPE, "kv_dtype %d is not KVMEM_F32, KVMEM_BF16 or KVMEM_FP8_E4M3",
                    g->kv_dtype);
    if (g->kv_dtype == KVMEM_FP8_E4M3 &&
        !(std::isfinite(g->k_scale) && g->k_scale > 0.f && std::isfinite(g->v_scale) && g->v_scale > 0.f))
        return fail(KVMEM_ERR_SHAPE, "FP8 pools need finite positive k_scale and v_scale (got %g, %g)",
                    (double)g->k_scale, (double)g->v_scale);
    return KVMEM_OK;
}

// FP8 codes carry one scale per pool; the other types are used as stored.
float k_scale_of(const kvmem_geom *g) { return g->kv_dtype == KVMEM_FP8_E4M3 ? g->k_scale : 1.f; }
float v_scale_of(const kvmem_geom *g) { return g->kv_dtype == KVMEM_FP8_E4M3 ? g->v_scale : 1.f; }

kvmem_status no_fp8(const kvmem_geom *g, const char *what) {
    if (g->kv_dtype == KVMEM_FP8_E4M3)
        return fail(KVMEM_ERR_UNSUPPORTED, "%s takes f32 or bf16 pools, not FP8", what);
    return KVMEM_OK;
}

kvmem_status plan_view(const kvmem_geom *g, int32_t n_blocks, int32_t n_sink, int32_t n_recent,
                       int64_t model_ctx, int64_t gpu_kv, int32_t *k_eff, int32_t *n_view) {
    if (n_blocks <= 0 || n_sink < 0 || n_recent < 0 || (int64_t)n_sink + n_recent >= n_blocks)
        return fail(KVMEM_ERR_SHAPE,
                    "need n_blocks > 0, n_sink >= 0, n_recent >= 0 and n_sink + n_recent < n_blocks "
                    "(got %d, %d, %d)", n_blocks, n_sink, n_recent);
    const int64_t b_a = model_ctx < gpu_kv ? model_ctx : gpu_kv;  // Eq. 5
    const int64_t mandatory = ((int64_t)n_sink + n_recent) * g->block_tokens;
    if (b_a < mandatory)
        return fail(KVMEM_ERR_BUDGET, "active budget %lld tokens is below the %lld mandatory sink+recent tokens",
                    (long long)b_a, (long long)mandatory);
    const int64_t n_cand = (int64_t)n_blocks - n_sink - n_recent;
    int64_t k = (b_a - mandatory) / g->block_tokens;  // Eq. 7
    if (k > n_cand) k = n_cand;
    if (k_eff) *k_eff = (int32_t)k;
    if (n_view) *n_view = (int32_t)(n_sink + k + n_recent);
    return KVMEM_OK;
}

kvmem_status make_select_plan(const kvmem_geom *g, int32_t n_layers, int32_t n_q, int32_t n_blocks,
                              int32_t n_sink, int32_t n_recent, int64_t model_ctx, int64_t gpu_kv,
                              int32_t mode, kvmem::SelectPlan &p) {
    kvmem_status st = check_geom(g);
    if (st != KVMEM_OK) return st;
    if (n_layers <= 0 || n_q <= 0)
        return fail(KVMEM_ERR_SHAPE, "n_layers (%d) and n_q_tokens (%d) must be positive", n_layers, n_q);
    if (mode != KVMEM_REDUCE_MEAN_ALL && mode != KVMEM_REDUCE_MAX_GROUP)
        return fail(KVMEM_ERR_SHAPE, "mode %d is not a kvmem_reduce value", mode);
    const int group = g->n_q_heads / g->n_kv_heads;
    if ((int64_t)group * n_q > kvmem::kRowsMaxPerHead)
        return fail(KVMEM_ERR_UNSUPPORTED, "G * n_q_tokens = %lld: at most %d query rows per KV head",
                    (long long)group * n_q, kvmem::kRowsMaxPerHead);
    const int rows = group * n_q;
    int32_t k_eff = 0, n_view = 0;
    st = plan_view(g, n_blocks, n_sink, n_recent, model_ctx, gpu_kv, &k_eff, &n_view);
    if (st != KVMEM_OK) return st;
    const int32_t n_cand = n_blocks - n_sink - n_recent;
    if (n_cand > kvmem::kTopkMaxCand)
        return fail(KVMEM_ERR_UNSUPPORTED, "%d candidate blocks: at most %d are supported", n_cand,
                    kvmem::kTopkMaxCand);
    if ((int64_t)n_layers * n_q * g->n_q_heads > (1 << 20))
        return fail(KVMEM_ERR_UNSUPPORTED, "too many query rows");
    p = kvmem::SelectPlan{};
    p.n_layers = n_layers;
    p.n_q = n_q;
    p.n_q_heads = g->n_q_heads;
    p.n_kv_heads = g->n_kv_heads;
    p.head_dim = g->head_dim;
    p.group = group;
    p.rows_per_head = rows;
    p.n_blocks = n_blocks;
    p.n_sink = n_sink;
    p.n_recent = n_recent;
    p.n_cand = n_cand;
    p.k_eff = k_eff;
    p.n_view = n_view;
    p.mode = mode;
    p.n_sel = mode == KVMEM_REDUCE_MEAN_ALL ? 1 : n_layers * g->n_kv_heads;
    kvmem::plan_select_layout(p);
    return KVMEM_OK;
}

kvmem_status make_attn_plan(const kvmem_geom *g, int32_t n_q, int32_t n_sel, int32_t n_view,
                            int32_t last_page_tokens, kvmem::AttnPlan &p) {
    kvmem_status st = check_geom(g);
    if (st != KVMEM_OK) return st;
    if (n_q <= 0) return fail(KVMEM_ERR_SHAPE, "n_q_tokens %d must be positive", n_q);
    if (n_sel != 1 && n_sel != g->n_kv_heads)
        return fail(KVMEM_ERR_SHAPE, "n_sel %d must be 1 or n_kv_heads (%d)", n_sel, g->n_kv_heads);
    if (n_view <= 0) return fail(KVMEM_ERR_SHAPE, "n_view %d must be positive", n_view);
    if (last_page_tokens < 1 || last_page_tokens > g->block_tokens)
        return fail(KVMEM_ERR_SHAPE, "last_page_tokens %d must be in [1, %d]", last_page_tokens,
                    g->block_tokens);
    const int group = g->n_q_heads / g->n_kv_heads;
    if ((int64_t)group * n_q > 4096) return fail(KVMEM_ERR_UNSUPPORTED, "too many query rows per KV head");
    p = kvmem::AttnPlan{};
    p.n_kv_heads = g->n_kv_heads;
    p.n_q_heads = g->n_q_heads;
    p.group = group;
    p.n_q = n_q;
    p.rows_per_head = group * n_q;
    p.head_dim = g->head_dim;
    p.block_tokens = g->block_tokens;
    p.kv_dtype = g->kv_dtype;
    p.k_scale = k_scale_of(g);
    p.v_scale = v_scale_of(g);
    p.n_sel = n_sel;
    p.n_view = n_view;
    p.last_page_tokens = last_page_tokens;
    kvmem::plan_attn_layout(p);
    if (p.n_splits > kvmem::kAttnMaxSplits)
        return fail(KVMEM_ERR_UNSUPPORTED, "a view of %d pages is longer than the library handles", n_view);
    return KVMEM_OK;
}

kvmem_status hip_status(hipError_t e, const char *what) {
    if (e == hipSuccess) return ok();
    return fail(KVMEM_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Arguments of kvmem_select other than the workspace: checked on the host.
kvmem_status check_select_args(const kvmem_geom *geom, const float *q, const float *index,
                               const int32_t *block_to_page, const int32_t *view_blocks,
                               const int32_t *view_pages, const float *scores) {
    if (!q || !index || !block_to_page || !view_blocks || !view_pages)
        return fail(KVMEM_ERR_NULL, "q, index, block_to_page, view_blocks and view_pages must be non-NULL");
    if (!aligned16(q) || !aligned16(index) || !aligned16(block_to_page) || !aligned16(view_blocks) ||
        !aligned16(view_pages) || (scores && !aligned16(scores)))
        return fail(KVMEM_ERR_ALIGN, "device pointers must be 16-byte aligned");
    return KVMEM_OK;
}

// Device address of `scratch` on the device that runs `stream` (which must be
// the current device), looked up on the first call on that device.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

kvmem_status scratch_for(void *stream, char **out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e, "hipGetDevice");
    if (stream) {
        int sdev = -1;
        if ((e = hipStreamGetDevice(static_cast<hipStream_t>(stream), &sdev)) != hipSuccess)
            return hip_status(e, "hipStreamGetDevice");
        if (sdev != dev)
            return fail(KVMEM_ERR_UNSUPPORTED, "the stream runs on device %d but device %d is current", sdev, dev);
    }
    if (dev < 0 || dev >= kMaxDevices)
        return fail(KVMEM_ERR_UNSUPPORTED, "device %d: at most %d devices are supported", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_status(e, "hipGetSymbolAddress(scratch)");
        if (!ptr) return fail(KVMEM_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL on device %d", dev);
        g_scratch_ptr[dev] = ptr;
    }
    *out = static_cast<char *>(g_scratch_ptr[dev]);
    return KVMEM_OK;
}

}  // namespace

extern "C" {

const char *kvmem_last_error(void) { return g_error.c_str(); }

size_t kvmem_index_bytes(const kvmem_geom *geom, int32_t n_blocks) {
    if (check_geom(geom) != KVMEM_OK) return 0;
    if (n_blocks < 0) {
        fail(KVMEM_ERR_SHAPE, "n_blocks %d is negative", n_blocks);
        return 0;
    }
    ok();
    return sizeof(float) * (size_t)kvmem::index_layer_floats(n_blocks, geom->n_kv_heads, geom->head_dim);
}

kvmem_status kvmem_build_index(const kvmem_geom *geom, const void *k_pool, int64_t n_pages,
                               const int32_t *block_to_page, int32_t first_block,
                               int32_t n_blocks, float *index, void *stream) {
    kvmem_status st = check_geom(geom);
    if (st != KVMEM_OK) return st;
    if (first_block < 0 || n_blocks < 0 || (int64_t)first_block + n_blocks > INT32_MAX)
        return fail(KVMEM_ERR_SHAPE, "block range [%d, %d + %d) is invalid", first_block, first_block,
                    n_blocks);
    if (n_blocks == 0) return ok();
    if (!k_pool || !block_to_page || !index)
        return fail(KVMEM_ERR_NULL, "k_pool, block_to_page and index must be non-NULL");
    if (n_pages <= 0) return fail(KVMEM_ERR_SHAPE, "n_pages %lld must be positive", (long long)n_pages);
    if (!aligned16(k_pool) || !aligned16(index) || !aligned16(block_to_page))
        return fail(KVMEM_ERR_ALIGN, "k_pool, block_to_page and index must be 16-byte aligned");
    return hip_status(kvmem::launch_build_index(geom->kv_dtype, geom->head_dim, geom->n_kv_heads,
                                                geom->block_tokens, k_scale_of(geom), k_pool, n_pages,
                                                block_to_page, first_block, n_blocks, index,
                                                static_cast<hipStream_t>(stream)),
                      "build_index launch");
}

kvmem_status kvmem_build_index_rope(const kvmem_geom *geom, const void *k_pool, int64_t n_pages,
                                    const int32_t *block_to_page, const int64_t *block_pos, double rope_base,
                                    int32_t first_block, int32_t n_blocks, float *index, void *stream) {
    kvmem_status st = check_geom(geom);
    if (st != KVMEM_OK) return st;
    if (!(rope_base > 1.0) || !std::isfinite(rope_base))
        return fail(KVMEM_ERR_SHAPE, "rope_base %g must be a finite value above 1", rope_base);
    if (first_block < 0 || n_blocks < 0 || (int64_t)first_block + n_blocks > INT32_MAX)
        return fail(KVMEM_ERR_SHAPE, "block range [%d, %d + %d) is invalid", first_block, first_block,
                    n_blocks);
    if (n_blocks == 0) return ok();
    if (!k_pool || !block_to_page || !index)
        return fail(KVMEM_ERR_NULL, "k_pool, block_to_page and index must be non-NULL");
    if (n_pages <= 0) return fail(KVMEM_ERR_SHAPE, "n_pages %lld must be positive", (long long)n_pages);
    if (!aligned16(k_pool) || !aligned16(index) || !aligned16(block_to_page) ||
        (block_pos && !aligned16(block_pos)))
        return fail(KVMEM_ERR_ALIGN, "k_pool, block_to_page, block_pos and index must be 16-byte aligned");
    kvmem::RopeFreqs fr;
    kvmem::rope_freqs(rope_base, geom->head_dim, fr);
    return hip_status(kvmem::launch_build_index(geom->kv_dtype, geom->head_dim, geom->n_kv_heads,
                                                geom->block_tokens, k_scale_of(geom), k_pool, n_pages,
                                                block_to_page, first_block, n_blocks, index,
                                                static_cast<hipStream_t>(stream), true, block_pos, &fr),
                      "build_index_rope launch");
}

kvmem_status kvmem_materialize(const kvmem_geom *geom, double rope_base, const void *raw_k_pool,
                               const void *v_pool, int64_t n_src_pages, const int32_t *src_pages,
                               const int64_t *positions, const int32_t *dst_pages, int32_t n_blocks,
                               void *k_dst_pool, void *v_dst_pool, int64_t n_dst_pages, void *stream) {
    kvmem_status st = check_geom(geom);
    if (st != KVMEM_OK) return st;
    if ((st = no_fp8(geom, "kvmem_materialize")) != KVMEM_OK) return st;
    if (!(rope_base > 1.0) || !std::isfinite(rope_base))
        return fail(KVMEM_ERR_SHAPE, "rope_base %g must be a finite value above 1", rope_base);
    if (n_blocks < 0 || n_blocks > (1 << 24))
        return fail(KVMEM_ERR_SHAPE, "n_blocks %d must be in [0, 2^24]", n_blocks);
    if (n_blocks == 0) return ok();
    if (!raw_k_pool || !v_pool || !src_pages || !positions || !dst_pages || !k_dst_pool || !v_dst_pool)
        return fail(KVMEM_ERR_NULL, "pools, page lists and positions must be non-NULL");
    if (n_src_pages <= 0 || n_dst_pages <= 0)
        return fail(KVMEM_ERR_SHAPE, "n_src_pages and n_dst_pages must be positive");
    if (!aligned16(raw_k_pool) || !aligned16(v_pool) || !aligned16(k_dst_pool) || !aligned16(v_dst_pool) ||
        !aligned16(src_pages) || !aligned16(positions) || !aligned16(dst_pages))
        return fail(KVMEM_ERR_ALIGN, "device arrays must be 16-byte aligned");
    kvmem::RopeFreqs fr;
    kvmem::rope_freqs(rope_base, geom->head_dim, fr);
    return hip_status(kvmem::launch_materialize(geom->kv_dtype, geom->head_dim, geom->n_kv_heads,
                                                geom->block_tokens, fr, raw_k_pool, v_pool, n_src_pages,
                                                src_pages, positions, dst_pages, n_blocks, k_dst_pool,
                                                v_dst_pool, n_dst_pages, static_cast<hipStream_t>(stream)),
                      "materialize launch");
}

kvmem_status kvmem_rerope(const kvmem_geom *geom, double rope_base, void *k_pool, int64_t n_pages,
                          const int32_t *pages, const int64_t *delta_positions, int32_t n_list, void *stream) {
    kvmem_status st = check_geom(geom);
    if (st != KVMEM_OK) return st;
    if ((st = no_fp8(geom, "kvmem_rerope")) != KVMEM_OK) return st;
    if (!(rope_base > 1.0) || !std::isfinite(rope_base))
        return fail(KVMEM_ERR_SHAPE, "rope_base %g must be a finite value above 1", rope_base);
    if (n_list < 0 || n_list > (1 << 24)) return fail(KVMEM_ERR_SHAPE, "n_list %d must be in [0, 2^24]", n_list);
    if (n_list == 0) return ok();
    if (!k_pool || !pages || !delta_positions)
        return fail(KVMEM_ERR_NULL, "k_pool, pages and delta_positions must be non-NULL");
    if (n_pages <= 0) return fail(KVMEM_ERR_SHAPE, "n_pages %lld must be positive", (long long)n_pages);
    if (!aligned16(k_pool) || !aligned16(pages) || !aligned16(delta_positions))
        return fail(KVMEM_ERR_ALIGN, "device arrays must be 16-byte aligned");
    kvmem::RopeFreqs fr;
    kvmem::rope_freqs(rope_base, geom->head_dim, fr);
    return hip_status(kvmem::launch_rope_delta(geom->kv_dtype, geom->head_dim, geom->n_kv_heads,
                                               geom->block_tokens, fr, k_pool, n_pages, pages, delta_positions,
                                               n_list, static_cast<hipStream_t>(stream)),
                      "rerope launch");
}

namespace {
kvmem_status ws_state(const kvmem_working_set *ws, kvmem::WorkingSetState &s) {
    if (!ws) return fail(KVMEM_ERR_NULL, "working set is NULL");
    if (ws->n_blocks <= 0 || ws->n_pages <= 0 || ws->n_pages > kvmem::kWsMaxPages)
        return fail(KVMEM_ERR_SHAPE, "working set needs n_blocks > 0 and 0 < n_pages <= %d (got %d, %d)",
                    kvmem::kWsMaxPages, ws->n_blocks, ws->n_pages);
    if (!ws->block_page || !ws->block_last_step || !ws->page_block || !ws->page_pos || !ws->page_deltas ||
        !ws->header)
        return fail(KVMEM_ERR_NULL, "every working-set array must be non-NULL");
    if (!aligned16(ws->block_page) || !aligned16(ws->block_last_step) || !aligned16(ws->page_block) ||
        !aligned16(ws->page_pos) || !aligned16(ws->page_deltas) || !aligned16(ws->header))
        return fail(KVMEM_ERR_ALIGN, "working-set arrays must be 16-byte aligned");
    s = kvmem::WorkingSetState{ws->n_blocks, ws->n_pages, ws->block_page, ws->block_last_step, ws->page_block,
                               ws->page_pos, ws->page_deltas, ws->header};
    return KVMEM_OK;
}
}  // namespace

kvmem_status kvmem_working_set_reset(const kvmem_working_set *ws, void *stream) {
    kvmem::WorkingSetState s;
    kvmem_status st = ws_state(ws, s);
    if (st != KVMEM_OK) return st;
    return hip_status(kvmem::launch_ws_reset(s, static_cast<hipStream_t>(stream)), "working_set_reset launch");
}

size_t kvmem_working_set_workspace_bytes(int32_t n_view, int32_t n_pages) {
    if (n_view < 0 || n_pages <= 0 || n_pages > kvmem::kWsMaxPages || n_view > n_pages) {
        fail(KVMEM_ERR_SHAPE, "need 0 <= n_view <= n_pages <= %d (got %d, %d)", kvmem::kWsMaxPages, n_view, n_pages);
        return 0;
    }
    ok();
    return kvmem::ws_scratch_bytes(n_view, n_pages);
}

kvmem_status kvmem_working_set_update(const kvmem_geom *geom, double rope_base, const kvmem_working_set *ws,
                                      int32_t step, const int32_t *view_blocks, int32_t n_view,
                                      int64_t first_position, int32_t max_deltas, const int32_t *block_to_page,
                                      const void *raw_k_pool, const void *v_pool, int64_t n_src_pages,
                                      void *k_exec_pool, void *v_exec_pool, int32_t *exec_pages, int32_t *counts,
                                      void *workspace, size_t workspace_bytes, void *stream) {
    kvmem_status st = check_geom(geom);
    if (st != KVMEM_OK) return st;
    if ((st = no_fp8(geom, "kvmem_working_set_update")) != KVMEM_OK) return st;
    kvmem::WorkingSetState s;
    if ((st = ws_state(ws, s)) != KVMEM_OK) return st;
    if (!(rope_base > 1.0) || !std::isfinite(rope_base))
        return fail(KVMEM_ERR_SHAPE, "rope_base %g must be a finite value above 1", rope_base);
    if (step < 0 || n_view < 0 || n_view > ws->n_pages || max_deltas < 0)
        return fail(KVMEM_ERR_SHAPE, "need step >= 0, 0 <= n_view <= n_pages (%d) and max_deltas >= 0 "
                    "(got %d, %d, %d)", ws->n_pages, step, n_view, max_deltas);
    if (n_src_pages <= 0) return fail(KVMEM_ERR_SHAPE, "n_src_pages must be positive");
    if (!view_blocks || !block_to_page || !raw_k_pool || !v_pool || !k_exec_pool || !v_exec_pool || !exec_pages ||
        !counts)
        return fail(KVMEM_ERR_NULL, "view, block table, pools, exec_pages and counts must be non-NULL");
    if (!aligned16(view_blocks) || !aligned16(block_to_page) || !aligned16(raw_k_pool) || !aligned16(v_pool) ||
        !aligned16(k_exec_pool) || !aligned16(v_exec_pool) || !aligned16(exec_pages) || !aligned16(counts))
        return fail(KVMEM_ERR_ALIGN, "device arrays must be 16-byte aligned");
    const size_t need = kvmem::ws_scratch_bytes(n_view, ws->n_pages);
    if (!workspace || workspace_bytes < need)
        return fail(KVMEM_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required", workspace_bytes,
                    need);
    kvmem::WsScratch w;
    kvmem::ws_scratch_bytes(n_view, ws->n_pages, &w, static_cast<char *>(workspace));
    kvmem::RopeFreqs fr;
    kvmem::rope_freqs(rope_base, geom->head_dim, fr);
    return hip_status(kvmem::launch_ws_update(s, w, geom->kv_dtype, geom->head_dim, geom->n_kv_heads,
                                              geom->block_tokens, fr, step, view_blocks, n_view, first_position,
                                              max_deltas, block_to_page, raw_k_pool, v_pool, n_src_pages,
                                              k_exec_pool, v_exec_pool, exec_pages, counts,
                                              static_cast<hipStream_t>(stream)),
                      "working_set_update launch");
}

kvmem_status kvmem_plan_view(const kvmem_geom *geom, int32_t n_blocks, int32_t n_sink_blocks,
                             int32_t n_recent_blocks, int64_t model_ctx_tokens,
                             int64_t gpu_kv_tokens, int32_t *k_eff, int32_t *n_view) {
    kvmem_status st = check_geom(geom);
    if (st != KVMEM_OK) return st;
    st = plan_view(geom, n_blocks, n_sink_blocks, n_recent_blocks, model_ctx_tokens, gpu_kv_tokens,
                   k_eff, n_view);
    return st == KVMEM_OK ? ok() : st;
}

size_t kvmem_select_workspace_bytes(const kvmem_geom *geom, int32_t n_layers, int32_t n_q_tokens,
                                    int32_t n_blocks, int32_t n_sink_blocks,
                                    int32_t n_recent_blocks, int32_t mode) {
    kvmem::SelectPlan p;
    // the budget does not change the workspace; use the largest one
    if (make_select_plan(geom, n_layers, n_q_tokens, n_blocks, n_sink_blocks, n_recent_blocks,
                         INT64_MAX, INT64_MAX, mode, p) != KVMEM_OK)
        return 0;
    ok();
    return p.total;
}

kvmem_status kvmem_select(const kvmem_geom *geom, int32_t n_layers, const float *q,
                          int32_t n_q_tokens, const float *index, int32_t n_blocks,
                          int32_t n_sink_blocks, int32_t n_recent_blocks,
                          int64_t model_ctx_tokens, int64_t gpu_kv_tokens, int32_t mode,
                          float scale, const int32_t *block_to_page, int32_t *view_blocks,
                          int32_t *view_pages, float *scores, int32_t *n_view_out,
                          void *workspace, size_t workspace_bytes, void *stream) {
    kvmem::SelectPlan p;
    kvmem_status st = make_select_plan(geom, n_layers, n_q_tokens, n_blocks, n_sink_blocks,
                                       n_recent_blocks, model_ctx_tokens, gpu_kv_tokens, mode, p);
    if (st != KVMEM_OK) return st;
    if ((st = check_select_args(geom, q, index, block_to_page, view_blocks, view_pages, scores)) != KVMEM_OK)
        return st;
    if (!workspace || workspace_bytes < p.total)
        return fail(KVMEM_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required",
                    workspace_bytes, p.total);
    if (!aligned16(workspace)) return fail(KVMEM_ERR_ALIGN, "device pointers must be 16-byte aligned");
    if (!(scale > 0.f)) scale = 1.0f / sqrtf((float)geom->head_dim);
    if (n_view_out) *n_view_out = p.n_view;
    return hip_status(kvmem::launch_select(p, q, index, scale, block_to_page, view_blocks, view_pages,
                                           scores, static_cast<char *>(workspace),
                                           static_cast<hipStream_t>(stream)),
                      "select launch");
}

kvmem_status kvmem_select_noalloc(const kvmem_geom *geom, int32_t n_layers, const float *q,
                                  int32_t n_q_tokens, const float *index, int32_t n_blocks,
                                  int32_t n_sink_blocks, int32_t n_recent_blocks,
                                  int64_t model_ctx_tokens, int64_t gpu_kv_tokens, int32_t mode,
                                  float scale, const int32_t *block_to_page, int32_t *view_blocks,
                                  int32_t *view_pages, float *scores, int32_t *n_view_out, void *stream) {
    kvmem::SelectPlan p;
    kvmem_status st = make_select_plan(geom, n_layers, n_q_tokens, n_blocks, n_sink_blocks,
                                       n_recent_blocks, model_ctx_tokens, gpu_kv_tokens, mode, p);
    if (st != KVMEM_OK) return st;
    if ((st = check_select_args(geom, q, index, block_to_page, view_blocks, view_pages, scores)) != KVMEM_OK)
        return st;
    if (p.total > (size_t)KVMEM_SELECT_NOALLOC_MAX_BYTES)
        return fail(KVMEM_ERR_WORKSPACE,
                    "this selection needs %zu bytes of scratch; kvmem_select_noalloc has %zu "
                    "(use kvmem_select with a workspace)", p.total, (size_t)KVMEM_SELECT_NOALLOC_MAX_BYTES);
    char *ws = nullptr;
    if ((st = scratch_for(stream, &ws)) != KVMEM_OK) return st;
    if (!(scale > 0.f)) scale = 1.0f / sqrtf((float)geom->head_dim);
    if (n_view_out) *n_view_out = p.n_view;
    return hip_status(kvmem::launch_select(p, q, index, scale, block_to_page, view_blocks, view_pages,
                                           scores, ws, static_cast<hipStream_t>(stream)),
                      "select launch");
}

size_t kvmem_sparse_attn_workspace_bytes(const kvmem_geom *geom, int32_t n_q_tokens, int32_t n_sel,
                                         int32_t n_view) {
    kvmem::AttnPlan p;
    if (make_attn_plan(geom, n_q_tokens, n_sel, n_view, 1, p) != KVMEM_OK) return 0;
    ok();
    return p.total;
}

kvmem_status kvmem_sparse_attn(const kvmem_geom *geom, const float *q, int32_t n_q_tokens,
                               const void *k_pool, const void *v_pool, int64_t n_pages,
                               const int32_t *view_pages, int32_t n_sel, int32_t n_view,
                               int32_t last_page_tokens, float scale, float *out, float *lse,
                               void *workspace, size_t workspace_bytes, void *stream) {
    kvmem::AttnPlan p;
    kvmem_status st = make_attn_plan(geom, n_q_tokens, n_sel, n_view, last_page_tokens, p);
    if (st != KVMEM_OK) return st;
    if (!q || !k_pool || !v_pool || !view_pages || !out)
        return fail(KVMEM_ERR_NULL, "q, k_pool, v_pool, view_pages and out must be non-NULL");
    if (n_pages <= 0) return fail(KVMEM_ERR_SHAPE, "n_pages %lld must be positive", (long long)n_pages);
    if (!workspace || workspace_bytes < p.total)
        return fail(KVMEM_ERR_WORKSPACE, "workspace of %zu bytes is smaller than the %zu required",
                    workspace_bytes, p.total);
    if (!aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(view_pages) ||
        !aligned16(out) || (lse && !aligned16(lse)) || !aligned16(workspace))
        return fail(KVMEM_ERR_ALIGN, "device pointers must be 16-byte aligned");
    if (!(scale > 0.f)) scale = 1.0f / sqrtf((float)geom->head_dim);
    return hip_status(kvmem::launch_sparse_attn(p, q, k_pool, v_pool, n_pages, view_pages, scale, out,
                                                lse, static_cast<char *>(workspace),
                                                static_cast<hipStream_t>(stream)),
                      "sparse_attn launch");
}

}  // extern "C"
