// Internal declarations of the KVMem HIP library: workspace plans and kernel
// launchers.  Host code in kvmem_api.cpp validates arguments, then calls these.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace kvmem {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// ---- select ------------------------------------------------------------
// Blocks scored by one workgroup of the logit kernel (at least; see score_tile_for).
constexpr int kScoreTile = 64;
// Tile size the logit kernel uses for this shape (a multiple of its step).
int score_tile_for(int head_dim, int n_kv_heads, int rows_per_head);
// Largest candidate count the single-workgroup top-k keeps in registers.
constexpr int kTopkMaxCand = 1024 * 64;

struct SelectPlan {
    int n_layers, n_q, n_q_heads, n_kv_heads, head_dim, group, rows_per_head;
    int n_blocks, n_sink, n_recent, n_cand, k_eff, n_view, n_sel, mode;
    int n_rows;   // n_layers * n_q * n_q_heads
    int score_tile;  // blocks per logit workgroup
    int n_tiles;     // ceil(n_cand / score_tile)
    // byte offsets into the workspace
    size_t off_logits;  // float  [n_rows][n_cand]
    size_t off_tmax;    // float  [n_rows][n_tiles]
    size_t off_tsum;    // double [n_rows][n_tiles]
    size_t off_rmax;    // float  [n_rows]
    size_t off_rinvz;   // double [n_rows]
    size_t off_r32;     // float  [n_sel][n_cand]
    size_t total;
};

inline void plan_select_layout(SelectPlan &p) {
    p.n_rows = p.n_layers * p.n_q * p.n_q_heads;
    p.score_tile = score_tile_for(p.head_dim, p.n_kv_heads, p.rows_per_head);
    p.n_tiles = (p.n_cand + p.score_tile - 1) / p.score_tile;
    size_t o = 0;
    p.off_logits = o; o = align_up(o + sizeof(float) * (size_t)p.n_rows * p.n_cand);
    p.off_tmax = o;   o = align_up(o + sizeof(float) * (size_t)p.n_rows * p.n_tiles);
    p.off_tsum = o;   o = align_up(o + sizeof(double) * (size_t)p.n_rows * p.n_tiles);
    p.off_rmax = o;   o = align_up(o + sizeof(float) * (size_t)p.n_rows);
    p.off_rinvz = o;  o = align_up(o + sizeof(double) * (size_t)p.n_rows);
    p.off_r32 = o;    o = align_up(o + sizeof(float) * (size_t)p.n_sel * p.n_cand);
    p.total = o;
}

// ---- attention ---------------------------------------------------------
constexpr int kAttnTargetGroups = 2048;  // workgroups the split-K launch aims for
constexpr int kAttnMinPages = 4;         // pages per split, lower bound
constexpr int kAttnMaxPages = 64;        // pages per split, upper bound

struct AttnPlan {
    int n_kv_heads, n_q_heads, group, n_q, rows_per_head, head_dim, block_tokens, kv_dtype;
    int n_sel, n_view, last_page_tokens;
    int pages_per_split, n_splits;
    size_t off_part;  // float [Hkv][n_splits][rows_per_head][head_dim + 2]
    size_t total;
};

inline void plan_attn_layout(AttnPlan &p) {
    long long want = ((long long)p.n_view * p.n_kv_heads + kAttnTargetGroups - 1) / kAttnTargetGroups;
    int pps = (int)(want < kAttnMinPages ? kAttnMinPages : (want > kAttnMaxPages ? kAttnMaxPages : want));
    p.pages_per_split = pps;
    p.n_splits = (p.n_view + pps - 1) / pps;
    p.off_part = 0;
    p.total = align_up(sizeof(float) * (size_t)p.n_kv_heads * p.n_splits * p.rows_per_head *
                       (p.head_dim + 2));
}

// ---- launchers (return the launch status) -------------------------------
hipError_t launch_build_index(int kv_dtype, int head_dim, int n_kv_heads, int block_tokens,
                              const void *k_pool, int64_t n_pages, const int32_t *block_to_page,
                              int32_t first_block, int32_t n_blocks, float *index,
                              hipStream_t stream);

hipError_t launch_select(const SelectPlan &p, const float *q, const float *index, float scale,
                         const int32_t *block_to_page, int32_t *view_blocks, int32_t *view_pages,
                         float *scores, char *workspace, hipStream_t stream);

hipError_t launch_sparse_attn(const AttnPlan &p, const float *q, const void *k_pool,
                              const void *v_pool, int64_t n_pages, const int32_t *view_pages,
                              float scale, float *out, float *lse, char *workspace,
                              hipStream_t stream);

}  // namespace kvmem
