/*
 * kvmem.h -- C ABI of the MI355X (gfx950) KVMem decode-step library.
 *
 * KVMem (arXiv 2609.04852) keeps an agent's overflowed history as paged KV and,
 * at each recall point, materializes a bounded execution view: it summarizes
 * every history block by the mean of its position-independent keys (Eq. 9),
 * scores every candidate block against the current query with a per-head
 * softmax over blocks (Eq. 10), keeps the configured sink and recent blocks,
 * fills the rest of the active budget (Eq. 5, Eq. 7) with the highest-scoring
 * blocks in chronological order (Sec. 4.3), and runs attention over that view
 * through a page table (Sec. 4.4, Sec. 5.3).  This library implements that
 * path on one GPU with every step in HIP kernels:
 *
 *   kvmem_build_index  Eq. 9   Mean-K index rows for a range of blocks
 *   kvmem_select       Eq. 10 + selector: scores, top-k under the budget,
 *                      chronological view tables
 *   kvmem_sparse_attn  decode attention over the view's pages (split-K)
 *   kvmem_build_index_rope, kvmem_materialize, kvmem_rerope
 *                      position handling: index from RoPE-encoded keys,
 *                      re-encoding of selected blocks at compact positions
 *   kvmem_working_set_reset, kvmem_working_set_workspace_bytes,
 *   kvmem_working_set_update
 *                      a recall point's working-set delta (Eq. 11, Eq. 12)
 *                      over a bounded execution page pool with page reuse
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.  Pointers marked "dev" are device pointers, "host" are host
 * pointers.  Every pointer is borrowed: the library never allocates or frees
 * memory.  Scratch space is passed in as `workspace`, sized by the matching
 * *_workspace_bytes query.  All arrays are dense, row-major (C order), and
 * device arrays must be 16-byte aligned.
 *
 * Layouts.  Hkv = n_kv_heads, Hq = n_q_heads (a multiple of Hkv, G = Hq/Hkv),
 * d = head_dim, Bt = block_tokens (one history block occupies one page):
 *   K/V page pool  [n_pages][Hkv][Bt][d]      kv_dtype (f32, bf16 bits, or FP8
 *                  E4M3 codes, one byte each, read as code value * k_scale
 *                  for K and * v_scale for V)
 *   Mean-K index   [n_layers][T][Hkv][d/4][64][4]  float, tiled: T = ceil(M/64)
 *                  tiles of 64 blocks, M = history blocks; the entry of block
 *                  b, KV head g, dimension j is at
 *                  (((b/64)*Hkv + g)*(d/4) + j/4)*256 + (b%64)*4 + j%4
 *                  within a layer (kvmem_index_bytes gives a layer's size)
 *   query          [n_layers][n_q][Hq][d]     float, position independent
 *   block_to_page  [M]                        int32, history block -> page
 *   view tables    [n_sel][n_view]            int32
 * Query head h attends through KV head floor(h / G).
 *
 * Streams.  Every call enqueues its kernels on `stream` (a hipStream_t, NULL
 * for the null stream) and returns without synchronizing; buffers must stay
 * valid until that work completes.  No call copies data between host and
 * device, so a decode step needs no host synchronization.
 *
 * Errors.  Arguments are checked on the host before any HIP call.  On an error
 * nothing is enqueued, no output is written, and kvmem_last_error() describes
 * the problem.  A failed launch returns KVMEM_ERR_HIP.  Device-side contents
 * cannot be checked on the host: a page id outside [0, n_pages) is never
 * dereferenced; the outputs that depend on it are set to NaN instead.
 *
 * Determinism.  Identical inputs give bitwise-identical outputs (fixed-order
 * reductions; integer atomics only).  Calls that share a workspace must not
 * overlap in time.
 */
#ifndef KVMEM_H
#define KVMEM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    KVMEM_OK = 0,
    KVMEM_ERR_NULL = -1,        /* a required pointer is NULL */
    KVMEM_ERR_SHAPE = -2,       /* inconsistent or out-of-range sizes */
    KVMEM_ERR_DTYPE = -3,       /* unknown kv_dtype */
    KVMEM_ERR_UNSUPPORTED = -4, /* valid, but not a shape the library handles */
    KVMEM_ERR_BUDGET = -5,      /* active budget cannot hold sink + recent (Eq. 7) */
    KVMEM_ERR_WORKSPACE = -6,   /* workspace missing or smaller than required */
    KVMEM_ERR_ALIGN = -7,       /* a device pointer is not 16-byte aligned */
    KVMEM_ERR_HIP = -8          /* a HIP runtime call or kernel launch failed */
} kvmem_status;

/* Element type of the K/V pools.  KVMEM_FP8_E4M3 is the OCP 8-bit float with
 * 4 exponent bits (bias 7) and 3 mantissa bits, no infinities and NaN at
 * S.1111.111 (the FP8 KV cache of the paper's evaluation platforms, Sec. 6);
 * each pool carries one fp32 scale (kvmem_geom.k_scale, .v_scale). */
typedef enum { KVMEM_F32 = 0, KVMEM_BF16 = 1, KVMEM_FP8_E4M3 = 2 } kvmem_dtype;

/* How Eq. 10's per-(layer, query token, query head) block softmaxes are
 * combined into selection scores. */
typedef enum {
    /* Eq. 10 as printed: R_b = sum_m mean_{l,h} softmax_{b' in C}(...)_b.
     * One selection shared by every KV head (n_sel = 1). */
    KVMEM_REDUCE_MEAN_ALL = 0,
    /* One selection per (layer, KV head): R[l][g][b] = max over the query
     * tokens m and the query heads h of group g of the same softmax values.
     * n_sel = n_layers * Hkv. */
    KVMEM_REDUCE_MAX_GROUP = 1
} kvmem_reduce;

/* Model geometry shared by all calls.  Supported: 1 <= Hkv <= 64, any
 * G = Hq/Hkv with G * n_q <= 4096 query rows per KV head (every call), d in
 * {64, 128}, Bt in {16, 32, 64}; anything else returns KVMEM_ERR_UNSUPPORTED. */
typedef struct {
    int32_t n_kv_heads;   /* Hkv */
    int32_t n_q_heads;    /* Hq */
    int32_t head_dim;     /* d */
    int32_t block_tokens; /* Bt, tokens per block and per page (Sec. 3.1, Sec. 5.2) */
    int32_t kv_dtype;     /* kvmem_dtype of the K/V pools */
    float k_scale;        /* KVMEM_FP8_E4M3: K element = decoded code * k_scale (finite, > 0);
                             ignored for the other types */
    float v_scale;        /* KVMEM_FP8_E4M3: V element = decoded code * v_scale (finite, > 0) */
} kvmem_geom;

/* Bytes of one layer's Mean-K index for n_blocks history blocks (the tiled
 * layout rounds the block count up to a multiple of 64).  0 on invalid input. */
size_t kvmem_index_bytes(const kvmem_geom *geom, int32_t n_blocks);

/* Mean-K retrieval index (Eq. 9; Sec. 4.3 "Mean-K Retrieval-Index
 * Construction", Sec. 5.3 "Incremental Indexing").
 *
 * For every block b in [first_block, first_block + n_blocks) and KV head g:
 *   index[b][g][j] = (1/Bt) * sum_{t < Bt} K[block_to_page[b]][g][t][j],
 * summed exactly (fp64) and rounded once to fp32, so the result does not depend
 * on summation order (FP8 pools: the decoded codes are summed exactly, and the
 * sum times k_scale / Bt is rounded once).  Keys are taken as position independent (any RoPE already
 * removed by the caller).  Call it once per layer, with that layer's pool and
 * index; it only writes the rows of the given range, so completed blocks can be
 * indexed incrementally while their keys are resident.
 *
 *   k_pool         dev  [n_pages][Hkv][Bt][d] kv_dtype
 *   n_pages             number of pages in k_pool (> 0)
 *   block_to_page  dev  int32, read at [first_block, first_block + n_blocks)
 *   index          dev  float, one layer in the tiled layout, at least
 *                       kvmem_index_bytes(geom, first_block + n_blocks) bytes
 *   stream              hipStream_t
 * n_blocks == 0 is a no-op.  A page id outside [0, n_pages) yields a NaN row. */
kvmem_status kvmem_build_index(const kvmem_geom *geom, const void *k_pool, int64_t n_pages,
                               const int32_t *block_to_page, int32_t first_block,
                               int32_t n_blocks, float *index, void *stream);

/* ---- Position handling (Sec. 4.3 index construction; Sec. 4.4 execution
 * view; Sec. 5.3 copy-free assembly) ---------------------------------------
 * RoPE in rotate-half form (the paper does not print the variant; this is the
 * form of the Qwen models its engine serves): for j < d/2 the pair
 * (x_j, x_{j+d/2}) at position p turns by the angle p * rope_base^(-2j/d),
 *   (x_j, x_{j+d/2}) -> (x_j cos a - x_{j+d/2} sin a, x_j sin a + x_{j+d/2} cos a).
 * Angles are formed and reduced in fp64 (positions up to 2^62), cos/sin and
 * the rotation are fp32, bf16 results are rounded to nearest even.
 * rope_base must be finite and above 1 (KVMEM_ERR_SHAPE otherwise). */

/* Eq. 9 from keys that carry RoPE (Sec. 4.3: RoPE is removed before the index
 * is built).  As kvmem_build_index, except that token t of block b is stored
 * encoded at position block_pos[b] + t -- its "baked position" (Sec. 5.3) --
 * and is turned back to position 0 before it enters the mean.
 *   block_pos  dev [M] int64, or NULL for the original frame b * Bt + t
 * Blocks whose page is outside the pool get NaN index rows. */
kvmem_status kvmem_build_index_rope(const kvmem_geom *geom, const void *k_pool, int64_t n_pages,
                                    const int32_t *block_to_page, const int64_t *block_pos, double rope_base,
                                    int32_t first_block, int32_t n_blocks, float *index, void *stream);

/* Execution-view materialisation (Sec. 4.4, Sec. 5.3): the keys of a block
 * are valid only at the positions they were encoded for, so a block placed at
 * a new compact position gets its K re-encoded from the position-independent
 * raw K, and V copied unchanged.  For i < n_blocks:
 *   K of page dst_pages[i] of k_dst_pool, token t  = RoPE(raw_k_pool[src_pages[i]] token t,
 *                                                         positions[i] + t)
 *   V of page dst_pages[i] of v_dst_pool            = v_pool[src_pages[i]]
 *   raw_k_pool, v_pool        dev [n_src_pages][Hkv][Bt][d] kv_dtype
 *   k_dst_pool, v_dst_pool    dev [n_dst_pages][Hkv][Bt][d] kv_dtype
 *   src_pages, dst_pages      dev [n_blocks] int32
 *   positions                 dev [n_blocks] int64 (first token's position)
 * A destination page outside its pool is skipped (nothing written); a source
 * page outside its pool makes the destination page all NaN.  Destination
 * pages must be distinct and must not overlap the source pools. */
kvmem_status kvmem_materialize(const kvmem_geom *geom, double rope_base, const void *raw_k_pool,
                               const void *v_pool, int64_t n_src_pages, const int32_t *src_pages,
                               const int64_t *positions, const int32_t *dst_pages, int32_t n_blocks,
                               void *k_dst_pool, void *v_dst_pool, int64_t n_dst_pages, void *stream);

/* Delta re-encoding in place (Sec. 4.4): a GPU-resident block whose compact
 * position moves by delta keeps its page; its K turns by delta positions
 * (every token by the same angle), V is untouched.  Each call rounds K again
 * (bf16): the paper bounds the number of such steps between rebuilds from raw
 * K (kvmem_materialize), which is the caller's policy.
 *   k_pool           dev [n_pages][Hkv][Bt][d] kv_dtype, updated in place
 *   pages            dev [n_list] int32 (distinct); delta_positions dev [n_list] int64
 * Pages outside the pool are skipped.  kvmem_materialize and kvmem_rerope take
 * f32 and bf16 pools; FP8 pools return KVMEM_ERR_UNSUPPORTED (re-encoding would
 * quantise K again). */
kvmem_status kvmem_rerope(const kvmem_geom *geom, double rope_base, void *k_pool, int64_t n_pages,
                          const int32_t *pages, const int64_t *delta_positions, int32_t n_list, void *stream);

/* ---- Working-set update at a recall point (Sec. 4.4 "Retrieval-Aware
 * Hierarchical Reuse", Eq. 11, Eq. 12) --------------------------------------
 * The selected blocks of a recall point (the working set W_t) are placed in a
 * bounded execution pool of P pages, reusing the pages of blocks that are still
 * resident from earlier recalls (the GPU set G).  With W_{t-1} the previous
 * recall's working set:
 *   R_t = W_t & W_{t-1}, L_t = W_t - W_{t-1}, E_t = W_{t-1} - W_t   (Eq. 11)
 *   L_t^physical = W_t - G_{t-1}                                    (Eq. 12)
 * Only L_t^physical is loaded: its raw K is re-encoded at the block's compact
 * position and V copied (as kvmem_materialize).  A resident block keeps its page
 * and V; if its compact position moved, its K is re-encoded in place by the
 * difference (as kvmem_rerope) while the page has had fewer than max_deltas
 * such steps since its K was last built from raw K, else it is rebuilt from raw
 * K.  The paper leaves two choices open; this library takes:
 *   - view block i (view_blocks ascending) sits at first_position + i * Bt;
 *   - the pages for L_t^physical are the pages holding no block of W_t, taken in
 *     clock order from a hand (hand, hand + 1, ... mod P), one per incoming block
 *     in view order; the hand then moves past the last page taken.  A taken
 *     page's previous block leaves G.
 * The repository view is a set of caller-owned device arrays: */
typedef struct {
    int32_t n_blocks;          /* M, history blocks */
    int32_t n_pages;           /* P, pages of the execution pool (<= 2^22) */
    int32_t *block_page;       /* dev [M] execution page of each block, -1 if not resident */
    int32_t *block_last_step;  /* dev [M] last recall step that selected the block, -1 never */
    int32_t *page_block;       /* dev [P] block held by each page, -1 if empty */
    int64_t *page_pos;         /* dev [P] position the page's K is encoded at (its first token) */
    int32_t *page_deltas;      /* dev [P] delta re-encodings since the page's K was built from raw K */
    int32_t *header;           /* dev [8] previous step, |W| at that step, clock hand */
} kvmem_working_set;

/* Empty pool: every block non-resident and never selected, hand at page 0. */
kvmem_status kvmem_working_set_reset(const kvmem_working_set *ws, void *stream);

/* Workspace bytes of kvmem_working_set_update for views of up to n_view blocks. */
size_t kvmem_working_set_workspace_bytes(int32_t n_view, int32_t n_pages);

/* One recall point: steps must increase from call to call (W_{t-1} is the set
 * of the previous call).
 *   view_blocks    dev int32 [n_view], ascending distinct block ids (a kvmem_select
 *                  row); ids outside [0, M) are ignored (counted, page -1)
 *   block_to_page  dev int32 [M] page of each block in raw_k_pool / v_pool
 *   raw_k_pool     dev [n_src_pages][Hkv][Bt][d] position-independent K
 *   v_pool         dev [n_src_pages][Hkv][Bt][d]
 *   k_exec_pool, v_exec_pool  dev [P][Hkv][Bt][d] the execution pool (updated)
 *   exec_pages     dev int32 [n_view] out: execution page of each view block
 *                  (the page table kvmem_sparse_attn reads over the execution pool)
 *   counts         dev int32 [16] out: |W_t|, |R_t|, |L_t|, |E_t|, |L_t^physical|,
 *                  delta re-encodings, rebuilds (delta bound reached), resident
 *                  blocks evicted, ignored ids
 * Requires n_view <= P, max_deltas >= 0, f32 or bf16 pools (FP8 pools return
 * KVMEM_ERR_UNSUPPORTED: re-encoding would quantise K again), and a valid
 * rope_base.  Calls that share the working-set arrays must not overlap. */
kvmem_status kvmem_working_set_update(const kvmem_geom *geom, double rope_base, const kvmem_working_set *ws,
                                      int32_t step, const int32_t *view_blocks, int32_t n_view,
                                      int64_t first_position, int32_t max_deltas, const int32_t *block_to_page,
                                      const void *raw_k_pool, const void *v_pool, int64_t n_src_pages,
                                      void *k_exec_pool, void *v_exec_pool, int32_t *exec_pages, int32_t *counts,
                                      void *workspace, size_t workspace_bytes, void *stream);

/* View plan (Eq. 5, Eq. 7; host only, no HIP call).  With the active budget
 * B_a = min(model_ctx_tokens, gpu_kv_tokens) and the mandatory context of
 * (n_sink + n_recent) * Bt tokens,
 *   k_eff  = min(floor((B_a - (n_sink + n_recent) * Bt) / Bt), M - n_sink - n_recent)
 *   n_view = n_sink + k_eff + n_recent.
 * Returns KVMEM_ERR_BUDGET when B_a is below the mandatory context.  k_eff and
 * n_view (host) may each be NULL. */
kvmem_status kvmem_plan_view(const kvmem_geom *geom, int32_t n_blocks, int32_t n_sink_blocks,
                             int32_t n_recent_blocks, int64_t model_ctx_tokens,
                             int64_t gpu_kv_tokens, int32_t *k_eff, int32_t *n_view);

/* Bytes of workspace kvmem_select needs for these sizes (0 on invalid input). */
size_t kvmem_select_workspace_bytes(const kvmem_geom *geom, int32_t n_layers, int32_t n_q_tokens,
                                    int32_t n_blocks, int32_t n_sink_blocks,
                                    int32_t n_recent_blocks, int32_t mode);

/* Query-conditioned block selection (Eq. 10 and the default selector of
 * Sec. 4.3; budget from Eq. 5 / Eq. 7).
 *
 * The candidate set is C = [n_sink, M - n_recent): the sink blocks [0, n_sink)
 * and the recent blocks [M - n_recent, M) are always kept and are not part of
 * the softmax.  For every layer l, query token m and query head h,
 *   p_{l,m,h,b} = softmax_{b' in C}( scale * q[l][m][h] . index[l][b'][h/G] )_b
 * then R combines them as `mode` states.  The k_eff candidates with the largest
 * fp32 R are selected (ties: lower block id first) and the view is emitted in
 * chronological order:
 *   view_blocks[s] = [0 .. n_sink) ++ ascending(selected) ++ [M - n_recent .. M)
 *   view_pages[s][i] = block_to_page[view_blocks[s][i]]
 *
 *   q              dev  float [n_layers][n_q][Hq][d]
 *   index          dev  float, n_layers consecutive layers in the tiled
 *                       layout, each kvmem_index_bytes(geom, M) bytes
 *   n_blocks            M; requires n_sink + n_recent < M and |C| <= 2^20
 *   model_ctx_tokens, gpu_kv_tokens   B_model and B_gpu of Eq. 5
 *   mode                kvmem_reduce
 *   scale               logit scale; <= 0 selects 1/sqrt(d)
 *   block_to_page  dev  int32 [M]
 *   view_blocks    dev  int32 [n_sel][n_view]  (n_sel = 1, or n_layers*Hkv)
 *   view_pages     dev  int32 [n_sel][n_view]
 *   scores         dev  float [n_sel][M] or NULL: R per block, rounded to
 *                       fp32; reserved blocks hold +inf
 *   n_view_out     host int32 or NULL: receives n_view (known before launch)
 *   workspace      dev  >= kvmem_select_workspace_bytes(...)
 *   stream              hipStream_t */
kvmem_status kvmem_select(const kvmem_geom *geom, int32_t n_layers, const float *q,
                          int32_t n_q_tokens, const float *index, int32_t n_blocks,
                          int32_t n_sink_blocks, int32_t n_recent_blocks,
                          int64_t model_ctx_tokens, int64_t gpu_kv_tokens, int32_t mode,
                          float scale, const int32_t *block_to_page, int32_t *view_blocks,
                          int32_t *view_pages, float *scores, int32_t *n_view_out,
                          void *workspace, size_t workspace_bytes, void *stream);

/* kvmem_select without a caller workspace, for callers that cannot allocate
 * device memory around the call (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc).  Arguments, results and errors are
 * those of kvmem_select; the scratch space is a device array inside the library
 * (one per GPU, KVMEM_SELECT_NOALLOC_MAX_BYTES, held until the process ends),
 * so the call never allocates or frees memory.  A selection whose workspace
 * (kvmem_select_workspace_bytes) exceeds that size returns KVMEM_ERR_WORKSPACE
 * -- 16 MiB covers a decode step's selection over 2^20 candidates at 32 query
 * rows, not a recall point's thousands of rows.  `stream` must run on the
 * current device (KVMEM_ERR_UNSUPPORTED otherwise).  Every call on one GPU
 * uses the same scratch: calls that overlap in time on one GPU (other streams,
 * other threads) race and must be serialised by the caller. */
#define KVMEM_SELECT_NOALLOC_MAX_BYTES (16u << 20)
kvmem_status kvmem_select_noalloc(const kvmem_geom *geom, int32_t n_layers, const float *q,
                                  int32_t n_q_tokens, const float *index, int32_t n_blocks,
                                  int32_t n_sink_blocks, int32_t n_recent_blocks,
                                  int64_t model_ctx_tokens, int64_t gpu_kv_tokens, int32_t mode,
                                  float scale, const int32_t *block_to_page, int32_t *view_blocks,
                                  int32_t *view_pages, float *scores, int32_t *n_view_out, void *stream);

/* Bytes of workspace kvmem_sparse_attn needs for these sizes (0 on invalid input). */
size_t kvmem_sparse_attn_workspace_bytes(const kvmem_geom *geom, int32_t n_q_tokens,
                                         int32_t n_sel, int32_t n_view);

/* Decode attention over the execution view (Sec. 4.4: the view maps the
 * selected blocks' physical pages through a page table instead of copying
 * them; Sec. 5.3 "Copy-free execution-view assembly").
 *
 * For query token m and query head h, with KV head g = h / G and view row
 * s = (n_sel == 1 ? 0 : g), the keys are every token of the pages
 * view_pages[s][0 .. n_view), in that order, except that the final page holds
 * only last_page_tokens tokens:
 *   a_t = scale * q[m][h] . K_t,   out[m][h] = sum_t softmax(a)_t V_t,
 *   lse[m][h] = log sum_t exp(a_t)   (natural log).
 * The view is split across workgroups (split-K) and the partial results are
 * merged exactly through their log-sum-exp.  All n_q query tokens attend to the
 * same view (no mask among them).
 *
 *   q              dev  float [n_q][Hq][d]   one layer
 *   k_pool, v_pool dev  [n_pages][Hkv][Bt][d] kv_dtype (FP8: K_t and V_t are
 *                       the decoded codes times k_scale and v_scale)
 *   view_pages     dev  int32 [n_sel][n_view], n_sel = 1 or Hkv
 *   last_page_tokens    1 .. Bt
 *   scale               <= 0 selects 1/sqrt(d)
 *   out            dev  float [n_q][Hq][d]
 *   lse            dev  float [n_q][Hq] or NULL
 *   workspace      dev  >= kvmem_sparse_attn_workspace_bytes(...)
 *   stream              hipStream_t */
kvmem_status kvmem_sparse_attn(const kvmem_geom *geom, const float *q, int32_t n_q_tokens,
                               const void *k_pool, const void *v_pool, int64_t n_pages,
                               const int32_t *view_pages, int32_t n_sel, int32_t n_view,
                               int32_t last_page_tokens, float scale, float *out, float *lse,
                               void *workspace, size_t workspace_bytes, void *stream);

/* Description of the last error on the calling thread ("" after success).
 * Valid until the next call on that thread. */
const char *kvmem_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KVMEM_H */
