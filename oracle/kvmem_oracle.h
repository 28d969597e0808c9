/*
 * kvmem_oracle.h -- CPU oracle for the KVMem per-decode-step path.
 *
 * TEST INFRASTRUCTURE ONLY.  This is a plain, slow, fp64 definition of what the
 * GPU path computes.  Only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg may call it.  It shares no code, header, table or helper
 * with the HIP library, and it never includes that library's header.
 *
 * Paper: "KVMem" (arXiv 2609.04852).  Every entry point cites the passage of
 * the paper it follows.  Layouts (all row-major, C order):
 *   K/V page pool   [n_pages][n_kv_heads][block_tokens][head_dim]  element type kv_type:
 *                   0 fp32, 1 bf16 bits, 2 fp64
 *   Mean-K index    [n_layers][n_blocks][n_kv_heads][head_dim]      float
 *   query           [n_layers][n_q][n_q_heads][head_dim]            float
 *   relevance       [n_sel][n_blocks]                                double
 *   view tables     [n_sel][n_view]                                  int32
 *
 * Readings of the paper that these functions fix (also listed in the design
 * notes): candidates exclude the sink and recent blocks; ties are broken by the
 * lower block id; the ranking decision is taken on scores rounded to fp32;
 * query head h belongs to KV head floor(h / G); scoring and attention take
 * keys and queries as given (position independent, or already encoded at the
 * positions the caller chose); the RoPE functions below move them between
 * frames.
 *
 * Return value of every int function: 0 on success, -1 on bad arguments.
 */
#ifndef KVMEM_ORACLE_H
#define KVMEM_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Reduction across query tokens, layers and heads (Eq. 10). */
#define ORACLE_MEAN_ALL 0  /* R_b = sum_m mean_{l,h} softmax(...)_b; one selection  */
#define ORACLE_MAX_GROUP 1 /* R[l][g][b] = max_{m, h in g} softmax(...)_b; L*Hkv selections */

/* Eq. 9 (Sec. 4.3, Mean-K retrieval-index construction): the index entry of a
 * block is the mean of the block's keys, per layer and KV head.  Sum in fp64,
 * divide by block_tokens in fp64, round once to fp32.  Rows
 * [first_block, first_block + n_blocks) of `index` ([*][Hkv][d]) are written;
 * block b reads page block_to_page[b] of k_pool. */
int oracle_mean_k(int n_kv_heads, int block_tokens, int head_dim, int kv_type,
                  const void *k_pool, int64_t n_pages, const int32_t *block_to_page,
                  int32_t first_block, int32_t n_blocks, float *index);

/* Positional encoding (Sec. 4.3: keys are freed of RoPE before the index is
 * built; Sec. 4.4 and Sec. 5.3: selected blocks are given contiguous positions
 * in the compact execution window and their keys re-encoded there).  The
 * paper does not print the RoPE variant; these functions use the rotate-half
 * form of the Qwen models its engine serves: for j < d/2 the pair
 * (x_j, x_{j+d/2}) at position p is rotated by the angle p * base^(-2j/d),
 *   (x_j, x_{j+d/2}) -> (x_j cos a - x_{j+d/2} sin a, x_j sin a + x_{j+d/2} cos a).
 * A negative position undoes the rotation.  Angles, cos and sin in fp64. */

/* Rotate each row of x [n_rows][head_dim] to the position pos[row]; out may
 * alias x. */
int oracle_rope(int64_t n_rows, int head_dim, const double *x, const int64_t *pos, double base,
                double *out);

/* Eq. 9 over position-independent keys, from a pool whose keys carry RoPE:
 * token t of block b sits at position block_pos[b] + t (block_pos NULL: the
 * block's original frame b * block_tokens + t), is rotated back to position
 * 0 in fp64, and the block's mean is rounded once to fp32 (index layout as
 * oracle_mean_k). */
int oracle_mean_k_rope(int n_kv_heads, int block_tokens, int head_dim, int kv_type,
                       const void *k_pool, int64_t n_pages, const int32_t *block_to_page,
                       const int64_t *block_pos, double base, int32_t first_block, int32_t n_blocks,
                       float *index);

/* Eq. 5 and Eq. 7 (Sec. 3.1): B_a = min(B_model, B_gpu); the mandatory context
 * is the sink and recent blocks; the remaining budget holds
 * floor((B_a - (S+Rr)*Bt) / Bt) historical blocks, capped by |C| = M - S - Rr.
 * Returns k_eff >= 0, or -1 when B_a cannot hold the mandatory context or the
 * shape is invalid. */
int64_t oracle_k_eff(int64_t model_ctx_tokens, int64_t gpu_kv_tokens, int block_tokens,
                     int32_t n_blocks, int32_t n_sink, int32_t n_recent);

/* Eq. 10 (Sec. 4.3, query-conditioned block scoring).  For every (l, m, h):
 * logits s_b = scale * q[l][m][h] . index[l][b][g(h)] over the candidate set
 * C = [n_sink, n_blocks - n_recent), softmax over C, then reduce:
 *   ORACLE_MEAN_ALL : R[0][b] = sum_m (1/(L*Hq)) sum_{l,h} p_{l,m,h,b}
 *   ORACLE_MAX_GROUP: R[l*Hkv+g][b] = max_{m, h: g(h)=g} p_{l,m,h,b}
 * scale <= 0 selects 1/sqrt(head_dim).  Entries of R for the reserved (sink and
 * recent) blocks are set to +inf.  All arithmetic in fp64. */
int oracle_block_relevance(int n_layers, int n_q, int n_q_heads, int n_kv_heads, int head_dim,
                           const float *q, const float *index, int32_t n_blocks,
                           int32_t n_sink, int32_t n_recent, int mode, double scale,
                           double *relevance);

/* Selector (Sec. 4.3, last paragraph of block scoring; Sec. 5.2): keep the sink
 * blocks [0,S) and the recent blocks [M-Rr,M), fill k_eff slots with the
 * candidates of largest R -- each R is first rounded to fp32, ties go to the
 * lower block id -- and emit the view in chronological (ascending) order:
 *   view_blocks[s] = [0..S) ++ sorted(selected) ++ [M-Rr..M),
 *   view_pages[s][i] = block_to_page[view_blocks[s][i]].
 * n_view = S + k_eff + Rr. */
int oracle_select(int n_sel, const double *relevance, int32_t n_blocks, int32_t n_sink,
                  int32_t n_recent, int64_t k_eff, const int32_t *block_to_page,
                  int32_t *view_blocks, int32_t *view_pages);

/* Decode attention over the execution view through its page table (Sec. 4.4
 * execution view; Sec. 5.3 copy-free execution-view assembly).  For each query
 * token m and query head h (KV head g = h / G, view row s = 0 if n_sel == 1,
 * else g): a_t = scale * q[m][h] . K[page][g][t] over every token of every view
 * page (the final view page holds only last_page_tokens tokens),
 * out[m][h] = sum_t softmax(a)_t V[page][g][t], lse[m][h] = log sum_t exp(a_t).
 * q is one layer: [n_q][Hq][d].  Outputs are fp64. */
int oracle_view_attention(int n_q, int n_q_heads, int n_kv_heads, int head_dim,
                          int block_tokens, int kv_type, const float *q,
                          const void *k_pool, const void *v_pool, int64_t n_pages,
                          const int32_t *view_pages, int n_sel, int32_t n_view,
                          int32_t last_page_tokens, double scale, double *out, double *lse);

/* The same attention written as dense attention over the whole history with
 * every block outside the view masked to -inf: iterate blocks b = 0..M-1 in
 * chronological order through block_to_page, and keep the keys of blocks that
 * appear in view_blocks[s].  The final view block (view_blocks[s][n_view-1])
 * keeps only last_page_tokens tokens.  Outputs are fp64. */
int oracle_masked_dense_attention(int n_q, int n_q_heads, int n_kv_heads, int head_dim,
                                  int block_tokens, int kv_type, const float *q,
                                  const void *k_pool, const void *v_pool, int64_t n_pages,
                                  const int32_t *block_to_page, int32_t n_blocks,
                                  const int32_t *view_blocks, int n_sel, int32_t n_view,
                                  int32_t last_page_tokens, double scale, double *out,
                                  double *lse);

/* Number of OpenMP threads the oracle uses (1 when built without OpenMP). */
int oracle_num_threads(void);

#ifdef __cplusplus
}
#endif

#endif /* KVMEM_ORACLE_H */
