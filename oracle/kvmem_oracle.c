/*
 * kvmem_oracle.c -- CPU oracle for the KVMem per-decode-step path.
 *
 * TEST INFRASTRUCTURE ONLY: a plain fp64 definition of the method, written
 * from the paper (KVMem, arXiv 2609.04852).  It is used by the test suite, the
 * smoke check and the benchmark's CPU-baseline leg, and by nothing else.  It
 * shares no code with the HIP library.  Loops are written in the order the
 * paper's definitions read; OpenMP only splits independent outputs across
 * threads and never changes the order of any sum.
 *
 * Build: gcc -O2 -ffp-contract=off -fopenmp -shared -fPIC (see build.py).
 */
#include "kvmem_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Widen one stored K/V element to fp64 (pool element type: 0 fp32, 1 bf16
 * bits, 2 fp64).  A bf16 value is the top half of the fp32 with the same
 * bits, so every widening is exact.  (FP8 pools reach the oracle decoded to
 * fp64, see the Python wrapper.) */
static double load_elem(const void *pool, int kv_type, int64_t i) {
    if (kv_type == 1) {
        uint32_t bits = (uint32_t)((const uint16_t *)pool)[i] << 16;
        float f;
        memcpy(&f, &bits, sizeof f);
        return (double)f;
    }
    if (kv_type == 2) return ((const double *)pool)[i];
    return (double)((const float *)pool)[i];
}

/* Offset of element (page, g, t, j) in a [P][Hkv][Bt][d] pool. */
static int64_t pool_offset(int64_t page, int g, int t, int j, int n_kv_heads, int block_tokens,
                           int head_dim) {
    return ((page * n_kv_heads + g) * (int64_t)block_tokens + t) * head_dim + j;
}

/* ---- Eq. 9: Mean-K block summary ------------------------------------- */
int oracle_mean_k(int n_kv_heads, int block_tokens, int head_dim, int kv_type,
                  const void *k_pool, int64_t n_pages, const int32_t *block_to_page,
                  int32_t first_block, int32_t n_blocks, float *index) {
    if (!k_pool || !block_to_page || !index || n_kv_heads <= 0 || block_tokens <= 0 ||
        head_dim <= 0 || first_block < 0 || n_blocks < 0)
        return -1;
    for (int32_t i = 0; i < n_blocks; ++i) {
        int64_t page = block_to_page[first_block + i];
        if (page < 0 || page >= n_pages) return -1;
    }
#pragma omp parallel for schedule(static)
    for (int32_t i = 0; i < n_blocks; ++i) {
        int32_t b = first_block + i;
        int64_t page = block_to_page[b];
        for (int g = 0; g < n_kv_heads; ++g) {
            for (int j = 0; j < head_dim; ++j) {
                double sum = 0.0;
                for (int t = 0; t < block_tokens; ++t)
                    sum += load_elem(k_pool, kv_type,
                                     pool_offset(page, g, t, j, n_kv_heads, block_tokens, head_dim));
                double mean = sum / (double)block_tokens;
                index[((int64_t)b * n_kv_heads + g) * head_dim + j] = (float)mean;
            }
        }
    }
    return 0;
}

/* ---- Position handling (Sec. 4.3 index construction; Sec. 4.4 execution
 * view; Sec. 5.3 copy-free assembly): RoPE in rotate-half form --------- */

/* Angle of pair j at position p: p * base^(-2j/d). */
static double rope_angle(int64_t pos, int j, int head_dim, double base) {
    return (double)pos * pow(base, -2.0 * (double)j / (double)head_dim);
}

/* Rotate one row x[d] to position `pos` (in place): the pair (x_j, x_{j+d/2})
 * becomes (x_j cos a - x_{j+d/2} sin a, x_j sin a + x_{j+d/2} cos a). */
static void rope_row(double *x, int64_t pos, int head_dim, double base) {
    int h = head_dim / 2;
    for (int j = 0; j < h; ++j) {
        double a = rope_angle(pos, j, head_dim, base);
        double c = cos(a), s = sin(a);
        double x0 = x[j], x1 = x[j + h];
        x[j] = x0 * c - x1 * s;
        x[j + h] = x0 * s + x1 * c;
    }
}

int oracle_rope(int64_t n_rows, int head_dim, const double *x, const int64_t *pos, double base,
                double *out) {
    if (!x || !pos || !out || n_rows < 0 || head_dim <= 0 || head_dim % 2 || !(base > 0.0)) return -1;
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < n_rows; ++r) {
        double *y = out + r * head_dim;
        if (y != x + r * head_dim) memcpy(y, x + r * head_dim, sizeof(double) * (size_t)head_dim);
        rope_row(y, pos[r], head_dim, base);
    }
    return 0;
}

int oracle_mean_k_rope(int n_kv_heads, int block_tokens, int head_dim, int kv_type,
                       const void *k_pool, int64_t n_pages, const int32_t *block_to_page,
                       const int64_t *block_pos, double base, int32_t first_block, int32_t n_blocks,
                       float *index) {
    if (!k_pool || !block_to_page || !index || n_kv_heads <= 0 || block_tokens <= 0 ||
        head_dim <= 0 || head_dim % 2 || first_block < 0 || n_blocks < 0 || !(base > 0.0))
        return -1;
    for (int32_t i = 0; i < n_blocks; ++i) {
        int64_t page = block_to_page[first_block + i];
        if (page < 0 || page >= n_pages) return -1;
    }
#pragma omp parallel
    {
        double *row = (double *)malloc(sizeof(double) * (size_t)head_dim);
        double *sum = (double *)malloc(sizeof(double) * (size_t)head_dim);
#pragma omp for schedule(static)
        for (int32_t i = 0; i < n_blocks; ++i) {
            int32_t b = first_block + i;
            int64_t page = block_to_page[b];
            int64_t p0 = block_pos ? block_pos[b] : (int64_t)b * block_tokens;
            for (int g = 0; g < n_kv_heads; ++g) {
                for (int j = 0; j < head_dim; ++j) sum[j] = 0.0;
                for (int t = 0; t < block_tokens; ++t) {
                    /* the stored key carries RoPE at p0 + t: rotate it back */
                    for (int j = 0; j < head_dim; ++j)
                        row[j] = load_elem(k_pool, kv_type,
                                           pool_offset(page, g, t, j, n_kv_heads, block_tokens, head_dim));
                    rope_row(row, -(p0 + t), head_dim, base);
                    for (int j = 0; j < head_dim; ++j) sum[j] += row[j];
                }
                for (int j = 0; j < head_dim; ++j)
                    index[((int64_t)b * n_kv_heads + g) * head_dim + j] = (float)(sum[j] / (double)block_tokens);
            }
        }
        free(row);
        free(sum);
    }
    return 0;
}

/* ---- Eq. 5 / Eq. 7: active budget -> number of selectable blocks ------- */
int64_t oracle_k_eff(int64_t model_ctx_tokens, int64_t gpu_kv_tokens, int block_tokens,
                     int32_t n_blocks, int32_t n_sink, int32_t n_recent) {
    if (block_tokens <= 0 || n_blocks < 0 || n_sink < 0 || n_recent < 0 ||
        n_sink + n_recent > n_blocks)
        return -1;
    int64_t b_a = model_ctx_tokens < gpu_kv_tokens ? model_ctx_tokens : gpu_kv_tokens; /* Eq. 5 */
    int64_t mandatory = (int64_t)(n_sink + n_recent) * block_tokens;                   /* N(Q) */
    if (b_a < mandatory) return -1;
    int64_t k = (b_a - mandatory) / block_tokens; /* Eq. 7: N(Q) + Bt |R| <= B_a */
    int64_t n_cand = (int64_t)n_blocks - n_sink - n_recent;
    return k < n_cand ? k : n_cand;
}

/* ---- Eq. 10: query-conditioned block relevance ------------------------ */
int oracle_block_relevance(int n_layers, int n_q, int n_q_heads, int n_kv_heads, int head_dim,
                           const float *q, const float *index, int32_t n_blocks,
                           int32_t n_sink, int32_t n_recent, int mode, double scale,
                           double *relevance) {
    if (!q || !index || !relevance || n_layers <= 0 || n_q <= 0 || n_kv_heads <= 0 ||
        n_q_heads <= 0 || n_q_heads % n_kv_heads != 0 || head_dim <= 0 || n_sink < 0 ||
        n_recent < 0 || n_sink + n_recent >= n_blocks ||
        (mode != ORACLE_MEAN_ALL && mode != ORACLE_MAX_GROUP))
        return -1;
    const int group = n_q_heads / n_kv_heads;
    const int32_t c_lo = n_sink, c_hi = n_blocks - n_recent; /* candidate set C */
    const int32_t n_cand = c_hi - c_lo;
    const int n_rows = n_layers * n_q * n_q_heads;
    const int n_sel = mode == ORACLE_MEAN_ALL ? 1 : n_layers * n_kv_heads;
    if (scale <= 0.0) scale = 1.0 / sqrt((double)head_dim);

    /* softmax_{b' in C}(q . kbar / sqrt(d)) for every (l, m, h), kept per row */
    double *prob = (double *)malloc(sizeof(double) * (size_t)n_rows * (size_t)n_cand);
    if (!prob) return -1;

#pragma omp parallel for schedule(dynamic, 1)
    for (int row = 0; row < n_rows; ++row) {
        int l = row / (n_q * n_q_heads);
        int h = row % n_q_heads;
        int g = h / group; /* GQA: query head h reads KV head floor(h/G) */
        const float *qv = q + (int64_t)row * head_dim; /* rows are [l][m][h] in order */
        double *p = prob + (int64_t)row * n_cand;
        double mx = -INFINITY;
        for (int32_t b = c_lo; b < c_hi; ++b) {
            const float *kb = index + (((int64_t)l * n_blocks + b) * n_kv_heads + g) * head_dim;
            double s = 0.0;
            for (int j = 0; j < head_dim; ++j) s += (double)qv[j] * (double)kb[j];
            s *= scale;
            p[b - c_lo] = s;
            if (s > mx) mx = s;
        }
        double z = 0.0;
        for (int32_t c = 0; c < n_cand; ++c) {
            p[c] = exp(p[c] - mx);
            z += p[c];
        }
        for (int32_t c = 0; c < n_cand; ++c) p[c] /= z;
    }

    for (int s = 0; s < n_sel; ++s)
        for (int32_t b = 0; b < n_blocks; ++b)
            relevance[(int64_t)s * n_blocks + b] = (b >= c_lo && b < c_hi) ? 0.0 : INFINITY;

    if (mode == ORACLE_MEAN_ALL) {
        /* R_b = sum_m mean_{l,h} p_{l,m,h,b} */
        double *r = relevance;
        for (int m = 0; m < n_q; ++m) {
            for (int32_t c = 0; c < n_cand; ++c) {
                double acc = 0.0;
                for (int l = 0; l < n_layers; ++l)
                    for (int h = 0; h < n_q_heads; ++h)
                        acc += prob[((int64_t)(l * n_q + m) * n_q_heads + h) * n_cand + c];
                r[c_lo + c] += acc / (double)(n_layers * n_q_heads);
            }
        }
    } else {
        /* R[l][g][b] = max over m and over the query heads h of group g */
        for (int l = 0; l < n_layers; ++l)
            for (int g = 0; g < n_kv_heads; ++g) {
                double *r = relevance + (int64_t)(l * n_kv_heads + g) * n_blocks;
                for (int32_t c = 0; c < n_cand; ++c) {
                    double best = 0.0;
                    for (int m = 0; m < n_q; ++m)
                        for (int h = g * group; h < (g + 1) * group; ++h) {
                            double v = prob[((int64_t)(l * n_q + m) * n_q_heads + h) * n_cand + c];
                            if (v > best) best = v;
                        }
                    r[c_lo + c] = best;
                }
            }
    }
    free(prob);
    return 0;
}

/* ---- Selector: reserve sink + recent, top-k by R, chronological view ---- */
typedef struct {
    float key;
    int32_t block;
} ranked_t;

/* Order by larger fp32 score first, then by lower block id. */
static int cmp_ranked(const void *pa, const void *pb) {
    const ranked_t *a = (const ranked_t *)pa, *b = (const ranked_t *)pb;
    if (a->key > b->key) return -1;
    if (a->key < b->key) return 1;
    return (a->block > b->block) - (a->block < b->block);
}

static int cmp_i32(const void *pa, const void *pb) {
    int32_t a = *(const int32_t *)pa, b = *(const int32_t *)pb;
    return (a > b) - (a < b);
}

int oracle_select(int n_sel, const double *relevance, int32_t n_blocks, int32_t n_sink,
                  int32_t n_recent, int64_t k_eff, const int32_t *block_to_page,
                  int32_t *view_blocks, int32_t *view_pages) {
    if (!relevance || !block_to_page || !view_blocks || !view_pages || n_sel <= 0 ||
        n_sink < 0 || n_recent < 0 || n_sink + n_recent > n_blocks || k_eff < 0 ||
        k_eff > (int64_t)n_blocks - n_sink - n_recent)
        return -1;
    const int32_t c_lo = n_sink, c_hi = n_blocks - n_recent;
    const int32_t n_cand = c_hi - c_lo;
    const int64_t n_view = n_sink + k_eff + n_recent;
    ranked_t *cand = (ranked_t *)malloc(sizeof(ranked_t) * (size_t)(n_cand > 0 ? n_cand : 1));
    int32_t *chosen = (int32_t *)malloc(sizeof(int32_t) * (size_t)(k_eff > 0 ? k_eff : 1));
    if (!cand || !chosen) {
        free(cand);
        free(chosen);
        return -1;
    }
    for (int s = 0; s < n_sel; ++s) {
        const double *r = relevance + (int64_t)s * n_blocks;
        for (int32_t c = 0; c < n_cand; ++c) {
            cand[c].key = (float)r[c_lo + c]; /* the decision is taken on fp32 scores */
            cand[c].block = c_lo + c;
        }
        qsort(cand, (size_t)n_cand, sizeof(ranked_t), cmp_ranked);
        for (int64_t i = 0; i < k_eff; ++i) chosen[i] = cand[i].block;
        qsort(chosen, (size_t)k_eff, sizeof(int32_t), cmp_i32); /* chronological order */
        int32_t *vb = view_blocks + (int64_t)s * n_view;
        int64_t o = 0;
        for (int32_t b = 0; b < n_sink; ++b) vb[o++] = b;
        for (int64_t i = 0; i < k_eff; ++i) vb[o++] = chosen[i];
        for (int32_t b = c_hi; b < n_blocks; ++b) vb[o++] = b;
        for (int64_t i = 0; i < n_view; ++i)
            view_pages[(int64_t)s * n_view + i] = block_to_page[vb[i]];
    }
    free(cand);
    free(chosen);
    return 0;
}

/* ---- Attention over a set of keys, two-pass softmax in fp64 ------------ */
/* a[t] is the scaled logit of token t (-inf when masked); v_row[t] is the pool
 * offset of that token's value row.  out = sum_t softmax(a)_t V_t,
 * lse = log sum_t exp(a_t). */
static void attend(int64_t n_tok, const double *a, const int64_t *v_row, const void *v_pool,
                   int kv_type, int head_dim, double *out, double *lse) {
    double mx = -INFINITY;
    for (int64_t t = 0; t < n_tok; ++t)
        if (a[t] > mx) mx = a[t];
    double z = 0.0;
    for (int j = 0; j < head_dim; ++j) out[j] = 0.0;
    for (int64_t t = 0; t < n_tok; ++t) {
        double w = exp(a[t] - mx); /* exp(-inf) = 0 for masked tokens */
        z += w;
        for (int j = 0; j < head_dim; ++j) out[j] += w * load_elem(v_pool, kv_type, v_row[t] + j);
    }
    for (int j = 0; j < head_dim; ++j) out[j] /= z;
    *lse = mx + log(z);
}

int oracle_view_attention(int n_q, int n_q_heads, int n_kv_heads, int head_dim,
                          int block_tokens, int kv_type, const float *q,
                          const void *k_pool, const void *v_pool, int64_t n_pages,
                          const int32_t *view_pages, int n_sel, int32_t n_view,
                          int32_t last_page_tokens, double scale, double *out, double *lse) {
    if (!q || !k_pool || !v_pool || !view_pages || !out || !lse || n_q <= 0 ||
        n_kv_heads <= 0 || n_q_heads % n_kv_heads != 0 || head_dim <= 0 || block_tokens <= 0 ||
        n_view <= 0 || last_page_tokens < 1 || last_page_tokens > block_tokens ||
        (n_sel != 1 && n_sel != n_kv_heads))
        return -1;
    for (int64_t i = 0; i < (int64_t)n_sel * n_view; ++i)
        if (view_pages[i] < 0 || view_pages[i] >= n_pages) return -1;
    const int group = n_q_heads / n_kv_heads;
    const int64_t n_tok = (int64_t)(n_view - 1) * block_tokens + last_page_tokens;
    if (scale <= 0.0) scale = 1.0 / sqrt((double)head_dim);
    int bad = 0;

#pragma omp parallel for schedule(dynamic, 1)
    for (int row = 0; row < n_q * n_q_heads; ++row) {
        int h = row % n_q_heads, g = h / group, s = n_sel == 1 ? 0 : g;
        const float *qv = q + (int64_t)row * head_dim;
        double *a = (double *)malloc(sizeof(double) * (size_t)n_tok);
        int64_t *v_row = (int64_t *)malloc(sizeof(int64_t) * (size_t)n_tok);
        if (!a || !v_row) {
#pragma omp atomic write
            bad = 1;
            free(a);
            free(v_row);
            continue;
        }
        int64_t t_out = 0;
        for (int32_t v = 0; v < n_view; ++v) {
            int64_t page = view_pages[(int64_t)s * n_view + v];
            int nt = v == n_view - 1 ? last_page_tokens : block_tokens;
            for (int t = 0; t < nt; ++t, ++t_out) {
                int64_t base = pool_offset(page, g, t, 0, n_kv_heads, block_tokens, head_dim);
                double dot = 0.0;
                for (int j = 0; j < head_dim; ++j)
                    dot += (double)qv[j] * load_elem(k_pool, kv_type, base + j);
                a[t_out] = scale * dot;
                v_row[t_out] = base;
            }
        }
        attend(n_tok, a, v_row, v_pool, kv_type, head_dim, out + (int64_t)row * head_dim,
               lse + row);
        free(a);
        free(v_row);
    }
    return bad ? -1 : 0;
}

int oracle_masked_dense_attention(int n_q, int n_q_heads, int n_kv_heads, int head_dim,
                                  int block_tokens, int kv_type, const float *q,
                                  const void *k_pool, const void *v_pool, int64_t n_pages,
                                  const int32_t *block_to_page, int32_t n_blocks,
                                  const int32_t *view_blocks, int n_sel, int32_t n_view,
                                  int32_t last_page_tokens, double scale, double *out,
                                  double *lse) {
    if (!q || !k_pool || !v_pool || !block_to_page || !view_blocks || !out || !lse ||
        n_q <= 0 || n_kv_heads <= 0 || n_q_heads % n_kv_heads != 0 || head_dim <= 0 ||
        block_tokens <= 0 || n_blocks <= 0 || n_view <= 0 || last_page_tokens < 1 ||
        last_page_tokens > block_tokens || (n_sel != 1 && n_sel != n_kv_heads))
        return -1;
    for (int32_t b = 0; b < n_blocks; ++b)
        if (block_to_page[b] < 0 || block_to_page[b] >= n_pages) return -1;
    for (int64_t i = 0; i < (int64_t)n_sel * n_view; ++i)
        if (view_blocks[i] < 0 || view_blocks[i] >= n_blocks) return -1;
    const int group = n_q_heads / n_kv_heads;
    const int64_t n_tok = (int64_t)n_blocks * block_tokens;
    if (scale <= 0.0) scale = 1.0 / sqrt((double)head_dim);
    int bad = 0;

#pragma omp parallel for schedule(dynamic, 1)
    for (int row = 0; row < n_q * n_q_heads; ++row) {
        int h = row % n_q_heads, g = h / group, s = n_sel == 1 ? 0 : g;
        const float *qv = q + (int64_t)row * head_dim;
        const int32_t *vb = view_blocks + (int64_t)s * n_view;
        char *in_view = (char *)calloc((size_t)n_blocks, 1);
        double *a = (double *)malloc(sizeof(double) * (size_t)n_tok);
        int64_t *v_row = (int64_t *)malloc(sizeof(int64_t) * (size_t)n_tok);
        if (!in_view || !a || !v_row) {
#pragma omp atomic write
            bad = 1;
            free(in_view);
            free(a);
            free(v_row);
            continue;
        }
        for (int32_t i = 0; i < n_view; ++i) in_view[vb[i]] = 1;
        const int32_t tail_block = vb[n_view - 1];
        for (int32_t b = 0; b < n_blocks; ++b) {
            int64_t page = block_to_page[b];
            for (int t = 0; t < block_tokens; ++t) {
                int64_t ti = (int64_t)b * block_tokens + t;
                int keep = in_view[b] && !(b == tail_block && t >= last_page_tokens);
                int64_t base = pool_offset(page, g, t, 0, n_kv_heads, block_tokens, head_dim);
                double dot = 0.0;
                for (int j = 0; j < head_dim; ++j)
                    dot += (double)qv[j] * load_elem(k_pool, kv_type, base + j);
                a[ti] = keep ? scale * dot : -INFINITY;
                v_row[ti] = base;
            }
        }
        attend(n_tok, a, v_row, v_pool, kv_type, head_dim, out + (int64_t)row * head_dim,
               lse + row);
        free(in_view);
        free(a);
        free(v_row);
    }
    return bad ? -1 : 0;
}
