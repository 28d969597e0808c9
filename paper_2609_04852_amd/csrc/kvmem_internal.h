// Internal declarations of the KVMem HIP library: workspace plans and kernel
// launchers.  Host code in kvmem_api.cpp validates arguments, then calls these.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>
#include <math.h>

namespace kvmem {

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// ---- Mean-K index layout -------------------------------------------------
// The index of one layer is stored in tiles of 64 blocks:
//   float [ceil(M/64)][Hkv][d/4][64][4]
// so that, for one KV head and one 4-float slice of the head dimension, the
// 64 blocks of a tile are 1 KB of contiguous memory: a wave scores 64 blocks
// with one lane per block and fully coalesced 16-byte loads.
constexpr int kIndexTile = 64;
__host__ __device__ inline int64_t index_tiles(int64_t n_blocks) { return (n_blocks + kIndexTile - 1) / kIndexTile; }
__host__ __device__ inline int64_t index_layer_floats(int64_t n_blocks, int n_kv_heads, int head_dim) {
    return index_tiles(n_blocks) * kIndexTile * n_kv_heads * head_dim;
}

// ---- select ------------------------------------------------------------
// Index tiles scored by one workgroup of the vector logit kernel (one per
// wave), of the 16-row kernel (each wave takes one 16-block group of each),
// and of the kernel for more rows.  Up to kScoreVectorRows query rows per KV
// head are scored on the vector units, 9 to 16 on the 16-row matrix-core
// kernel (rows past the head's count padded with zero queries), more by
// 16-row chunks.
constexpr int kScoreTilesPerGroup = 4;
constexpr int kScoreVectorRows = 8;
// The 16-row kernel's waves are persistent: about kMfma16Waves of them over
// all (layer, KV head) pairs, four per workgroup, each leaving one partial.
constexpr int kMfma16Waves = 2048;
// More than 16 query rows per KV head (a recall point's prefill query): one
// workgroup per index tile runs every row of its (layer, KV head) in chunks of
// 16 on the matrix cores; the block relevance then sums the rows in
// partitions of about kReduceRowsPerPart rows (at most kReduceMaxParts).
constexpr int kRowsMaxPerHead = 4096;
constexpr int kReduceRowsPerPart = 512;
constexpr int kReduceMaxParts = 64;
// Small selections merge the per-tile (max, sum exp) pairs of their rows
// inside the reduction (no separate stats launch) when a relevance value has at
// most kFusedStatsRows logit rows behind it, each row has at most
// kFusedStatsParts pairs and all of them together at most kFusedStatsPairs;
// the vector logits kernel then clears the histograms. (At 32 rows x 16 pairs,
// 64K tokens, this saves 2 us a step; at 32 x 64 the merge costs more than the
// launch it replaces.)
constexpr int kFusedStatsRows = 64;
constexpr int kFusedStatsParts = 64;
constexpr int kFusedStatsPairs = 1024;
// A vector logits launch of at most kLogitsBatchGroups workgroups (one per
// compute unit) issues all of a tile's loads before its first product: with
// so few waves each one's chain of load round trips is the kernel's time.
// With more workgroups the 138 registers this takes cost more occupancy
// than the batching gains.
constexpr int kLogitsBatchGroups = 256;
// Selection: candidates are handled in chunks of kSelChunk (one workgroup
// each); the key histogram has kSelBins bins (bits 30..19 of the score key),
// the second level inside the pivot bin kSelBins2 (bits 18..8).
constexpr int kSelChunk = 1024;
constexpr int kSelBinBits = 12;
constexpr int kSelBins = 1 << kSelBinBits;
constexpr int kSelShift1 = 31 - kSelBinBits;  // first-level digit: key bits 30 .. kSelShift1
constexpr int kSelBins2 = 2048;
// The first-level histogram is kept in kHistCopies copies (reduction
// workgroup i adds into copy i mod kHistCopies), so that each hot bin takes a
// quarter of the atomics; the refine stage sums the copies.  At 1M the
// selection took 70.3 us with 4 copies against 71.8 with 1 and 72.0 with 8.
constexpr int kHistCopies = 4;
constexpr int kSelHistWords = kHistCopies * kSelBins + kSelBins2 + 1;  // per selection row, with the pivot-bin count
constexpr int kTopkMaxCand = 1 << 20;  // candidates per selection row (1,024 chunks)

struct SelectPlan {
    int n_layers, n_q, n_q_heads, n_kv_heads, head_dim, group, rows_per_head;
    int n_blocks, n_sink, n_recent, n_cand, k_eff, n_view, n_sel, mode;
    int n_rows;   // n_layers * n_q * n_q_heads
    int tile_lo;     // first index tile holding a candidate
    int n_tiles;     // index tiles holding candidates
    int tiles_per_part;  // index tiles per logit workgroup (0: the persistent 16-row kernel)
    int n_parts;     // logit workgroups along the candidates = partial stats per row
    int n_rsplit;    // row partitions of the block-relevance sum (1: one pass)
    int fused_stats; // 1: the reduction merges the row stats itself (no stats launch)
    int batch_loads; // 1: the vector logits kernel issues all of a tile's loads first
    int cand_stride; // row stride of logits and score rows (n_cand rounded up to 64)
    int n_chunks;    // ceil(n_cand / kSelChunk)
    // byte offsets into the workspace
    size_t off_logits;  // float  [n_rows][cand_stride]
    size_t off_tmax;    // float  [n_rows][n_parts]
    size_t off_tsum;    // double [n_rows][n_parts]
    size_t off_rmax;    // float  [n_rows]
    size_t off_rinvz;   // double [n_rows]
    size_t off_r32;     // float  [n_sel][cand_stride]
    size_t off_rpart;   // double [n_rsplit][n_sel][cand_stride] partial relevance (n_rsplit > 1)
    // uint32 [kHistCopies][n_sel][kSelBins] key histogram, [n_sel][kSelBins2]
    // pivot-bin histogram, [n_sel] pivot-bin key count (all zeroed by the score stats)
    size_t off_hist;
    size_t off_ctrl;    // uint32 [n_sel][8]            pivot bin, rank inside it
    size_t off_above;   // uint32 [n_sel][n_chunks]     keys above the pivot bin per chunk
    size_t off_seg;     // uint2  [n_sel][n_chunks * kSelChunk] pivot-bin (key, candidate), unordered
    size_t total;
};

inline void plan_select_layout(SelectPlan &p) {
    p.n_rows = p.n_layers * p.n_q * p.n_q_heads;
    p.tile_lo = p.n_sink / kIndexTile;
    p.n_tiles = (int)index_tiles(p.n_blocks - p.n_recent) - p.tile_lo;
    if (p.rows_per_head > 16) {
        p.tiles_per_part = 1;
        p.n_parts = p.n_tiles;
    } else if (p.rows_per_head > kScoreVectorRows) {  // persistent waves: n_parts = 4 x workgroups
        const int heads = p.n_layers * p.n_kv_heads;
        int wg = (kMfma16Waves / 4 + heads - 1) / heads;
        if (wg > p.n_tiles) wg = p.n_tiles;  // at least one 16-block group per wave
        p.tiles_per_part = 0;
        p.n_parts = 4 * (wg > 0 ? wg : 1);
    } else {
        p.tiles_per_part = kScoreTilesPerGroup;
        p.n_parts = (p.n_tiles + p.tiles_per_part - 1) / p.tiles_per_part;
    }
    {
        const int nr = p.mode == 0 ? p.n_rows : p.n_q * p.group;  // logit rows behind one relevance value
        int parts = nr / kReduceRowsPerPart;
        p.n_rsplit = parts < 2 ? 1 : (parts > kReduceMaxParts ? kReduceMaxParts : parts);
        const bool vec = p.rows_per_head <= kScoreVectorRows;
        p.fused_stats = vec && p.n_rsplit == 1 && nr <= kFusedStatsRows && p.n_parts <= kFusedStatsParts &&
                        (long long)nr * p.n_parts <= kFusedStatsPairs;
        p.batch_loads = vec && (long long)p.n_parts * p.n_kv_heads * p.n_layers <= kLogitsBatchGroups;
    }
    p.cand_stride = (p.n_cand + 63) / 64 * 64;
    p.n_chunks = (p.n_cand + kSelChunk - 1) / kSelChunk;
    size_t o = 0;
    p.off_logits = o; o = align_up(o + sizeof(float) * (size_t)p.n_rows * p.cand_stride);
    p.off_tmax = o;   o = align_up(o + sizeof(float) * (size_t)p.n_rows * p.n_parts);
    p.off_tsum = o;   o = align_up(o + sizeof(double) * (size_t)p.n_rows * p.n_parts);
    p.off_rmax = o;   o = align_up(o + sizeof(float) * (size_t)p.n_rows);
    p.off_rinvz = o;  o = align_up(o + sizeof(double) * (size_t)p.n_rows);
    p.off_r32 = o;    o = align_up(o + sizeof(float) * (size_t)p.n_sel * p.cand_stride);
    p.off_rpart = o;  o = align_up(o + (p.n_rsplit > 1 ? sizeof(double) * (size_t)p.n_rsplit * p.n_sel * p.cand_stride : 0));
    p.off_hist = o;   o = align_up(o + sizeof(uint32_t) * (size_t)p.n_sel * kSelHistWords);
    p.off_ctrl = o;   o = align_up(o + sizeof(uint32_t) * (size_t)p.n_sel * 8);
    p.off_above = o;  o = align_up(o + sizeof(uint32_t) * (size_t)p.n_sel * p.n_chunks);
    p.off_seg = o;    o = align_up(o + 8 * (size_t)p.n_sel * p.n_chunks * kSelChunk);
    p.total = o;
}

// ---- attention ---------------------------------------------------------
constexpr int kAttnTargetGroups = 256;   // workgroups the split-K launch aims for: one per compute unit
constexpr int kAttnMinPages = 4;         // pages per split, lower bound
constexpr int kAttnMaxPages = 512;       // pages per split, upper bound
constexpr int kAttnMaxSplits = 16384;    // split weights the merge keeps in LDS
constexpr int kPartStride = 4;           // floats after the D outputs of a partial row: m, l, pad

struct AttnPlan {
    int n_kv_heads, n_q_heads, group, n_q, rows_per_head, head_dim, block_tokens, kv_dtype;
    float k_scale, v_scale;  // FP8 pool scales (1 for the other types)
    int n_sel, n_view, last_page_tokens;
    int pages_per_split, n_splits;
    size_t off_part;  // float [Hkv][n_splits][rows_per_head][head_dim + kPartStride]
    size_t total;
};

inline void plan_attn_layout(AttnPlan &p) {
    // one workgroup per compute unit for decode (4 to 47 rows per KV head):
    // with two per unit the second one dispatched to each unit falls behind
    // the first and finishes alone, and the gather of random pages runs
    // slower with both resident (measured at 1M: 169.4 against 172.5 us per
    // call).  The many-row kernel keeps two per unit.
    const long long target = p.rows_per_head >= 48 ? 2 * kAttnTargetGroups : kAttnTargetGroups;
    long long want = ((long long)p.n_view * p.n_kv_heads + target - 1) / target;
    int pps = (int)(want < kAttnMinPages ? kAttnMinPages : (want > kAttnMaxPages ? kAttnMaxPages : want));
    p.pages_per_split = pps;
    p.n_splits = (p.n_view + pps - 1) / pps;
    p.off_part = 0;
    p.total = align_up(sizeof(float) * (size_t)p.n_kv_heads * p.n_splits * p.rows_per_head *
                       (p.head_dim + kPartStride));
}

// ---- RoPE (rotate-half form) ---------------------------------------------
// Frequencies f_j = base^(-2j/d), j < d/2, computed on the host with the same
// expression as the definition and passed to the kernels by value.
struct RopeFreqs {
    double f[64];
};
inline void rope_freqs(double base, int head_dim, RopeFreqs &fr) {
    for (int j = 0; j < 64; ++j) fr.f[j] = j < head_dim / 2 ? pow(base, -2.0 * (double)j / (double)head_dim) : 0.0;
}

// ---- working-set update (Eq. 11, Eq. 12) ---------------------------------
constexpr int kWsHeaderWords = 8;   // [0] previous step (-1: none), [1] |W| then, [2] clock hand
constexpr int kWsMaxPages = 1 << 22;

struct WorkingSetState {  // caller-owned device arrays (see kvmem_working_set in kvmem.h)
    int32_t n_blocks, n_pages;
    int32_t *block_page, *block_last_step, *page_block;
    int64_t *page_pos;
    int32_t *page_deltas, *header;
};

struct WsScratch {  // per-update scratch carved from the caller's workspace
    int32_t *kept;       // [P] page holds a selected block
    int32_t *kind;       // [n_view] unchanged / delta / rebuild / load / invalid
    int32_t *retained;   // [n_view] selected at the previous recall too
    int32_t *rank;       // [n_view] rank inside its kind
    int32_t *taken;      // [n_view] pages for the loads, in order
    int32_t *build_src, *build_dst, *delta_page;  // [n_view] lists
    int32_t *lists;      // [16] build length, delta length, loads in the build list
    int64_t *build_pos, *delta_shift;            // [n_view]
};

inline size_t ws_scratch_bytes(int n_view, int n_pages, WsScratch *w = nullptr, char *base = nullptr) {
    size_t o = 0;
    auto take = [&](size_t bytes) { const size_t at = o; o = align_up(o + bytes); return base + at; };
    int32_t *kept = (int32_t *)take(4 * (size_t)n_pages);
    int32_t *kind = (int32_t *)take(4 * (size_t)n_view);
    int32_t *retained = (int32_t *)take(4 * (size_t)n_view);
    int32_t *rank = (int32_t *)take(4 * (size_t)n_view);
    int32_t *taken = (int32_t *)take(4 * (size_t)n_view);
    int32_t *build_src = (int32_t *)take(4 * (size_t)n_view);
    int32_t *build_dst = (int32_t *)take(4 * (size_t)n_view);
    int32_t *delta_page = (int32_t *)take(4 * (size_t)n_view);
    int32_t *lists = (int32_t *)take(4 * 16);
    int64_t *build_pos = (int64_t *)take(8 * (size_t)n_view);
    int64_t *delta_shift = (int64_t *)take(8 * (size_t)n_view);
    if (w) *w = WsScratch{kept, kind, retained, rank, taken, build_src, build_dst, delta_page, lists, build_pos,
                          delta_shift};
    return o;
}

// ---- launchers (return the launch status) -------------------------------
// kv_dtype: 0 fp32, 1 bf16 bits, 2 FP8 E4M3 codes (scaled by k_scale, v_scale).
// materialize / rope_delta: with n_dev set, the first *n_dev of the n list
// entries are processed (the count is known on the device only).
// block_pos / fr are used only when rope is set: the keys carry RoPE at
// positions block_pos[b] + t (block_pos NULL: b * block_tokens + t).
hipError_t launch_build_index(int kv_dtype, int head_dim, int n_kv_heads, int block_tokens,
                              float k_scale, const void *k_pool, int64_t n_pages, const int32_t *block_to_page,
                              int32_t first_block, int32_t n_blocks, float *index,
                              hipStream_t stream, bool rope = false, const int64_t *block_pos = nullptr,
                              const RopeFreqs *fr = nullptr);

hipError_t launch_materialize(int kv_dtype, int head_dim, int n_kv_heads, int block_tokens,
                              const RopeFreqs &fr, const void *raw_k, const void *v_src,
                              int64_t n_src_pages, const int32_t *src_pages, const int64_t *positions,
                              const int32_t *dst_pages, int32_t n, void *k_dst, void *v_dst,
                              int64_t n_dst_pages, hipStream_t stream, const int32_t *n_dev = nullptr);

hipError_t launch_rope_delta(int kv_dtype, int head_dim, int n_kv_heads, int block_tokens, const RopeFreqs &fr,
                             void *k_pool, int64_t n_pages, const int32_t *pages, const int64_t *delta,
                             int32_t n, hipStream_t stream, const int32_t *n_dev = nullptr);

hipError_t launch_ws_reset(const WorkingSetState &s, hipStream_t stream);

hipError_t launch_ws_update(const WorkingSetState &s, const WsScratch &w, int kv_dtype, int head_dim, int n_kv_heads,
                            int block_tokens, const RopeFreqs &fr, int step, const int32_t *view, int n_view,
                            int64_t first_pos, int max_deltas, const int32_t *block_to_page, const void *raw_k,
                            const void *v_src, int64_t n_src_pages, void *k_exec, void *v_exec,
                            int32_t *exec_pages, int32_t *counts, hipStream_t stream);

hipError_t launch_topk(const SelectPlan &p, const int32_t *block_to_page, int32_t *view_blocks,
                       int32_t *view_pages, char *workspace, hipStream_t stream);

hipError_t launch_select(const SelectPlan &p, const float *q, const float *index, float scale,
                         const int32_t *block_to_page, int32_t *view_blocks, int32_t *view_pages,
                         float *scores, char *workspace, hipStream_t stream);

hipError_t launch_sparse_attn(const AttnPlan &p, const float *q, const void *k_pool,
                              const void *v_pool, int64_t n_pages, const int32_t *view_pages,
                              float scale, float *out, float *lse, char *workspace,
                              hipStream_t stream);

}  // namespace kvmem
