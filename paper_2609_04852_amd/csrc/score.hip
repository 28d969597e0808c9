// Query-conditioned block scoring (Eq. 10).
//
//   score_logits  streams the candidate tiles of the Mean-K index once.  The
//                 tiled layout puts 64 consecutive blocks of one KV head and one
//                 4-float slice of d in 1 KB, so a wave gives one block to each
//                 lane, reads with fully coalesced 16-byte loads, and every lane
//                 finishes its own dot products with the head's G * n_q query
//                 rows -- no cross-lane sums.  Logits go to the workspace, and
//                 every workgroup also leaves a (max, sum of exp) pair per query
//                 row for its four tiles.
//   score_stats   merges the tile pairs of one query row into the row's global
//                 softmax normalizer (max, 1/Z), so the tiled result equals the
//                 softmax over the full candidate set (Sec. 5.2 notes the same
//                 property for host-staged tiles).
//   score_reduce  turns logits into probabilities and combines them per block:
//                 the mean over layers and heads summed over query tokens
//                 (Eq. 10), or the per-(layer, KV head) maximum, and builds the
//                 score-key histogram the selection stages start from.
#include <math.h>

#include "kvmem_device.h"
#include "kvmem_internal.h"

namespace kvmem {
namespace {

constexpr int kScoreThreads = 256;

// One wave per (index tile of 64 blocks, KV head): lane i owns block
// 64*tile + i and accumulates its full dot products with the RH query rows of
// the head.  For every 4-float slice of the head dimension the wave reads 1 KB
// of contiguous index; the query values are the same for the whole wave.
template <int D, int RH, bool BATCH>
__global__ __launch_bounds__(kScoreThreads) void score_logits_kernel(
    const float *__restrict__ q, const float *__restrict__ index, int n_blocks, int n_kv_heads,
    int n_q_heads, int group, int n_q, int n_sink, int n_cand, int64_t cand_stride, int tile_lo,
    int n_tiles, int n_parts, float scale, float *__restrict__ logits, float *__restrict__ tmax,
    double *__restrict__ tsum, uint32_t *__restrict__ hist, int hist_words) {
    constexpr int NW = kScoreThreads / kWave;
    // with the row stats merged in the reduction, the histograms it fills are cleared here
    if (hist_words > 0) {
        const int wg = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
        const int n_wg = gridDim.x * gridDim.y * gridDim.z;
        for (int i = wg * kScoreThreads + threadIdx.x; i < hist_words; i += n_wg * kScoreThreads) hist[i] = 0u;
    }
    __shared__ float sm_m[NW][RH];
    __shared__ double sm_s[NW][RH];
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int g = blockIdx.y, l = blockIdx.z;
    const int tile = tile_lo + blockIdx.x * NW + wave;
    const int64_t b = (int64_t)tile * kIndexTile + lane;
    const int64_t c = b - n_sink;
    const bool valid = blockIdx.x * NW + wave < n_tiles && c >= 0 && c < n_cand;

    int64_t qrow[RH];
#pragma unroll
    for (int r = 0; r < RH; ++r)
        qrow[r] = ((int64_t)l * n_q + r / group) * n_q_heads + g * group + r % group;

    float acc[RH];
#pragma unroll
    for (int r = 0; r < RH; ++r) acc[r] = 0.f;
    if (blockIdx.x * NW + wave < n_tiles) {
        const int64_t tiles_per_layer = index_tiles(n_blocks);
        const float *src = index + (((int64_t)l * tiles_per_layer + tile) * n_kv_heads + g) *
                                       (int64_t)(D / 4) * (kIndexTile * 4) + lane * 4;
        if constexpr (BATCH) {  // every load of the tile in flight at once
            float4 xs[D / 4];
#pragma unroll
            for (int j4 = 0; j4 < D / 4; ++j4) xs[j4] = *reinterpret_cast<const float4 *>(src + j4 * (kIndexTile * 4));
            __builtin_amdgcn_sched_barrier(0);  // the scheduler keeps every load above the products
#pragma unroll
            for (int j4 = 0; j4 < D / 4; ++j4) {
                const float4 x = xs[j4];
#pragma unroll
                for (int r = 0; r < RH; ++r) {
                    const float4 qv = *reinterpret_cast<const float4 *>(q + qrow[r] * D + j4 * 4);
                    acc[r] += qv.x * x.x + qv.y * x.y + qv.z * x.z + qv.w * x.w;
                }
            }
        } else {
#pragma unroll
            for (int j4 = 0; j4 < D / 4; ++j4) {  // unrolled: the compiler keeps several loads in flight
                const float4 x = *reinterpret_cast<const float4 *>(src + j4 * (kIndexTile * 4));
#pragma unroll
                for (int r = 0; r < RH; ++r) {
                    const float4 qv = *reinterpret_cast<const float4 *>(q + qrow[r] * D + j4 * 4);
                    acc[r] += qv.x * x.x + qv.y * x.y + qv.z * x.z + qv.w * x.w;
                }
            }
        }
    }
    // logits of this tile (rows contiguous over candidates), and per-wave stats
#pragma unroll
    for (int r = 0; r < RH; ++r) {
        const float s = acc[r] * scale;
        if (valid) logits[qrow[r] * cand_stride + c] = s;
        float mx = wave_max(valid ? s : -INFINITY);
        double e = (valid && mx != -INFINITY) ? (double)expf(s - mx) : 0.0;
        e = wave_sum_d(e);
        if (lane == 0) {
            sm_m[wave][r] = mx;
            sm_s[wave][r] = e;
        }
    }
    __syncthreads();
    if ((int)threadIdx.x < RH) {
        const int r = threadIdx.x;
        float mx = sm_m[0][r];
#pragma unroll
        for (int w = 1; w < NW; ++w) mx = fmaxf(mx, sm_m[w][r]);
        double sum = 0.0;
#pragma unroll
        for (int w = 0; w < NW; ++w)
            if (sm_m[w][r] != -INFINITY) sum += sm_s[w][r] * exp((double)sm_m[w][r] - (double)mx);
        tmax[qrow[r] * n_parts + blockIdx.x] = mx;
        tsum[qrow[r] * n_parts + blockIdx.x] = sum;
    }
}

// 9 to 16 query rows per KV head (GQA heads x query tokens; a tile of 16 rows
// whose rows past the head's count are zero queries): the dot products run
// on the fp64 matrix cores (v_mfma_f64_16x16x4f64).  The fp32 inputs widen
// exactly, their products are exact in fp64 and the sums barely round, so the
// logit is the fp32 rounding of the exact dot product (the vector kernel's
// fp32 accumulation, and the fp32 matrix cores even more, lose a few ulps at
// the logit magnitudes of clustered keys, which the selection's 1e-5 band
// cannot afford).  For one 16-block group of a tile, S^T = index Q^T: lane l
// loads, for each 16-dim slice c, the 4 dims 16c + 4kg .. of block l%16 (kg =
// l/16) as one float4 from the tiled index and feeds them to 4 MFMAs whose
// contraction slot kg stands for those dims; Q^T is the matching B operand,
// kept in registers.  Lane l receives the logits of row l%16 for blocks kg,
// kg+4, kg+8, kg+12 of the group.
// The waves are persistent and pipelined: wave w of workgroup j takes the
// head's groups 4j + w, 4j + w + n_parts, ... and loads the next group while
// the current group's 32 MFMAs run, so the index stream and the matrix cores
// overlap.  Each wave keeps an online (max, sum of exp) per row over its
// groups -- the sum rescaled in fp64 when the maximum grows -- and leaves one
// partial per row: n_parts = workgroups x 4 partials per row.
typedef double f64x4_t __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(kScoreThreads) void score_logits_mfma16_kernel(
    const float *__restrict__ q, const float *__restrict__ index, int n_blocks, int n_kv_heads,
    int n_q_heads, int group, int n_q, int n_sink, int n_cand, int64_t cand_stride, int tile_lo,
    int n_tiles, int n_parts, float scale, float *__restrict__ logits, float *__restrict__ tmax,
    double *__restrict__ tsum) {
    constexpr int NW = kScoreThreads / kWave, NC = D / 16;
    static_assert(NW * 16 == kIndexTile, "four 16-block groups per tile");
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int r16 = lane % 16, kg = lane / 16;
    const int g = blockIdx.y, l = blockIdx.z;
    // the head's rows (9 to 16): lanes of rows past them hold zero queries
    // (a copy of the last row's address, never written)
    const int rows = group * n_q;
    const bool row_ok = r16 < rows;
    const int rr = row_ok ? r16 : rows - 1;
    const int64_t qrow = ((int64_t)l * n_q + rr / group) * n_q_heads + g * group + rr % group;
    const int64_t tiles_per_layer = index_tiles(n_blocks);
    const int part = blockIdx.x * NW + wave;  // this wave's partial; n_parts waves per (layer, head)
    const int n_groups = n_tiles * NW;

    auto load = [&](int gi, float4 (&x)[NC]) {
        const int tile = tile_lo + gi / NW, gb = gi % NW;
        const float *src = index + (((int64_t)l * tiles_per_layer + tile) * n_kv_heads + g) *
                                       (int64_t)(D / 4) * (kIndexTile * 4) + (16 * gb + r16) * 4;
#pragma unroll
        for (int c = 0; c < NC; ++c) x[c] = *reinterpret_cast<const float4 *>(src + (4 * c + kg) * (kIndexTile * 4));
    };
    float4 xa[NC], xb[NC];
    int gi = part;
    // every load is issued unconditionally at a clamped (in-bounds) group:
    // behind a branch the compiler must wait at the join for every load,
    // including the prefetch just issued
    const int g_last = n_groups - 1;
    load(min(gi, g_last), xa);
    // B operand: q[row r16][16c + 4kg + e] (the scale is applied to the sum)
    float qv[NC][4];
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const float4 v = *reinterpret_cast<const float4 *>(q + qrow * D + 16 * c + 4 * kg);
        qv[c][0] = row_ok ? v.x : 0.f; qv[c][1] = row_ok ? v.y : 0.f;
        qv[c][2] = row_ok ? v.z : 0.f; qv[c][3] = row_ok ? v.w : 0.f;
    }
    float mrun = -INFINITY;  // row r16 (the same in its 4 kg lanes)
    double srun = 0.0;
    auto compute = [&](int gj, const float4 (&x)[NC]) {
        // two accumulator chains, so that a wave's products do not each wait
        // for the one before (20.7 against 21.0 us per MTP layer; four: 20.8)
        f64x4_t st = f64x4_t{0.0, 0.0, 0.0, 0.0}, st1 = f64x4_t{0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const float xv[4] = {x[c].x, x[c].y, x[c].z, x[c].w};
#pragma unroll
            for (int e = 0; e < 4; e += 2) {
                st = __builtin_amdgcn_mfma_f64_16x16x4f64((double)xv[e], (double)qv[c][e], st, 0, 0, 0);
                st1 = __builtin_amdgcn_mfma_f64_16x16x4f64((double)xv[e + 1], (double)qv[c][e + 1], st1, 0, 0, 0);
            }
        }
        st += st1;
        // logits of blocks kg + 4i of the group, and the online row stats
        const int64_t c0 = (int64_t)(tile_lo + gj / NW) * kIndexTile + 16 * (gj % NW) + kg - n_sink;
        float s[4];
        bool ok[4];
        float gm = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            s[i] = (float)(st[i] * (double)scale);
            const int64_t c = c0 + 4 * i;
            ok[i] = c >= 0 && c < n_cand;
            if (ok[i] && row_ok) logits[qrow * cand_stride + c] = s[i];
            gm = fmaxf(gm, ok[i] ? s[i] : -INFINITY);
        }
        gm = fmaxf(gm, shfl_xor_f(gm, 16));
        gm = fmaxf(gm, shfl_xor_f(gm, 32));
        if (gm > mrun) {
            srun = mrun == -INFINITY ? 0.0 : srun * exp((double)mrun - (double)gm);
            mrun = gm;
        }
        double e = 0.0;
        if (mrun != -INFINITY) {
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (ok[i]) e += (double)expf(s[i] - mrun);
        }
        e += __shfl_xor(e, 16, kWave);
        e += __shfl_xor(e, 32, kWave);
        srun += e;
    };
    // two register buffers: the next group's loads are in flight during the
    // current group's products
    while (gi < n_groups) {
        const int g1 = gi + n_parts;
        load(min(g1, g_last), xb);
        compute(gi, xa);
        if (g1 >= n_groups) break;
        const int g2 = g1 + n_parts;
        load(min(g2, g_last), xa);
        compute(g1, xb);
        gi = g2;
    }
    if (kg == 0 && row_ok) {
        tmax[qrow * n_parts + part] = mrun;
        tsum[qrow * n_parts + part] = srun;
    }
}

// More than 16 query rows per KV head (a recall point: the prefill's query
// tokens x the group's heads; a ragged last 16-row chunk repeats its last row,
// whose copies are never written).  The scoring is then a dense contraction,
// S = Q index^T, run on the fp64 matrix cores for the same reason as above.
// One workgroup per (index tile, KV head, layer): the tile's 64 x D floats are
// staged in LDS once and serve every row of that (layer, KV head); each wave
// takes 16-row chunks in turn.  Per chunk and 16-dim slice c, lane l (r16 =
// l % 16, kg = l / 16) holds the 4 dims 16c + 4kg .. of query row r16 (A
// operand) and of block 16gb + r16 (B operand, gb = 0..3); contraction slot kg
// stands for those dims on both sides.  Lane l receives the logits of rows
// kg + 4i of the chunk for block 16gb + r16, so every row's 64 logits sit in
// the 16 lanes of one kg group, which also reduce its (max, sum of exp).
template <int D>
__global__ __launch_bounds__(kScoreThreads) void score_logits_rows_kernel(
    const float *__restrict__ q, const float *__restrict__ index, int n_blocks, int n_kv_heads,
    int n_q_heads, int group, int n_q, int n_sink, int n_cand, int64_t cand_stride, int tile_lo,
    int n_parts, float scale, float *__restrict__ logits, float *__restrict__ tmax,
    double *__restrict__ tsum) {
    constexpr int NW = kScoreThreads / kWave, NC = D / 16;
    __shared__ float4 sm_idx[D / 4][kIndexTile];  // the tile in its stored layout: [j4][block]
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int r16 = lane % 16, kg = lane / 16;
    const int g = blockIdx.y, l = blockIdx.z;
    const int tile = tile_lo + blockIdx.x;
    {
        const int64_t tiles_per_layer = index_tiles(n_blocks);
        const float4 *src = reinterpret_cast<const float4 *>(
            index + (((int64_t)l * tiles_per_layer + tile) * n_kv_heads + g) * (int64_t)(D / 4) * (kIndexTile * 4));
        for (int i = threadIdx.x; i < (D / 4) * kIndexTile; i += kScoreThreads)
            sm_idx[i / kIndexTile][i % kIndexTile] = src[i];
    }
    __syncthreads();
    const int64_t b0 = (int64_t)tile * kIndexTile - n_sink;  // candidate of the tile's first block
    // candidates of this lane's 4 blocks (16gb + r16) that are in C
    bool cok[4];
#pragma unroll
    for (int gb = 0; gb < 4; ++gb) cok[gb] = b0 + 16 * gb + r16 >= 0 && b0 + 16 * gb + r16 < n_cand;
    const int rows = n_q * group;
    for (int chunk = wave; chunk < (rows + 15) / 16; chunk += NW) {
        // A operand: query row chunk*16 + r16 of (layer l, KV head g); in a
        // ragged last chunk the rows past the head's count repeat the last
        // row and their results are never written
        const int r = min(chunk * 16 + r16, rows - 1);
        const int64_t qrow = ((int64_t)l * n_q + r / group) * n_q_heads + g * group + r % group;
        f64x4_t st[4];
#pragma unroll
        for (int gb = 0; gb < 4; ++gb) st[gb] = f64x4_t{0.0, 0.0, 0.0, 0.0};
        float4 qa[NC];  // the chunk's query slices, all in flight before the products start
#pragma unroll
        for (int c = 0; c < NC; ++c) qa[c] = *reinterpret_cast<const float4 *>(q + qrow * D + 16 * c + 4 * kg);
        float4 bn[4];
#pragma unroll
        for (int gb = 0; gb < 4; ++gb) bn[gb] = sm_idx[kg][16 * gb + r16];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            float4 bv[4];
#pragma unroll
            for (int gb = 0; gb < 4; ++gb) bv[gb] = bn[gb];
            if (c + 1 < NC) {
#pragma unroll
                for (int gb = 0; gb < 4; ++gb) bn[gb] = sm_idx[4 * (c + 1) + kg][16 * gb + r16];
            }
            const float av[4] = {qa[c].x, qa[c].y, qa[c].z, qa[c].w};
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int gb = 0; gb < 4; ++gb) {
                    const float be = e == 0 ? bv[gb].x : e == 1 ? bv[gb].y : e == 2 ? bv[gb].z : bv[gb].w;
                    st[gb] = __builtin_amdgcn_mfma_f64_16x16x4f64((double)av[e], (double)be, st[gb], 0, 0, 0);
                }
            __builtin_amdgcn_sched_barrier(0);  // next slice's LDS reads overlap these products, no further
        }
        // lane: rows kg + 4i of the chunk, blocks 16gb + r16
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int rr0 = chunk * 16 + kg + 4 * i;
            const bool rok = rr0 < rows;  // the same in the 16 lanes that share this row
            const int rr = rok ? rr0 : rows - 1;
            const int64_t row = ((int64_t)l * n_q + rr / group) * n_q_heads + g * group + rr % group;
            float sv[4];
            float mx = -INFINITY;
#pragma unroll
            for (int gb = 0; gb < 4; ++gb) {
                sv[gb] = (float)(st[gb][i] * (double)scale);
                if (cok[gb]) {
                    if (rok) logits[row * cand_stride + b0 + 16 * gb + r16] = sv[gb];
                    mx = fmaxf(mx, sv[gb]);
                }
            }
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) mx = fmaxf(mx, shfl_xor_f(mx, o));
            double e = 0.0;
            if (mx != -INFINITY) {
#pragma unroll
                for (int gb = 0; gb < 4; ++gb)
                    if (cok[gb]) e += (double)expf(sv[gb] - mx);
            }
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) e += __shfl_xor(e, o, kWave);
            if (r16 == 0 && rok) {
                tmax[row * n_parts + blockIdx.x] = mx;
                tsum[row * n_parts + blockIdx.x] = e;
            }
        }
    }
}

__global__ __launch_bounds__(kScoreThreads) void score_stats_kernel(const float *__restrict__ tmax,
                                                                    const double *__restrict__ tsum,
                                                                    int n_parts, float *__restrict__ rmax,
                                                                    double *__restrict__ rinvz,
                                                                    uint32_t *__restrict__ hist,
                                                                    int hist_words) {
    // the selection histograms are filled by the next kernels; clear them here
    for (int i = blockIdx.x * kScoreThreads + threadIdx.x; i < hist_words; i += gridDim.x * kScoreThreads)
        hist[i] = 0u;
    __shared__ float sm_f[kScoreThreads / kWave];
    __shared__ double sm_d[kScoreThreads / kWave];
    const int row = blockIdx.x;
    const float *tm = tmax + (int64_t)row * n_parts;
    const double *ts = tsum + (int64_t)row * n_parts;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    float mx = -INFINITY;
    for (int i = threadIdx.x; i < n_parts; i += kScoreThreads) mx = fmaxf(mx, tm[i]);
    mx = wave_max(mx);
    if (lane == 0) sm_f[wave] = mx;
    __syncthreads();
    mx = sm_f[0];
    for (int w = 1; w < kScoreThreads / kWave; ++w) mx = fmaxf(mx, sm_f[w]);
    double z = 0.0;
    for (int i = threadIdx.x; i < n_parts; i += kScoreThreads)
        if (tm[i] != -INFINITY) z += ts[i] * exp((double)tm[i] - (double)mx);
    z = wave_sum_d(z);
    if (lane == 0) sm_d[wave] = z;
    __syncthreads();
    if (threadIdx.x == 0) {
        double tot = 0.0;
        for (int w = 0; w < kScoreThreads / kWave; ++w) tot += sm_d[w];
        rmax[row] = mx;
        rinvz[row] = 1.0 / tot;
    }
}

// Block relevance for one selection row and kReduceCols * 4 candidates:
// thread (slice rs, column col) sums every 4th contributing logit row for the
// 4 candidates of its column (float4 loads), the 4 slices are then combined in
// LDS in a fixed order:
//   mean-all:  R_b = (1/(L*Hq)) * sum over every (l, m, h) row of p  (Eq. 10)
//   group-max: R[l][g][b] = max over the (m, h in g) rows of layer l of p
// with p = exp(s - max_row) / Z_row summed in fp64.  R is rounded once to fp32.
// Each workgroup also histograms the selection key (bits(R) + 1) of its
// candidates by bits 30..19 in LDS and adds the non-empty bins to the row's
// global histogram, which the selection stages start from.
constexpr int kReduceCols = kScoreThreads / 4;  // float4 columns per workgroup
constexpr int kReduceCands = 4 * kReduceCols;

// With many logit rows behind each relevance value (a recall point), the sum
// (or max) over rows is split: workgroup (candidate chunk, selection row, part)
// covers rows [part * nr / n_part, (part + 1) * nr / n_part) exactly as
// score_reduce does all of them, and leaves its fp64 partial in rpart;
// score_reduce then combines the parts in order.
__global__ __launch_bounds__(kScoreThreads) void score_reduce_part_kernel(
    const float *__restrict__ logits, const float *__restrict__ rmax, const double *__restrict__ rinvz,
    int n_layers, int n_q, int n_q_heads, int n_kv_heads, int group, int n_cand, int64_t cand_stride, int mode,
    int n_sel, double *__restrict__ rpart) {
    __shared__ double sm_acc[4][kReduceCols][4];
    const int sel = blockIdx.y, part = blockIdx.z, n_part = gridDim.z;
    const int col = threadIdx.x % kReduceCols, rs = threadIdx.x / kReduceCols;
    const int c0 = blockIdx.x * kReduceCands + 4 * col;
    const int nr = mode == 0 ? n_layers * n_q * n_q_heads : n_q * group;
    const int i0 = (int)((int64_t)part * nr / n_part), i1 = (int)((int64_t)(part + 1) * nr / n_part);
    const int l = mode == 0 ? 0 : sel / n_kv_heads, g = mode == 0 ? 0 : sel % n_kv_heads;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    if (c0 < n_cand) {
#pragma unroll 8
        for (int i = i0 + rs; i < i1; i += 4) {
            const int64_t row = mode == 0 ? (int64_t)i
                                          : ((int64_t)l * n_q + i / group) * n_q_heads + g * group + i % group;
            const float4 x = *reinterpret_cast<const float4 *>(logits + row * cand_stride + c0);
            const float mx = rmax[row];
            const double iz = rinvz[row];
            const float xs[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const double pr = (double)expf(xs[e] - mx) * iz;
                if (mode == 0) acc[e] += pr;
                else acc[e] = pr > acc[e] ? pr : acc[e];
            }
        }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) sm_acc[rs][col][e] = acc[e];
    __syncthreads();
    if (rs == 0 && c0 < n_cand) {
        double out[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            double a = sm_acc[0][col][e];
#pragma unroll
            for (int k = 1; k < 4; ++k) {
                const double b = sm_acc[k][col][e];
                a = mode == 0 ? a + b : (b > a ? b : a);
            }
            out[e] = a;
        }
        double *dst = rpart + ((int64_t)part * n_sel + sel) * cand_stride + c0;
#pragma unroll
        for (int e = 0; e < 4; ++e) dst[e] = out[e];
    }
}

__global__ __launch_bounds__(kScoreThreads) void score_reduce_kernel(
    const float *__restrict__ logits, const float *__restrict__ rmax,
    const double *__restrict__ rinvz, int n_layers, int n_q, int n_q_heads, int n_kv_heads,
    int group, int n_blocks, int n_sink, int n_cand, int64_t cand_stride, int mode,
    float *__restrict__ r32, float *__restrict__ scores, uint32_t *__restrict__ hist,
    const double *__restrict__ rpart, int n_rsplit, const float *__restrict__ tmax,
    const double *__restrict__ tsum, int n_parts, int fused) {
    __shared__ uint32_t lh[kSelBins];
    __shared__ double sm_acc[4][kReduceCols][4];
    __shared__ float sm_rmax[kFusedStatsRows];
    __shared__ double sm_rinvz[kFusedStatsRows];
    const int sel = blockIdx.y;
    const int col = threadIdx.x % kReduceCols, rs = threadIdx.x / kReduceCols;
    for (int i = threadIdx.x; i < kSelBins; i += kScoreThreads) lh[i] = 0u;
    const int c0 = blockIdx.x * kReduceCands + 4 * col;
    // mean-all: every (l, m, h) row; group-max: the (m, h in g) rows of layer l
    const int nr = mode == 0 ? n_layers * n_q * n_q_heads : n_q * group;
    const int l = mode == 0 ? 0 : sel / n_kv_heads, g = mode == 0 ? 0 : sel % n_kv_heads;
    if (fused) {
        // the rows' max and 1 / Z from their per-tile pairs (the merge of
        // score_stats, in another order): one 16-lane DPP row per logit row,
        // rows grp + 16 j, every pair loaded at once (clamped, no branch)
        constexpr int NG = kScoreThreads / 16;
        constexpr int RPG = kFusedStatsRows / NG, PPL = kFusedStatsParts / 16;
        const int grp = threadIdx.x / 16, l16 = threadIdx.x % 16;
        float tmv[RPG][PPL];
        double tsv[RPG][PPL];
#pragma unroll
        for (int j = 0; j < RPG; ++j) {
            const int i = min(grp + NG * j, nr - 1);
            const int64_t row = mode == 0 ? (int64_t)i
                                          : ((int64_t)l * n_q + i / group) * n_q_heads + g * group + i % group;
#pragma unroll
            for (int u = 0; u < PPL; ++u) {
                const int k = min(l16 + 16 * u, n_parts - 1);
                tmv[j][u] = tmax[row * n_parts + k];
                tsv[j][u] = tsum[row * n_parts + k];
            }
        }
#pragma unroll
        for (int j = 0; j < RPG; ++j) {
            float mx = -INFINITY;
#pragma unroll
            for (int u = 0; u < PPL; ++u) mx = l16 + 16 * u < n_parts ? fmaxf(mx, tmv[j][u]) : mx;
            mx = row16_max(mx);
            double z = 0.0;
#pragma unroll
            for (int u = 0; u < PPL; ++u)
                if (l16 + 16 * u < n_parts && tmv[j][u] != -INFINITY)
                    z += tsv[j][u] * exp((double)tmv[j][u] - (double)mx);
            z = row16_sum_d(z);
            const int i = grp + NG * j;
            if (l16 == 0 && i < nr) {
                sm_rmax[i] = mx;
                sm_rinvz[i] = 1.0 / z;
            }
        }
        __syncthreads();
    }
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
    if (c0 < n_cand && rpart) {
        // the row partitions' partials, in order (slice 0 only)
        if (rs == 0) {
            for (int k = 0; k < n_rsplit; ++k) {
                const double *src = rpart + ((int64_t)k * gridDim.y + sel) * cand_stride + c0;
#pragma unroll
                for (int e = 0; e < 4; ++e) acc[e] = mode == 0 ? acc[e] + src[e] : (src[e] > acc[e] ? src[e] : acc[e]);
            }
        }
    } else if (c0 < n_cand) {
#pragma unroll 8
        for (int i = rs; i < nr; i += 4) {
            const int64_t row = mode == 0 ? (int64_t)i
                                          : ((int64_t)l * n_q + i / group) * n_q_heads + g * group + i % group;
            const float4 x = *reinterpret_cast<const float4 *>(logits + row * cand_stride + c0);
            const float mx = fused ? sm_rmax[i] : rmax[row];
            const double iz = fused ? sm_rinvz[i] : rinvz[row];
            const float xs[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const double pr = (double)expf(xs[e] - mx) * iz;
                if (mode == 0) acc[e] += pr;
                else acc[e] = pr > acc[e] ? pr : acc[e];
            }
        }
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) sm_acc[rs][col][e] = acc[e];
    __syncthreads();
    if (rs == 0 && c0 < n_cand) {
        float r[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            double a = sm_acc[0][col][e];
#pragma unroll
            for (int k = 1; k < 4; ++k) {
                const double b = sm_acc[k][col][e];
                a = mode == 0 ? a + b : (b > a ? b : a);
            }
            r[e] = mode == 0 ? (float)(a / (double)(n_layers * n_q_heads)) : (float)a;
        }
        float *dst = r32 + (int64_t)sel * cand_stride + c0;
        *reinterpret_cast<float4 *>(dst) = make_float4(r[0], r[1], r[2], r[3]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            if (c0 + e >= n_cand) continue;
            const uint32_t key = __float_as_uint(r[e]) + 1u;
            atomicAdd(&lh[(key >> kSelShift1) & (kSelBins - 1)], 1u);
            if (scores) scores[(int64_t)sel * n_blocks + n_sink + c0 + e] = r[e];
        }
    }
    if (scores && blockIdx.x == 0) {
        const int n_res = n_blocks - n_cand;  // sink blocks, then recent blocks
        for (int i = threadIdx.x; i < n_res; i += kScoreThreads) {
            const int b = i < n_sink ? i : n_sink + n_cand + (i - n_sink);
            scores[(int64_t)sel * n_blocks + b] = INFINITY;
        }
    }
    __syncthreads();
    uint32_t *gh = hist + ((int64_t)(blockIdx.x % kHistCopies) * gridDim.y + sel) * kSelBins;
    // the thread's bins read from LDS at once, then the non-empty ones added
    constexpr int PER = kSelBins / kScoreThreads;
    static_assert(PER * kScoreThreads == kSelBins, "bins split evenly");
    uint32_t cnt[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) cnt[u] = lh[threadIdx.x + kScoreThreads * u];
#pragma unroll
    for (int u = 0; u < PER; ++u)
        if (cnt[u]) atomicAdd(&gh[threadIdx.x + kScoreThreads * u], cnt[u]);
}

template <int D, int RH>
hipError_t launch_logits(const SelectPlan &p, const float *q, const float *index, float scale,
                         float *logits, float *tmax, double *tsum, uint32_t *hist, hipStream_t stream) {
    dim3 grid(p.n_parts, p.n_kv_heads, p.n_layers);
    const int hist_words = p.fused_stats ? p.n_sel * kSelHistWords : 0;
    if (p.batch_loads)
        hipLaunchKernelGGL((score_logits_kernel<D, RH, true>), grid, dim3(kScoreThreads), 0, stream, q, index,
                           p.n_blocks, p.n_kv_heads, p.n_q_heads, p.group, p.n_q, p.n_sink, p.n_cand,
                           (int64_t)p.cand_stride, p.tile_lo, p.n_tiles, p.n_parts, scale, logits, tmax,
                           tsum, hist, hist_words);
    else
        hipLaunchKernelGGL((score_logits_kernel<D, RH, false>), grid, dim3(kScoreThreads), 0, stream, q, index,
                           p.n_blocks, p.n_kv_heads, p.n_q_heads, p.group, p.n_q, p.n_sink, p.n_cand,
                           (int64_t)p.cand_stride, p.tile_lo, p.n_tiles, p.n_parts, scale, logits, tmax,
                           tsum, hist, hist_words);
    return hipGetLastError();
}

template <int D>
hipError_t launch_logits_d(const SelectPlan &p, const float *q, const float *index, float scale,
                           float *logits, float *tmax, double *tsum, uint32_t *hist, hipStream_t stream) {
    static_assert(kScoreVectorRows == 8, "vector kernels for 1 to 8 rows");
    switch (p.rows_per_head) {
        case 1: return launch_logits<D, 1>(p, q, index, scale, logits, tmax, tsum, hist, stream);
        case 2: return launch_logits<D, 2>(p, q, index, scale, logits, tmax, tsum, hist, stream);
        case 3: return launch_logits<D, 3>(p, q, index, scale, logits, tmax, tsum, hist, stream);
        case 4: return launch_logits<D, 4>(p, q, index, scale, logits, tmax, tsum, hist, stream);
        case 5: return launch_logits<D, 5>(p, q, index, scale, logits, tmax, tsum, hist, stream);
        case 6: return launch_logits<D, 6>(p, q, index, scale, logits, tmax, tsum, hist, stream);
        case 7: return launch_logits<D, 7>(p, q, index, scale, logits, tmax, tsum, hist, stream);
        case 8: return launch_logits<D, 8>(p, q, index, scale, logits, tmax, tsum, hist, stream);
        case 9: case 10: case 11: case 12: case 13: case 14: case 15: case 16: {
            dim3 grid(p.n_parts / 4, p.n_kv_heads, p.n_layers);
            hipLaunchKernelGGL((score_logits_mfma16_kernel<D>), grid, dim3(kScoreThreads), 0, stream, q, index,
                               p.n_blocks, p.n_kv_heads, p.n_q_heads, p.group, p.n_q, p.n_sink, p.n_cand,
                               (int64_t)p.cand_stride, p.tile_lo, p.n_tiles, p.n_parts, scale, logits, tmax,
                               tsum);
            return hipGetLastError();
        }
        default: {
            if (p.tiles_per_part != 1) return hipErrorInvalidValue;
            dim3 grid(p.n_tiles, p.n_kv_heads, p.n_layers);
            hipLaunchKernelGGL((score_logits_rows_kernel<D>), grid, dim3(kScoreThreads), 0, stream, q, index,
                               p.n_blocks, p.n_kv_heads, p.n_q_heads, p.group, p.n_q, p.n_sink, p.n_cand,
                               (int64_t)p.cand_stride, p.tile_lo, p.n_parts, scale, logits, tmax, tsum);
            return hipGetLastError();
        }
    }
}

}  // namespace

hipError_t launch_select(const SelectPlan &p, const float *q, const float *index, float scale,
                         const int32_t *block_to_page, int32_t *view_blocks, int32_t *view_pages,
                         float *scores, char *ws, hipStream_t stream) {
    float *logits = reinterpret_cast<float *>(ws + p.off_logits);
    float *tmax = reinterpret_cast<float *>(ws + p.off_tmax);
    double *tsum = reinterpret_cast<double *>(ws + p.off_tsum);
    float *rmax = reinterpret_cast<float *>(ws + p.off_rmax);
    double *rinvz = reinterpret_cast<double *>(ws + p.off_rinvz);
    float *r32 = reinterpret_cast<float *>(ws + p.off_r32);
    uint32_t *hist = reinterpret_cast<uint32_t *>(ws + p.off_hist);
    hipError_t e = hipSuccess;
    if (p.n_cand > 0) {  // with no candidate the view is sink + recent only
        e = p.head_dim == 128 ? launch_logits_d<128>(p, q, index, scale, logits, tmax, tsum, hist, stream)
                              : launch_logits_d<64>(p, q, index, scale, logits, tmax, tsum, hist, stream);
        if (e != hipSuccess) return e;
        if (!p.fused_stats) {
            hipLaunchKernelGGL(score_stats_kernel, dim3(p.n_rows), dim3(kScoreThreads), 0, stream, tmax, tsum,
                               p.n_parts, rmax, rinvz, hist, p.n_sel * kSelHistWords);
            if ((e = hipGetLastError()) != hipSuccess) return e;
        }
    }
    // at least one workgroup per row, which also marks the reserved blocks' scores
    const int n_red = (p.n_cand + kReduceCands - 1) / kReduceCands;
    double *rpart = nullptr;
    if (p.n_rsplit > 1 && p.n_cand > 0) {
        rpart = reinterpret_cast<double *>(ws + p.off_rpart);
        hipLaunchKernelGGL(score_reduce_part_kernel, dim3(n_red, p.n_sel, p.n_rsplit), dim3(kScoreThreads), 0,
                           stream, logits, rmax, rinvz, p.n_layers, p.n_q, p.n_q_heads, p.n_kv_heads, p.group,
                           p.n_cand, (int64_t)p.cand_stride, p.mode, p.n_sel, rpart);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(score_reduce_kernel, dim3(n_red > 0 ? n_red : 1, p.n_sel), dim3(kScoreThreads), 0, stream,
                       logits, rmax, rinvz, p.n_layers, p.n_q, p.n_q_heads, p.n_kv_heads, p.group,
                       p.n_blocks, p.n_sink, p.n_cand, (int64_t)p.cand_stride, p.mode, r32, scores, hist, rpart,
                       p.n_rsplit, tmax, tsum, p.n_parts, p.fused_stats && p.n_cand > 0);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_topk(p, block_to_page, view_blocks, view_pages, ws, stream);
}

}  // namespace kvmem
