// Query-conditioned block scoring (Eq. 10).
//
//   score_logits  streams the candidate rows of the Mean-K index once.  A team
//                 of d/4 lanes owns one KV head; every lane holds 16 bytes of
//                 each index row and the matching slice of the group's query
//                 rows in registers.  NBK blocks are processed per step and the
//                 NBK * rows partial dot products are summed across the team
//                 with a transposing butterfly, so each lane ends with one
//                 finished logit.  Logits go to the workspace, and every
//                 workgroup also leaves a (max, sum of exp) pair per query row
//                 for its tile of blocks.
//   score_stats   merges the tile pairs of one query row into the row's global
//                 softmax normalizer (max, 1/Z), so the tiled result equals the
//                 softmax over the full candidate set (Sec. 5.2 notes the same
//                 property for host-staged tiles).
//   score_reduce  turns logits into probabilities and combines them per block:
//                 the mean over layers and heads summed over query tokens
//                 (Eq. 10), or the per-(layer, KV head) maximum.
#include <math.h>

#include "kvmem_device.h"
#include "kvmem_internal.h"

namespace kvmem {
namespace {

constexpr int kScoreThreads = 256;

template <int D, int RH>
struct ScoreShape {
    static constexpr int TEAM = D / 4;                       // lanes per index row
    static constexpr int TEAMS = kScoreThreads / TEAM;       // teams per workgroup
    static constexpr int NBK = (TEAM / RH) < 8 ? (TEAM / RH) : 8;  // blocks per step
    static constexpr int N = NBK * RH;                       // partial sums per lane per step
    static constexpr int SHIFT = __builtin_ctz(TEAM / N);    // lanes per finished value = 1<<SHIFT
};

template <int D, int RH>
__global__ __launch_bounds__(kScoreThreads) void score_logits_kernel(
    const float *__restrict__ q, const float *__restrict__ index, int n_blocks, int n_kv_heads,
    int n_q_heads, int group, int n_q, int n_sink, int n_cand, int tile, int n_tiles,
    int heads_per_wg, float scale, float *__restrict__ logits, float *__restrict__ tmax,
    double *__restrict__ tsum) {
    using S = ScoreShape<D, RH>;
    constexpr int TEAM = S::TEAM, TEAMS = S::TEAMS, NBK = S::NBK, N = S::N;
    __shared__ float sm_m[kScoreThreads];
    __shared__ double sm_s[kScoreThreads];

    const int team = threadIdx.x / TEAM, lt = threadIdx.x % TEAM;
    const int bls = TEAMS / heads_per_wg;  // teams sharing one head
    const int hw = team % heads_per_wg, bl = team / heads_per_wg;
    const int g = blockIdx.y * heads_per_wg + hw;
    const int l = blockIdx.z;
    const int c0 = blockIdx.x * tile;

    // this lane's slice of the group's query rows, r = m * G + hh
    float qr[RH][4];
#pragma unroll
    for (int r = 0; r < RH; ++r) {
        const int m = r / group, hh = r % group;
        const int64_t row = ((int64_t)l * n_q + m) * n_q_heads + g * group + hh;
        const float4 v = *reinterpret_cast<const float4 *>(q + row * D + lt * 4);
        qr[r][0] = v.x * scale; qr[r][1] = v.y * scale; qr[r][2] = v.z * scale; qr[r][3] = v.w * scale;
    }
    // after the team reduction this lane holds value v = row slot * NBK + block slot
    const int v = lt >> S::SHIFT;
    const bool writer = (lt & ((1 << S::SHIFT) - 1)) == 0;
    const int vr = v / NBK, vk = v % NBK;
    const int64_t my_row = ((int64_t)l * n_q + vr / group) * n_q_heads + g * group + vr % group;

    const float *ibase = index + (((int64_t)l * n_blocks + n_sink) * n_kv_heads + g) * D + lt * 4;
    const int64_t row_stride = (int64_t)n_kv_heads * D;
    float run_m = -INFINITY;
    double run_s = 0.0;
    const int steps = tile / (NBK * bls);
    for (int it = 0; it < steps; ++it) {
        const int cb = c0 + (it * bls + bl) * NBK;
        float kv[NBK][4];
#pragma unroll
        for (int k = 0; k < NBK; ++k) {
            const int c = cb + k;
            if (c < n_cand) {
                const float4 x = *reinterpret_cast<const float4 *>(ibase + (int64_t)c * row_stride);
                kv[k][0] = x.x; kv[k][1] = x.y; kv[k][2] = x.z; kv[k][3] = x.w;
            } else {
                kv[k][0] = kv[k][1] = kv[k][2] = kv[k][3] = 0.f;
            }
        }
        float part[N];
#pragma unroll
        for (int r = 0; r < RH; ++r)
#pragma unroll
            for (int k = 0; k < NBK; ++k)
                part[r * NBK + k] = qr[r][0] * kv[k][0] + qr[r][1] * kv[k][1] +
                                    qr[r][2] * kv[k][2] + qr[r][3] * kv[k][3];
        const float s = team_transpose_reduce<N, TEAM>(part, lt);
        const int c = cb + vk;
        if (c < n_cand) {
            if (writer) logits[my_row * n_cand + c] = s;
            // running (max, sum exp) with one exponential per value
            const float dlt = s - run_m;
            const double e = (double)expf(-fabsf(dlt));
            if (dlt > 0.f) {
                run_s = run_s * e + 1.0;
                run_m = s;
            } else {
                run_s += e;
            }
        }
    }
    sm_m[threadIdx.x] = writer ? run_m : -INFINITY;
    sm_s[threadIdx.x] = writer ? run_s : 0.0;
    __syncthreads();
    // merge the lanes and teams that hold the same (head, row slot)
    if ((int)threadIdx.x < heads_per_wg * RH) {
        const int h2 = threadIdx.x / RH, r = threadIdx.x % RH;
        float mx = -INFINITY;
        for (int b2 = 0; b2 < bls; ++b2)
            for (int k = 0; k < NBK; ++k) {
                const int idx = (b2 * heads_per_wg + h2) * TEAM + ((r * NBK + k) << S::SHIFT);
                mx = fmaxf(mx, sm_m[idx]);
            }
        double sum = 0.0;
        for (int b2 = 0; b2 < bls; ++b2)
            for (int k = 0; k < NBK; ++k) {
                const int idx = (b2 * heads_per_wg + h2) * TEAM + ((r * NBK + k) << S::SHIFT);
                if (sm_m[idx] != -INFINITY) sum += sm_s[idx] * exp((double)sm_m[idx] - (double)mx);
            }
        const int g2 = blockIdx.y * heads_per_wg + h2;
        const int64_t row = ((int64_t)l * n_q + r / group) * n_q_heads + g2 * group + r % group;
        tmax[row * n_tiles + blockIdx.x] = mx;
        tsum[row * n_tiles + blockIdx.x] = sum;
    }
}

__global__ __launch_bounds__(kScoreThreads) void score_stats_kernel(const float *__restrict__ tmax,
                                                                    const double *__restrict__ tsum,
                                                                    int n_tiles, float *__restrict__ rmax,
                                                                    double *__restrict__ rinvz) {
    __shared__ float sm_f[kScoreThreads / kWave];
    __shared__ double sm_d[kScoreThreads / kWave];
    const int row = blockIdx.x;
    const float *tm = tmax + (int64_t)row * n_tiles;
    const double *ts = tsum + (int64_t)row * n_tiles;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    float mx = -INFINITY;
    for (int i = threadIdx.x; i < n_tiles; i += kScoreThreads) mx = fmaxf(mx, tm[i]);
    mx = wave_max(mx);
    if (lane == 0) sm_f[wave] = mx;
    __syncthreads();
    mx = sm_f[0];
    for (int w = 1; w < kScoreThreads / kWave; ++w) mx = fmaxf(mx, sm_f[w]);
    double z = 0.0;
    for (int i = threadIdx.x; i < n_tiles; i += kScoreThreads)
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

__global__ __launch_bounds__(kScoreThreads) void score_reduce_kernel(
    const float *__restrict__ logits, const float *__restrict__ rmax,
    const double *__restrict__ rinvz, int n_layers, int n_q, int n_q_heads, int n_kv_heads,
    int group, int n_blocks, int n_sink, int n_cand, int mode, float *__restrict__ r32,
    float *__restrict__ scores) {
    const int n_sel = mode == 0 ? 1 : n_layers * n_kv_heads;
    for (int64_t b = (int64_t)blockIdx.x * kScoreThreads + threadIdx.x; b < n_blocks;
         b += (int64_t)gridDim.x * kScoreThreads) {
        const int64_t c = b - n_sink;
        if (c < 0 || c >= n_cand) {
            if (scores)
                for (int s = 0; s < n_sel; ++s) scores[(int64_t)s * n_blocks + b] = INFINITY;
            continue;
        }
        if (mode == 0) {
            // R_b = sum_m mean_{l,h} p_{l,m,h,b}
            double acc = 0.0;
            const int n_rows = n_layers * n_q * n_q_heads;
            for (int row = 0; row < n_rows; ++row)
                acc += (double)expf(logits[(int64_t)row * n_cand + c] - rmax[row]) * rinvz[row];
            const float r = (float)(acc / (double)(n_layers * n_q_heads));
            r32[c] = r;
            if (scores) scores[b] = r;
        } else {
            for (int l = 0; l < n_layers; ++l)
                for (int g = 0; g < n_kv_heads; ++g) {
                    double best = 0.0;
                    for (int m = 0; m < n_q; ++m)
                        for (int hh = 0; hh < group; ++hh) {
                            const int64_t row = ((int64_t)l * n_q + m) * n_q_heads + g * group + hh;
                            const double p = (double)expf(logits[row * n_cand + c] - rmax[row]) * rinvz[row];
                            best = p > best ? p : best;
                        }
                    const int s = l * n_kv_heads + g;
                    r32[(int64_t)s * n_cand + c] = (float)best;
                    if (scores) scores[(int64_t)s * n_blocks + b] = (float)best;
                }
        }
    }
}

template <int D, int RH>
hipError_t launch_logits(const SelectPlan &p, const float *q, const float *index, float scale,
                         float *logits, float *tmax, double *tsum, hipStream_t stream) {
    using S = ScoreShape<D, RH>;
    const int hpw = p.n_kv_heads < S::TEAMS ? p.n_kv_heads : S::TEAMS;
    dim3 grid(p.n_tiles, p.n_kv_heads / hpw, p.n_layers);
    hipLaunchKernelGGL((score_logits_kernel<D, RH>), grid, dim3(kScoreThreads), 0, stream, q, index,
                       p.n_blocks, p.n_kv_heads, p.n_q_heads, p.group, p.n_q, p.n_sink, p.n_cand,
                       p.score_tile, p.n_tiles, hpw, scale, logits, tmax, tsum);
    return hipGetLastError();
}

template <int D>
hipError_t launch_logits_d(const SelectPlan &p, const float *q, const float *index, float scale,
                           float *logits, float *tmax, double *tsum, hipStream_t stream) {
    switch (p.rows_per_head) {
        case 1: return launch_logits<D, 1>(p, q, index, scale, logits, tmax, tsum, stream);
        case 2: return launch_logits<D, 2>(p, q, index, scale, logits, tmax, tsum, stream);
        case 4: return launch_logits<D, 4>(p, q, index, scale, logits, tmax, tsum, stream);
        case 8: return launch_logits<D, 8>(p, q, index, scale, logits, tmax, tsum, stream);
        case 16: return launch_logits<D, 16>(p, q, index, scale, logits, tmax, tsum, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

int score_tile_for(int head_dim, int n_kv_heads, int rows_per_head) {
    const int team = head_dim / 4, teams = kScoreThreads / team;
    const int hpw = n_kv_heads < teams ? n_kv_heads : teams;
    const int nbk = (team / rows_per_head) < 8 ? (team / rows_per_head) : 8;
    const int per_step = nbk * (teams / hpw);
    return per_step > kScoreTile ? per_step : kScoreTile;
}

hipError_t launch_topk(const SelectPlan &p, const float *r32, const int32_t *block_to_page,
                       int32_t *view_blocks, int32_t *view_pages, hipStream_t stream);

hipError_t launch_select(const SelectPlan &p, const float *q, const float *index, float scale,
                         const int32_t *block_to_page, int32_t *view_blocks, int32_t *view_pages,
                         float *scores, char *ws, hipStream_t stream) {
    float *logits = reinterpret_cast<float *>(ws + p.off_logits);
    float *tmax = reinterpret_cast<float *>(ws + p.off_tmax);
    double *tsum = reinterpret_cast<double *>(ws + p.off_tsum);
    float *rmax = reinterpret_cast<float *>(ws + p.off_rmax);
    double *rinvz = reinterpret_cast<double *>(ws + p.off_rinvz);
    float *r32 = reinterpret_cast<float *>(ws + p.off_r32);
    hipError_t e = p.head_dim == 128
                       ? launch_logits_d<128>(p, q, index, scale, logits, tmax, tsum, stream)
                       : launch_logits_d<64>(p, q, index, scale, logits, tmax, tsum, stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(score_stats_kernel, dim3(p.n_rows), dim3(kScoreThreads), 0, stream, tmax, tsum,
                       p.n_tiles, rmax, rinvz);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    int groups = (p.n_blocks + kScoreThreads - 1) / kScoreThreads;
    if (groups > 4096) groups = 4096;
    hipLaunchKernelGGL(score_reduce_kernel, dim3(groups), dim3(kScoreThreads), 0, stream, logits, rmax,
                       rinvz, p.n_layers, p.n_q, p.n_q_heads, p.n_kv_heads, p.group, p.n_blocks,
                       p.n_sink, p.n_cand, p.mode, r32, scores);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_topk(p, r32, block_to_page, view_blocks, view_pages, stream);
}

}  // namespace kvmem
