// Decode attention over the execution view through its page table (Sec. 4.4,
// Sec. 5.3): split-K flash-decode plus an exact log-sum-exp merge.
//
// attn_splitk: one workgroup per (split of the view, KV head, chunk of query
// rows).  The rows of a KV head are the G * n_q (query token, query head) pairs
// that read it (GQA), so every K/V byte fetched serves all of them.  A token's
// row of d elements is read by LPT = d*elem/16 consecutive lanes, 16 bytes
// each, so one wave instruction covers TPW = 64/LPT whole rows of a page; the
// 4 waves of a workgroup take the split's pages in turn.  Each lane keeps the
// query rows' values for its 16-byte slice in registers.  Logits are summed
// across the LPT lanes with a butterfly, then a page's tokens update an online
// softmax (running max, sum, and output accumulator per row) in base 2.  The
// per-lane-group and per-wave states are merged at the end and one partial
// (O, max, sum) per row is written for the split.
//
// attn_combine: merges the splits of each (KV head, row) exactly:
//   M = max_s m_s,  L = sum_s l_s 2^(m_s - M),  out = sum_s O_s 2^(m_s - M) / L.
#include <math.h>

#include "kvmem_device.h"
#include "kvmem_internal.h"

namespace kvmem {
namespace {

constexpr int kAttnWaves = 4;
constexpr int kAttnThreads = kAttnWaves * kWave;

template <typename T, int D, int BT, int RH>
__global__ __launch_bounds__(kAttnThreads) void attn_splitk_kernel(
    const float *__restrict__ q, const T *__restrict__ k_pool, const T *__restrict__ v_pool,
    int64_t n_pages, const int32_t *__restrict__ view_pages, int n_sel, int n_view,
    int last_page_tokens, int n_kv_heads, int n_q_heads, int group, int rows_total,
    int pages_per_split, int n_splits, float qscale, float *__restrict__ part) {
    constexpr int VEC = Vec16<T>::N;
    constexpr int LPT = D / VEC;      // lanes per token row
    constexpr int TPW = kWave / LPT;  // token rows per wave instruction
    constexpr int NI = BT / TPW;      // tokens of a page per lane group
    static_assert(NI >= 1, "page smaller than one wave step");
    __shared__ float sm_o[kAttnWaves][RH][D];
    __shared__ float sm_m[kAttnWaves][RH], sm_l[kAttnWaves][RH];
    __shared__ int sm_bad[kAttnWaves];

    const int split = blockIdx.x, g = blockIdx.y, row0 = blockIdx.z * RH;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int lg = lane / LPT, lp = lane % LPT;
    const int32_t *vpages = view_pages + (int64_t)(n_sel == 1 ? 0 : g) * n_view;
    const int p_begin = split * pages_per_split;
    const int p_end = min(n_view, p_begin + pages_per_split);

    float qr[RH][VEC];
#pragma unroll
    for (int r = 0; r < RH; ++r) {
        const int row = row0 + r, m = row / group, hh = row % group;
        const float *qp = q + ((int64_t)m * n_q_heads + g * group + hh) * D + lp * VEC;
#pragma unroll
        for (int e = 0; e < VEC; e += 4) {
            const float4 v = *reinterpret_cast<const float4 *>(qp + e);
            qr[r][e] = v.x * qscale; qr[r][e + 1] = v.y * qscale;
            qr[r][e + 2] = v.z * qscale; qr[r][e + 3] = v.w * qscale;
        }
    }
    float mrun[RH], lrun[RH], o[RH][VEC];
#pragma unroll
    for (int r = 0; r < RH; ++r) {
        mrun[r] = -INFINITY;
        lrun[r] = 0.f;
#pragma unroll
        for (int e = 0; e < VEC; ++e) o[r][e] = 0.f;
    }
    int bad = 0;

    for (int pi = p_begin + wave; pi < p_end; pi += kAttnWaves) {
        const int64_t page = vpages[pi];
        if (page < 0 || page >= n_pages) {
            bad = 1;
            continue;
        }
        const int ntok = pi == n_view - 1 ? last_page_tokens : BT;
        const int64_t base = ((page * n_kv_heads + g) * (int64_t)BT) * D + lp * VEC;
        float sc[NI][RH];
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int t = i * TPW + lg;
            float kx[VEC];
            if (t < ntok) {
                Vec16<T>::load(k_pool + base + (int64_t)t * D, kx);
            } else {
#pragma unroll
                for (int e = 0; e < VEC; ++e) kx[e] = 0.f;
            }
#pragma unroll
            for (int r = 0; r < RH; ++r) {
                float acc = 0.f;
#pragma unroll
                for (int e = 0; e < VEC; ++e) acc += qr[r][e] * kx[e];
                acc = team_sum<LPT>(acc);
                sc[i][r] = t < ntok ? acc : -INFINITY;
            }
        }
        float msafe[RH];
#pragma unroll
        for (int r = 0; r < RH; ++r) {
            float cm = sc[0][r];
#pragma unroll
            for (int i = 1; i < NI; ++i) cm = fmaxf(cm, sc[i][r]);
            const float mn = fmaxf(mrun[r], cm);
            msafe[r] = mn == -INFINITY ? 0.f : mn;
            const float alpha = exp2f(mrun[r] - msafe[r]);
            lrun[r] *= alpha;
#pragma unroll
            for (int e = 0; e < VEC; ++e) o[r][e] *= alpha;
            mrun[r] = mn;
        }
#pragma unroll
        for (int i = 0; i < NI; ++i) {
            const int t = i * TPW + lg;
            if (t < ntok) {
                float vx[VEC];
                Vec16<T>::load(v_pool + base + (int64_t)t * D, vx);
#pragma unroll
                for (int r = 0; r < RH; ++r) {
                    const float p = exp2f(sc[i][r] - msafe[r]);
                    lrun[r] += p;
#pragma unroll
                    for (int e = 0; e < VEC; ++e) o[r][e] += p * vx[e];
                }
            }
        }
    }

    // merge the TPW lane groups of this wave (lanes lp, lp+LPT, ...)
#pragma unroll
    for (int r = 0; r < RH; ++r) {
        float mx = mrun[r];
#pragma unroll
        for (int off = LPT; off < kWave; off <<= 1) mx = fmaxf(mx, shfl_xor_f(mx, off));
        const float f = mrun[r] == -INFINITY ? 0.f : exp2f(mrun[r] - mx);
        float l = lrun[r] * f;
#pragma unroll
        for (int off = LPT; off < kWave; off <<= 1) l += shfl_xor_f(l, off);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            float x = o[r][e] * f;
#pragma unroll
            for (int off = LPT; off < kWave; off <<= 1) x += shfl_xor_f(x, off);
            o[r][e] = x;
        }
        if (lg == 0) {
#pragma unroll
            for (int e = 0; e < VEC; ++e) sm_o[wave][r][lp * VEC + e] = o[r][e];
        }
        if (lane == 0) {
            sm_m[wave][r] = mx;
            sm_l[wave][r] = l;
        }
    }
    // any lane of the wave saw a bad page -> whole wave reports it
    if (lane == 0) sm_bad[wave] = 0;
    __syncthreads();
    if (bad) atomicOr(&sm_bad[wave], 1);
    __syncthreads();
    const bool any_bad = sm_bad[0] | sm_bad[1] | sm_bad[2] | sm_bad[3];
    for (int idx = threadIdx.x; idx < RH * D; idx += kAttnThreads) {
        const int r = idx / D, d = idx % D;
        float mx = sm_m[0][r];
#pragma unroll
        for (int w = 1; w < kAttnWaves; ++w) mx = fmaxf(mx, sm_m[w][r]);
        float acc = 0.f, l = 0.f;
#pragma unroll
        for (int w = 0; w < kAttnWaves; ++w) {
            const float f = sm_m[w][r] == -INFINITY ? 0.f : exp2f(sm_m[w][r] - mx);
            acc += sm_o[w][r][d] * f;
            l += sm_l[w][r] * f;
        }
        float *dst = part + (((int64_t)g * n_splits + split) * rows_total + row0 + r) * (D + 2);
        dst[d] = any_bad ? __builtin_nanf("") : acc;
        if (d == 0) {
            dst[D] = mx;
            dst[D + 1] = l;
        }
    }
}

template <int D>
__global__ __launch_bounds__(D) void attn_combine_kernel(const float *__restrict__ part, int n_splits,
                                                         int rows_total, int n_q_heads, int group,
                                                         float *__restrict__ out,
                                                         float *__restrict__ lse) {
    const int g = blockIdx.x / rows_total, r = blockIdx.x % rows_total, d = threadIdx.x;
    const int64_t stride = (int64_t)rows_total * (D + 2);
    const float *pr = part + ((int64_t)g * n_splits * rows_total + r) * (D + 2);
    float mx = -INFINITY;
    for (int s = 0; s < n_splits; ++s) mx = fmaxf(mx, pr[s * stride + D]);
    float acc = 0.f, l = 0.f;
    for (int s = 0; s < n_splits; ++s) {
        const float ms = pr[s * stride + D];
        const float f = ms == -INFINITY ? 0.f : exp2f(ms - mx);
        acc += pr[s * stride + d] * f;
        l += pr[s * stride + D + 1] * f;
    }
    const int m = r / group, h = (blockIdx.x / rows_total) * group + r % group;
    out[((int64_t)m * n_q_heads + h) * D + d] = acc / l;
    if (lse && d == 0) lse[(int64_t)m * n_q_heads + h] = (mx + log2f(l)) * kLn2;
}

template <typename T, int D, int BT, int RH>
hipError_t launch_rh(const AttnPlan &p, const float *q, const void *k_pool, const void *v_pool,
                     int64_t n_pages, const int32_t *view_pages, float qscale, float *part,
                     hipStream_t stream) {
    dim3 grid(p.n_splits, p.n_kv_heads, p.rows_per_head / RH);
    hipLaunchKernelGGL((attn_splitk_kernel<T, D, BT, RH>), grid, dim3(kAttnThreads), 0, stream, q,
                       static_cast<const T *>(k_pool), static_cast<const T *>(v_pool), n_pages,
                       view_pages, p.n_sel, p.n_view, p.last_page_tokens, p.n_kv_heads, p.n_q_heads,
                       p.group, p.rows_per_head, p.pages_per_split, p.n_splits, qscale, part);
    return hipGetLastError();
}

template <typename T, int D, int BT>
hipError_t launch_bt(const AttnPlan &p, const float *q, const void *k, const void *v, int64_t n_pages,
                     const int32_t *vp, float qscale, float *part, hipStream_t stream) {
    const int rows = p.rows_per_head;
    if (rows % 8 == 0) return launch_rh<T, D, BT, 8>(p, q, k, v, n_pages, vp, qscale, part, stream);
    if (rows % 4 == 0) return launch_rh<T, D, BT, 4>(p, q, k, v, n_pages, vp, qscale, part, stream);
    if (rows % 2 == 0) return launch_rh<T, D, BT, 2>(p, q, k, v, n_pages, vp, qscale, part, stream);
    return launch_rh<T, D, BT, 1>(p, q, k, v, n_pages, vp, qscale, part, stream);
}

template <typename T, int D>
hipError_t launch_d(const AttnPlan &p, const float *q, const void *k, const void *v, int64_t n_pages,
                    const int32_t *vp, float qscale, float *part, hipStream_t stream) {
    switch (p.block_tokens) {
        case 16: return launch_bt<T, D, 16>(p, q, k, v, n_pages, vp, qscale, part, stream);
        case 32: return launch_bt<T, D, 32>(p, q, k, v, n_pages, vp, qscale, part, stream);
        case 64: return launch_bt<T, D, 64>(p, q, k, v, n_pages, vp, qscale, part, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace

hipError_t launch_sparse_attn(const AttnPlan &p, const float *q, const void *k_pool,
                              const void *v_pool, int64_t n_pages, const int32_t *view_pages,
                              float scale, float *out, float *lse, char *ws, hipStream_t stream) {
    float *part = reinterpret_cast<float *>(ws + p.off_part);
    const float qscale = scale * kLog2e;
    hipError_t e;
    const bool bf16 = p.kv_dtype == 1;
    if (p.head_dim == 128)
        e = bf16 ? launch_d<uint16_t, 128>(p, q, k_pool, v_pool, n_pages, view_pages, qscale, part, stream)
                 : launch_d<float, 128>(p, q, k_pool, v_pool, n_pages, view_pages, qscale, part, stream);
    else
        e = bf16 ? launch_d<uint16_t, 64>(p, q, k_pool, v_pool, n_pages, view_pages, qscale, part, stream)
                 : launch_d<float, 64>(p, q, k_pool, v_pool, n_pages, view_pages, qscale, part, stream);
    if (e != hipSuccess) return e;
    const dim3 grid(p.n_kv_heads * p.rows_per_head);
    if (p.head_dim == 128)
        hipLaunchKernelGGL((attn_combine_kernel<128>), grid, dim3(128), 0, stream, part, p.n_splits,
                           p.rows_per_head, p.n_q_heads, p.group, out, lse);
    else
        hipLaunchKernelGGL((attn_combine_kernel<64>), grid, dim3(64), 0, stream, part, p.n_splits,
                           p.rows_per_head, p.n_q_heads, p.group, out, lse);
    return hipGetLastError();
}

}  // namespace kvmem
