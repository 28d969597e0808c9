// Mean-K retrieval index (Eq. 9): index[b][g][:] = mean over the Bt keys of
// block b's page for KV head g.
//
// One wave per (block, KV head).  The page slice [Bt][d] is contiguous, so each
// lane reads 16 bytes per token row (a row is d*elem bytes; 64/LPR rows per
// wave instruction) and the loads of a wave cover whole rows.  Sums are kept in
// fp64, where adding at most 64 bf16 or fp32 values of ordinary range is
// exact; the result is rounded once to fp32, so it does not depend on the
// order of summation.
#include <math.h>

#include "kvmem_device.h"
#include "kvmem_internal.h"

namespace kvmem {
namespace {

constexpr int kWavesPerGroup = 4;

template <typename T, int D>
__global__ __launch_bounds__(kWavesPerGroup *kWave) void build_index_kernel(
    const T *__restrict__ k_pool, int64_t n_pages, const int32_t *__restrict__ block_to_page,
    int32_t first_block, int32_t n_blocks, int n_kv_heads, int block_tokens,
    float *__restrict__ index) {
    constexpr int VEC = Vec16<T>::N;  // elements per lane per row
    constexpr int LPR = D / VEC;      // lanes per token row
    constexpr int TG = kWave / LPR;   // token rows per wave instruction
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int64_t pair = (int64_t)blockIdx.x * kWavesPerGroup + wave;
    if (pair >= (int64_t)n_blocks * n_kv_heads) return;  // uniform per wave
    const int32_t b = first_block + (int32_t)(pair / n_kv_heads);
    const int g = (int)(pair % n_kv_heads);
    const int tg = lane / LPR, lp = lane % LPR;
    const int64_t page = block_to_page[b];
    const bool ok = page >= 0 && page < n_pages;

    double acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.0;
    if (ok) {
        const T *base = k_pool + ((page * n_kv_heads + g) * (int64_t)block_tokens) * D + lp * VEC;
        for (int t = tg; t < block_tokens; t += TG) {
            float v[VEC];
            Vec16<T>::load(base + (int64_t)t * D, v);
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[e] += (double)v[e];
        }
    }
#pragma unroll
    for (int o = LPR; o < kWave; o <<= 1)
#pragma unroll
        for (int e = 0; e < VEC; ++e) acc[e] += shfl_xor_d(acc[e], o);
    if (tg == 0) {
        float *dst = index + ((int64_t)b * n_kv_heads + g) * D + lp * VEC;
        const double inv = 1.0 / (double)block_tokens;
        float outv[VEC];
#pragma unroll
        for (int e = 0; e < VEC; ++e) outv[e] = ok ? (float)(acc[e] * inv) : __builtin_nanf("");
#pragma unroll
        for (int e = 0; e < VEC; e += 4)
            *reinterpret_cast<float4 *>(dst + e) = make_float4(outv[e], outv[e + 1], outv[e + 2], outv[e + 3]);
    }
}

template <typename T, int D>
hipError_t launch_t(int n_kv_heads, int block_tokens, const void *k_pool, int64_t n_pages,
                    const int32_t *block_to_page, int32_t first_block, int32_t n_blocks,
                    float *index, hipStream_t stream) {
    const int64_t pairs = (int64_t)n_blocks * n_kv_heads;
    const int64_t groups = (pairs + kWavesPerGroup - 1) / kWavesPerGroup;
    hipLaunchKernelGGL((build_index_kernel<T, D>), dim3((unsigned)groups), dim3(kWavesPerGroup * kWave),
                       0, stream, static_cast<const T *>(k_pool), n_pages, block_to_page,
                       first_block, n_blocks, n_kv_heads, block_tokens, index);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_build_index(int kv_dtype, int head_dim, int n_kv_heads, int block_tokens,
                              const void *k_pool, int64_t n_pages, const int32_t *block_to_page,
                              int32_t first_block, int32_t n_blocks, float *index,
                              hipStream_t stream) {
    if (n_blocks == 0) return hipSuccess;
    const bool bf16 = kv_dtype == 1;
    if (head_dim == 128)
        return bf16 ? launch_t<uint16_t, 128>(n_kv_heads, block_tokens, k_pool, n_pages, block_to_page,
                                              first_block, n_blocks, index, stream)
                    : launch_t<float, 128>(n_kv_heads, block_tokens, k_pool, n_pages, block_to_page,
                                           first_block, n_blocks, index, stream);
    return bf16 ? launch_t<uint16_t, 64>(n_kv_heads, block_tokens, k_pool, n_pages, block_to_page,
                                         first_block, n_blocks, index, stream)
                : launch_t<float, 64>(n_kv_heads, block_tokens, k_pool, n_pages, block_to_page,
                                      first_block, n_blocks, index, stream);
}

}  // namespace kvmem
