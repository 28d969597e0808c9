// Position handling of the execution view (Sec. 4.3 index construction,
// Sec. 4.4 execution view, Sec. 5.3 copy-free assembly), RoPE in rotate-half
// form: for j < d/2 the pair (x_j, x_{j+d/2}) at position p turns by the
// angle a = p * f_j with f_j = base^(-2j/d) (the frequencies come from the
// host).  Angles are formed in fp64 and reduced in fp64 (rope_cos_sin), so
// even positions far beyond the window lose nothing before the fp32 sin/cos.
//
//   rope_materialize  block i: K of page src[i] of the position-independent
//                     pool is re-encoded at positions pos[i] + t and written to
//                     page dst[i] of the execution pool; V is copied as is.
//   rope_delta        in place: K of page pages[i] turns by delta[i]
//                     positions (a GPU-resident block whose compact position
//                     moved); every token of the page turns by the same angle.
//
// The (cos, sin) of a page's angles are computed once per workgroup into LDS
// (they depend on the token and the pair, not on the head).  A lane owns VEC
// consecutive pairs of one token row: it loads the matching 16-byte slices of
// the row's two halves, rotates in fp32 and stores them back (bf16 by round to
// nearest even).  Both kernels are streams: the bytes
// moved are the roofline.
#include <math.h>

#include "kvmem_device.h"
#include "kvmem_internal.h"

namespace kvmem {
namespace {

constexpr int kRopeThreads = 256;
constexpr int kMaxBt = 64;  // largest block_tokens

template <typename T>
struct Lanes;
template <>
struct Lanes<float> {
    static constexpr int VEC = 4;
    __device__ static void load(const float *p, float (&x)[4]) {
        const float4 v = *reinterpret_cast<const float4 *>(p);
        x[0] = v.x; x[1] = v.y; x[2] = v.z; x[3] = v.w;
    }
    __device__ static void store(float *p, const float (&x)[4]) {
        *reinterpret_cast<float4 *>(p) = make_float4(x[0], x[1], x[2], x[3]);
    }
};
template <>
struct Lanes<uint16_t> {
    static constexpr int VEC = 8;
    __device__ static void load(const uint16_t *p, float (&x)[8]) {
        const uint4 v = *reinterpret_cast<const uint4 *>(p);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            x[2 * i] = __uint_as_float(w[i] << 16);
            x[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
    __device__ static uint32_t rne(float f) {  // bf16 bits, round to nearest even (NaN kept)
        const uint32_t u = __float_as_uint(f);
        if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
        return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
    }
    __device__ static void store(uint16_t *p, const float (&x)[8]) {
        uint32_t w[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) w[i] = rne(x[2 * i]) | (rne(x[2 * i + 1]) << 16);
        *reinterpret_cast<uint4 *>(p) = make_uint4(w[0], w[1], w[2], w[3]);
    }
};

// Rotate a row slice: x0 = dims [j0, j0+VEC), x1 = dims [j0+d/2, ...), by
// the angles whose (cos, sin) are cs[0 .. VEC).
template <int VEC>
__device__ inline void rotate(float (&x0)[VEC], float (&x1)[VEC], const float2 *cs) {
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
        const float2 t = cs[e];
        const float a = x0[e], b = x1[e];
        x0[e] = a * t.x - b * t.y;
        x1[e] = a * t.y + b * t.x;
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kRopeThreads) void rope_materialize_kernel(
    const T *__restrict__ raw_k, const T *__restrict__ v_src, int64_t n_src_pages,
    const int32_t *__restrict__ src_pages, const int64_t *__restrict__ positions,
    const int32_t *__restrict__ dst_pages, T *__restrict__ k_dst, T *__restrict__ v_dst,
    int64_t n_dst_pages, int n_kv_heads, int block_tokens, RopeFreqs fr, const int32_t *__restrict__ n_dev) {
    using L = Lanes<T>;
    constexpr int VEC = L::VEC, HL = D / 2 / VEC;  // lanes per half row
    __shared__ float2 cs[kMaxBt * (D / 2)];        // (cos, sin) per (token, pair), shared by the heads
    const int i = blockIdx.x;
    if (n_dev && i >= *n_dev) return;  // the list's length is known on the device only
    const int64_t src = src_pages[i], dst = dst_pages[i];
    if (dst < 0 || dst >= n_dst_pages) return;  // nowhere to write
    const bool src_ok = src >= 0 && src < n_src_pages;
    const int64_t p0 = positions[i];
    for (int k = threadIdx.x; k < block_tokens * (D / 2); k += kRopeThreads) {
        float c, sn;
        rope_cos_sin(p0 + k / (D / 2), fr.f[k % (D / 2)], &c, &sn);
        cs[k] = make_float2(c, sn);
    }
    __syncthreads();
    const int64_t page_elems = (int64_t)n_kv_heads * block_tokens * D;
    const T *ks = raw_k + (src_ok ? src : 0) * page_elems;
    const T *vs = v_src + (src_ok ? src : 0) * page_elems;
    T *kd = k_dst + dst * page_elems;
    T *vd = v_dst + dst * page_elems;
    const int rows = n_kv_heads * block_tokens;  // (head, token) rows of the page
    for (int task = threadIdx.x; task < rows * HL; task += kRopeThreads) {
        const int row = task / HL, c = task % HL;
        const int t = row % block_tokens;
        const int64_t o0 = (int64_t)row * D + c * VEC, o1 = o0 + D / 2;
        float x0[VEC], x1[VEC], y0[VEC], y1[VEC];
        if (src_ok) {
            L::load(ks + o0, x0);
            L::load(ks + o1, x1);
            rotate<VEC>(x0, x1, cs + t * (D / 2) + c * VEC);
            L::load(vs + o0, y0);
            L::load(vs + o1, y1);
        } else {
#pragma unroll
            for (int e = 0; e < VEC; ++e) x0[e] = x1[e] = y0[e] = y1[e] = __builtin_nanf("");
        }
        L::store(kd + o0, x0);
        L::store(kd + o1, x1);
        L::store(vd + o0, y0);
        L::store(vd + o1, y1);
    }
}

template <typename T, int D>
__global__ __launch_bounds__(kRopeThreads) void rope_delta_kernel(
    T *__restrict__ k_pool, int64_t n_pages, const int32_t *__restrict__ pages,
    const int64_t *__restrict__ delta, int n_kv_heads, int block_tokens, RopeFreqs fr,
    const int32_t *__restrict__ n_dev) {
    using L = Lanes<T>;
    constexpr int VEC = L::VEC, HL = D / 2 / VEC;
    __shared__ float2 cs[D / 2];  // every token of the page turns by the same angles
    if (n_dev && (int)blockIdx.x >= *n_dev) return;
    const int64_t page = pages[blockIdx.x];
    if (page < 0 || page >= n_pages) return;
    const int64_t dp = delta[blockIdx.x];
    for (int k = threadIdx.x; k < D / 2; k += kRopeThreads) {
        float c, sn;
        rope_cos_sin(dp, fr.f[k], &c, &sn);
        cs[k] = make_float2(c, sn);
    }
    __syncthreads();
    const int64_t page_elems = (int64_t)n_kv_heads * block_tokens * D;
    T *k = k_pool + page * page_elems;
    const int rows = n_kv_heads * block_tokens;
    for (int task = threadIdx.x; task < rows * HL; task += kRopeThreads) {
        const int row = task / HL, c = task % HL;
        const int64_t o0 = (int64_t)row * D + c * VEC, o1 = o0 + D / 2;
        float x0[VEC], x1[VEC];
        L::load(k + o0, x0);
        L::load(k + o1, x1);
        rotate<VEC>(x0, x1, cs + c * VEC);
        L::store(k + o0, x0);
        L::store(k + o1, x1);
    }
}

template <int D>
hipError_t materialize_d(int kv_dtype, const void *raw_k, const void *v_src, int64_t n_src_pages,
                         const int32_t *src_pages, const int64_t *positions, const int32_t *dst_pages,
                         int32_t n, void *k_dst, void *v_dst, int64_t n_dst_pages, int n_kv_heads,
                         int block_tokens, const RopeFreqs &fr, hipStream_t stream, const int32_t *n_dev) {
    if (kv_dtype == 1)
        hipLaunchKernelGGL((rope_materialize_kernel<uint16_t, D>), dim3(n), dim3(kRopeThreads), 0, stream,
                           static_cast<const uint16_t *>(raw_k), static_cast<const uint16_t *>(v_src),
                           n_src_pages, src_pages, positions, dst_pages, static_cast<uint16_t *>(k_dst),
                           static_cast<uint16_t *>(v_dst), n_dst_pages, n_kv_heads, block_tokens, fr, n_dev);
    else
        hipLaunchKernelGGL((rope_materialize_kernel<float, D>), dim3(n), dim3(kRopeThreads), 0, stream,
                           static_cast<const float *>(raw_k), static_cast<const float *>(v_src), n_src_pages,
                           src_pages, positions, dst_pages, static_cast<float *>(k_dst),
                           static_cast<float *>(v_dst), n_dst_pages, n_kv_heads, block_tokens, fr, n_dev);
    return hipGetLastError();
}

template <int D>
hipError_t delta_d(int kv_dtype, void *k_pool, int64_t n_pages, const int32_t *pages, const int64_t *delta,
                   int32_t n, int n_kv_heads, int block_tokens, const RopeFreqs &fr, hipStream_t stream,
                   const int32_t *n_dev) {
    if (kv_dtype == 1)
        hipLaunchKernelGGL((rope_delta_kernel<uint16_t, D>), dim3(n), dim3(kRopeThreads), 0, stream,
                           static_cast<uint16_t *>(k_pool), n_pages, pages, delta, n_kv_heads, block_tokens, fr,
                           n_dev);
    else
        hipLaunchKernelGGL((rope_delta_kernel<float, D>), dim3(n), dim3(kRopeThreads), 0, stream,
                           static_cast<float *>(k_pool), n_pages, pages, delta, n_kv_heads, block_tokens, fr,
                           n_dev);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_materialize(int kv_dtype, int head_dim, int n_kv_heads, int block_tokens,
                              const RopeFreqs &fr, const void *raw_k, const void *v_src,
                              int64_t n_src_pages, const int32_t *src_pages, const int64_t *positions,
                              const int32_t *dst_pages, int32_t n, void *k_dst, void *v_dst,
                              int64_t n_dst_pages, hipStream_t stream, const int32_t *n_dev) {
    if (n == 0) return hipSuccess;
    return head_dim == 128
               ? materialize_d<128>(kv_dtype, raw_k, v_src, n_src_pages, src_pages, positions, dst_pages, n,
                                    k_dst, v_dst, n_dst_pages, n_kv_heads, block_tokens, fr, stream, n_dev)
               : materialize_d<64>(kv_dtype, raw_k, v_src, n_src_pages, src_pages, positions, dst_pages, n,
                                   k_dst, v_dst, n_dst_pages, n_kv_heads, block_tokens, fr, stream, n_dev);
}

hipError_t launch_rope_delta(int kv_dtype, int head_dim, int n_kv_heads, int block_tokens, const RopeFreqs &fr,
                             void *k_pool, int64_t n_pages, const int32_t *pages, const int64_t *delta,
                             int32_t n, hipStream_t stream, const int32_t *n_dev) {
    if (n == 0) return hipSuccess;
    return head_dim == 128 ? delta_d<128>(kv_dtype, k_pool, n_pages, pages, delta, n, n_kv_heads, block_tokens,
                                          fr, stream, n_dev)
                           : delta_d<64>(kv_dtype, k_pool, n_pages, pages, delta, n, n_kv_heads, block_tokens,
                                         fr, stream, n_dev);
}

}  // namespace kvmem
