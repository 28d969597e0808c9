// Device-side helpers for the KVMem kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace kvmem {

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// One 16-byte load of K/V elements widened to fp32.  bf16 values are stored as
// raw 16-bit patterns; widening is exact.
template <typename T>
struct Vec16;

template <>
struct Vec16<float> {
    static constexpr int N = 4;
    __device__ static inline void load(const float *p, float (&out)[4]) {
        float4 v = *reinterpret_cast<const float4 *>(p);
        out[0] = v.x; out[1] = v.y; out[2] = v.z; out[3] = v.w;
    }
};

template <>
struct Vec16<uint16_t> {
    static constexpr int N = 8;
    __device__ static inline void load(const uint16_t *p, float (&out)[8]) {
        uint4 v = *reinterpret_cast<const uint4 *>(p);
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            out[2 * i] = __uint_as_float(w[i] << 16);
            out[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
};

__device__ inline float shfl_xor_f(float v, int mask) { return __shfl_xor(v, mask, kWave); }
__device__ inline double shfl_xor_d(double v, int mask) { return __shfl_xor(v, mask, kWave); }

// Reduce N partial values held by every lane of a team of W consecutive lanes
// (W, N powers of two, N <= W) so that the team's total of value v ends up in
// the lanes whose in-team index i satisfies i >> log2(W/N) == v.  The first
// log2(N) butterfly steps halve the value array at each step (each lane keeps
// half and sends the other half to its partner); the remaining steps are a
// plain butterfly sum.  Uses N-1 + log2(W/N) shuffles instead of N*log2(W).
template <int N, int W>
__device__ inline float team_transpose_reduce(float (&v)[N], int lane_in_team) {
    static_assert((N & (N - 1)) == 0 && (W & (W - 1)) == 0 && N <= W, "powers of two, N <= W");
    int n = N;
    int off = W / 2;
#pragma unroll
    for (int step = 0; (N >> step) > 1; ++step) {
        const int half = N >> (step + 1);
        const bool upper = (lane_in_team & off) != 0;
#pragma unroll
        for (int k = 0; k < half; ++k) {
            float send = upper ? v[k] : v[k + half];
            float keep = upper ? v[k + half] : v[k];
            v[k] = keep + shfl_xor_f(send, off);
        }
        off >>= 1;
        n = half;
    }
    float r = v[0];
#pragma unroll
    for (int o = W / (2 * N); o >= 1; o >>= 1) r += shfl_xor_f(r, o);
    (void)n;
    return r;
}

// Sum over the W consecutive lanes of a team; every lane receives the total.
template <int W>
__device__ inline float team_sum(float v) {
#pragma unroll
    for (int o = W / 2; o >= 1; o >>= 1) v += shfl_xor_f(v, o);
    return v;
}

__device__ inline float wave_max(float v) {
#pragma unroll
    for (int o = kWave / 2; o >= 1; o >>= 1) v = fmaxf(v, shfl_xor_f(v, o));
    return v;
}

__device__ inline double wave_sum_d(double v) {
#pragma unroll
    for (int o = kWave / 2; o >= 1; o >>= 1) v += shfl_xor_d(v, o);
    return v;
}

// Exclusive prefix sum of one uint32 per thread across a workgroup of
// NT threads (multiple of 64).  `scratch` needs NT/64 + 1 entries.  Returns
// the exclusive prefix; *total receives the workgroup sum.
template <int NT>
__device__ inline uint32_t block_exclusive_scan(uint32_t x, uint32_t *scratch, uint32_t *total) {
    constexpr int NW = NT / kWave;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    uint32_t incl = x;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        uint32_t y = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += y;
    }
    if (lane == kWave - 1) scratch[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        uint32_t t = lane < NW ? scratch[lane] : 0u;
        uint32_t ti = t;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            uint32_t y = __shfl_up(ti, o, kWave);
            if (lane >= o) ti += y;
        }
        if (lane < NW) scratch[lane] = ti - t;  // exclusive wave offsets
        if (lane == NW - 1) scratch[NW] = ti;
    }
    __syncthreads();
    uint32_t res = scratch[wave] + incl - x;
    *total = scratch[NW];
    __syncthreads();
    return res;
}

}  // namespace kvmem
