// Device-side helpers for the KVMem kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace kvmem {

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// 16-byte load of data read exactly once per step (K/V pages, raw keys): the
// non-temporal hint keeps this stream from evicting what is reused from the
// caches (the index, logits and tables of the next kernels).
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
template <typename T>
__device__ inline uint4 load_stream16(const T *p) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// The same for 8 bytes.
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
template <typename T>
__device__ inline uint2 load_stream8(const T *p) {
    const u32x2_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t *>(p));
    return make_uint2(v.x, v.y);
}

// One 16-byte load of K/V elements widened to fp32.  bf16 values are stored as
// raw 16-bit patterns; widening is exact.
template <typename T>
struct Vec16;

template <>
struct Vec16<float> {
    static constexpr int N = 4;
    __device__ static inline void decode(const uint4 &v, float (&out)[4]) {
        out[0] = __uint_as_float(v.x); out[1] = __uint_as_float(v.y);
        out[2] = __uint_as_float(v.z); out[3] = __uint_as_float(v.w);
    }
    __device__ static inline void load(const float *p, float (&out)[4]) { decode(load_stream16(p), out); }
};

template <>
struct Vec16<uint16_t> {
    static constexpr int N = 8;
    __device__ static inline void load(const uint16_t *p, float (&out)[8]) { decode(load_stream16(p), out); }
    __device__ static inline void decode(const uint4 &v, float (&out)[8]) {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            out[2 * i] = __uint_as_float(w[i] << 16);
            out[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
        }
    }
};

// FP8 pools hold OCP E4M3 codes (one byte each).  gfx950's conversion
// instructions read this format: every code, subnormals, -0 and NaN included,
// widens exactly to fp32 and to bf16.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
template <>
struct Vec16<uint8_t> {
    static constexpr int N = 16;
    __device__ static inline void load(const uint8_t *p, float (&out)[16]) { decode(load_stream16(p), out); }
    __device__ static inline void decode(const uint4 &v, float (&out)[16]) {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const f32x2_t lo = __builtin_amdgcn_cvt_pk_f32_fp8(w[i], false);  // bytes 0, 1
            const f32x2_t hi = __builtin_amdgcn_cvt_pk_f32_fp8(w[i], true);   // bytes 2, 3
            out[4 * i] = lo[0]; out[4 * i + 1] = lo[1];
            out[4 * i + 2] = hi[0]; out[4 * i + 3] = hi[1];
        }
    }
};

// cos and sin of the RoPE angle pos * f (fp64).  The angle is reduced to about
// [-pi, pi] with a two-part 2*pi (Cody-Waite, fused multiply-adds), so the
// reduced angle is accurate to about 1e-16 rad for any fp64 angle, then cos
// and sin are taken in fp32.
__device__ inline void rope_cos_sin(int64_t pos, double f, float *c, float *s) {
    constexpr double kTwoPiHi = 6.283185307179586;        // fp64 nearest to 2*pi
    constexpr double kTwoPiLo = 2.4492935982947064e-16;   // 2*pi - kTwoPiHi
    constexpr double kInvTwoPi = 0.15915494309189535;
    const double a = (double)pos * f;
    const double k = rint(a * kInvTwoPi);
    const double r = fma(-k, kTwoPiLo, fma(-k, kTwoPiHi, a));
    sincosf((float)r, s, c);
}

__device__ inline float shfl_xor_f(float v, int mask) { return __shfl_xor(v, mask, kWave); }

// 2^x by the hardware instruction alone (v_exp_f32).  Results below 2^-126
// come out as zero; the softmax weights that use it are relative to a running
// maximum, so such a weight is negligible next to the maximum's own weight 1.
__device__ inline float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// DPP lane patterns inside one 16-lane row (gfx9 encodings; row_newbcast is gfx90a+).
constexpr int kDppRowMirror = 0x140;      // lane i <- lane 15-i
constexpr int kDppRowHalfMirror = 0x141;  // lane i <- lane 7-i within each half row
constexpr int kDppQuadXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int dpp_row_ror(int n) { return 0x120 + n; }       // rotate within the row by n
constexpr int dpp_row_bcast(int n) { return 0x150 + n; }     // lane n of the row to all 16

// Calls f(std::integral_constant<int, i>{}) for i = 0 .. N-1, so that i can be
// used where a constant expression is needed (DPP controls, array indices).
template <typename F, int... I>
__device__ inline void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ inline void static_for(F &&f) {
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

template <int CTRL>
__device__ inline float dpp_f(float x) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum 16 values held by each of the 16 lanes of a DPP row so that lane i ends
// with the row's total of value i.  Four halving steps pair lane i with its
// mirror (bit 3), half-mirror (bit 2) and quad neighbours (bits 1, 0): each lane
// keeps the half of its values selected by that bit and adds the partner's copy
// of the same half.  15 DPP adds for 16 sums; no LDS traffic.
__device__ inline float row_transpose_reduce16(const float (&in)[16], int lp) {
    float v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = in[k];
    {
        const bool up = (lp & 8) != 0;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const float a = v[k] + dpp_f<kDppRowMirror>(v[k]);
            const float b = v[k + 8] + dpp_f<kDppRowMirror>(v[k + 8]);
            v[k] = up ? b : a;
        }
    }
    {
        const bool up = (lp & 4) != 0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const float a = v[k] + dpp_f<kDppRowHalfMirror>(v[k]);
            const float b = v[k + 4] + dpp_f<kDppRowHalfMirror>(v[k + 4]);
            v[k] = up ? b : a;
        }
    }
    {
        const bool up = (lp & 2) != 0;
#pragma unroll
        for (int k = 0; k < 2; ++k) {
            const float a = v[k] + dpp_f<kDppQuadXor2>(v[k]);
            const float b = v[k + 2] + dpp_f<kDppQuadXor2>(v[k + 2]);
            v[k] = up ? b : a;
        }
    }
    {
        const bool up = (lp & 1) != 0;
        const float a = v[0] + dpp_f<kDppQuadXor1>(v[0]);
        const float b = v[1] + dpp_f<kDppQuadXor1>(v[1]);
        v[0] = up ? b : a;
    }
    return v[0];
}
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

// Reductions over a whole wave on the DPP lane paths (no LDS round trip):
// inside each 16-lane row by quad_perm xor 1, xor 2 and row_ror 4, 8 (every
// lane then holds its row's result), then row_bcast:15 takes rows 0 and 2
// into rows 1 and 3 and row_bcast:31 takes row 1 into rows 2 and 3 (rows the
// mask leaves out read the identity), and lane 63's result goes to every lane.
// Every lane of the wave must be active.
constexpr int kDppRowBcast15 = 0x142;
constexpr int kDppRowBcast31 = 0x143;
template <int CTRL, int ROW_MASK = 0xF>
__device__ inline float dpp_or(float x, float identity) {
    return __int_as_float(
        __builtin_amdgcn_update_dpp(__float_as_int(identity), __float_as_int(x), CTRL, ROW_MASK, 0xF, false));
}
template <int CTRL, int ROW_MASK = 0xF>
__device__ inline double dpp_d0(double x) {  // identity 0.0: all bits zero
    const uint64_t b = __double_as_longlong(x);
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, CTRL, ROW_MASK, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), CTRL, ROW_MASK, 0xF, false);
    return __longlong_as_double((int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo));
}

__device__ inline float wave_max(float v) {
    const float id = -INFINITY;
    v = fmaxf(v, dpp_or<kDppQuadXor1>(v, id));
    v = fmaxf(v, dpp_or<kDppQuadXor2>(v, id));
    v = fmaxf(v, dpp_or<dpp_row_ror(4)>(v, id));
    v = fmaxf(v, dpp_or<dpp_row_ror(8)>(v, id));
    v = fmaxf(v, dpp_or<kDppRowBcast15, 0xA>(v, id));
    v = fmaxf(v, dpp_or<kDppRowBcast31, 0xC>(v, id));
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), kWave - 1));
}

// Max and fp64 sum over each 16-lane row (every lane of the row receives its
// row's result): the first four steps of the wave reductions. Every lane of
// the row must be active.
__device__ inline float row16_max(float v) {
    const float id = -INFINITY;
    v = fmaxf(v, dpp_or<kDppQuadXor1>(v, id));
    v = fmaxf(v, dpp_or<kDppQuadXor2>(v, id));
    v = fmaxf(v, dpp_or<dpp_row_ror(4)>(v, id));
    v = fmaxf(v, dpp_or<dpp_row_ror(8)>(v, id));
    return v;
}

__device__ inline double row16_sum_d(double v) {
    v += dpp_d0<kDppQuadXor1>(v);
    v += dpp_d0<kDppQuadXor2>(v);
    v += dpp_d0<dpp_row_ror(4)>(v);
    v += dpp_d0<dpp_row_ror(8)>(v);
    return v;
}

__device__ inline float wave_sum_f(float v) {
    v += dpp_or<kDppQuadXor1>(v, 0.f);
    v += dpp_or<kDppQuadXor2>(v, 0.f);
    v += dpp_or<dpp_row_ror(4)>(v, 0.f);
    v += dpp_or<dpp_row_ror(8)>(v, 0.f);
    v += dpp_or<kDppRowBcast15, 0xA>(v, 0.f);
    v += dpp_or<kDppRowBcast31, 0xC>(v, 0.f);
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), kWave - 1));
}

__device__ inline double wave_sum_d(double v) {
    v += dpp_d0<kDppQuadXor1>(v);
    v += dpp_d0<kDppQuadXor2>(v);
    v += dpp_d0<dpp_row_ror(4)>(v);
    v += dpp_d0<dpp_row_ror(8)>(v);
    v += dpp_d0<kDppRowBcast15, 0xA>(v);
    v += dpp_d0<kDppRowBcast31, 0xC>(v);
    const uint64_t b = __double_as_longlong(v);
    const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)b, kWave - 1);
    const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), kWave - 1);
    return __longlong_as_double((int64_t)(((uint64_t)hi << 32) | lo));
}

// Inclusive prefix sum over the 64 lanes of a wave on the DPP lane paths
// (no LDS round trip): a Kogge-Stone scan inside each 16-lane row by
// row_shr 1, 2, 4, 8, then row_bcast:15 adds row 0's total to row 1 and row
// 2's to row 3, and row_bcast:31 adds the total of rows 0-1 to rows 2-3.
// Lanes without a source (and rows the mask leaves out) add 0.
constexpr int kDppRowShr = 0x110;      // row_shr:n is kDppRowShr + n
__device__ inline uint32_t wave_inclusive_scan(uint32_t x) {
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppRowShr + 1, 0xf, 0xf, false);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppRowShr + 2, 0xf, 0xf, false);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppRowShr + 4, 0xf, 0xf, false);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppRowShr + 8, 0xf, 0xf, false);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppRowBcast15, 0xa, 0xf, false);
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, kDppRowBcast31, 0xc, 0xf, false);
    return x;
}

// Exclusive prefix sum of one uint32 per thread across a workgroup of
// NT threads (multiple of 64).  `scratch` needs NT/64 + 1 entries.  Returns
// the exclusive prefix; *total receives the workgroup sum.
template <int NT>
__device__ inline uint32_t block_exclusive_scan(uint32_t x, uint32_t *scratch, uint32_t *total) {
    constexpr int NW = NT / kWave;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const uint32_t incl = wave_inclusive_scan(x);
    if (lane == kWave - 1) scratch[wave] = incl;
    __syncthreads();
    if (wave == 0) {
        const uint32_t t = lane < NW ? scratch[lane] : 0u;
        const uint32_t ti = wave_inclusive_scan(t);
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
