// Mean-K retrieval index (Eq. 9): for block b and KV head g, the mean over the
// Bt keys of page block_to_page[b], written in the tiled index layout
// (float [ceil(M/64)][Hkv][d/4][64][4]).
//
// One workgroup per (64-block tile, KV head).  Each wave reduces 16 of the
// tile's blocks: a page slice [Bt][d] is contiguous, so LPR = d*elem/16 lanes
// read one token row with 16-byte loads and 64/LPR rows go per instruction;
// the loads of 16 tokens of several blocks are issued together (see below).  Sums are kept in
// fp64: adding Bt <= 64 bf16 values (8-bit significands) or fp32 values whose
// magnitudes span less than 2^23 is exact there, so the result -- rounded once
// to fp32 -- does not depend on the order of summation.  The finished means
// are staged as a [64][d] tile in LDS and written out so that each wave store
// covers 1 KB of contiguous index.  FP8 codes widen exactly, and their sum (Bt
// <= 64 values on a 2^-9 grid below 448, so below 2^15) is exact even in fp32,
// which is where it is kept; in fp64 the sum times k_scale (24 bits) is exact
// too, so the mean is again rounded once.
#include <math.h>

#include "kvmem_device.h"
#include "kvmem_internal.h"

namespace kvmem {
namespace {

constexpr int kWaves = 4;
// blocks per workgroup: a whole index tile, or half of one with RoPE, whose
// (cos, sin) table also takes LDS: the staging of the means (part * (D + 4)
// floats) then leaves room for 4 waves per SIMD instead of 3 (2-7% faster
// at 1M on two boxes; the plain build is 8% slower with half tiles)
template <bool ROPE>
constexpr int part_blocks() { return ROPE ? kIndexTile / 2 : kIndexTile; }

// 4-byte load of raw keys read once (the non-temporal hint of load_stream16)
template <typename T>
__device__ inline uint32_t load_stream4(const T *p) {
    return __builtin_nontemporal_load(reinterpret_cast<const unsigned int *>(p));
}

// ROPE: the stored keys carry RoPE (rotate-half form) at positions
// block_pos[b] + t (block_pos NULL: b * block_tokens + t); each token row is
// turned back to position 0 before it enters the sum (Sec. 4.3: the index is
// built from position-independent keys).  A lane then reads its row as two
// pieces (8 bytes; 4 for FP8 codes), the VEC/2 dims [j0, j0 + VEC/2) and the
// matching dims of the other half, so that it holds both members of its pairs.
// The angle of token t is the fp64 product a_t = (p0 + t) f_j (as in the
// definition), turned into a rotation without a sin/cos per token: with
// a_0 = p0 f_j (its cos/sin taken once per block and pair, the angle reduced
// in fp64 by rope_cos_sin) and the cos/sin of t f_j from a per-workgroup LDS
// table, a_t = a_0 + t f_j + eps, where eps = (a_t - a_0) - t f_j is the
// rounding of the products (computed exactly enough in fp64: a_t - a_0 is
// exact there).  The three rotations are composed in fp32, eps to first order
// (cos eps = 1 - eps^2/2, and eps stays below an fp64 ulp of the angle: 2.4e-4
// rad even at positions of 2^40).  That is sixteen to sixty-four times fewer
// sin/cos than one per token, at about two fp32 ulps of the cos and sin.
// Below kEpsMinPos (2^26) eps is under 1.5e-8 rad and is left out.  From
// kDirectMinPos (2^42) on, eps reaches 5e-4 rad and its dropped second-order
// term (and, past 2^53, the inexact difference a_t - a_0) would show, so such
// blocks take the cos/sin of every token's own angle a_t instead.
//
// Every block_tokens is a multiple of 16, so a wave reads a block 16 tokens
// at a time: NI = 16 / TG loads per lane, all issued before the first sum,
// for BPS blocks at once (about 16 loads of 16 bytes in flight per lane).

constexpr int kMaxBlockTokens = 64;

// Sum over the lanes of the wave that share lane % L (L = 4 .. 32, a power of
// two): inside each 16-lane row by row_ror L, 2L, .. 8 (DPP), then across
// rows by the permlane swaps (xor 16, xor 32), every lane ending with its
// class's sum.  All register moves, no LDS.  Every lane must be active.
template <int CTRL>
__device__ inline uint32_t dpp_u(uint32_t x) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, CTRL, 0xF, 0xF, false);
}
template <int L, typename V>
__device__ inline V sum_lanes_mod(V v) {
    static_assert(L >= 4 && L <= 32 && (L & (L - 1)) == 0, "lane classes of 4 .. 32");
    auto move = [](V x, auto op) {  // apply op to each 32-bit half of x
        if constexpr (sizeof(V) == 8) {
            const uint64_t b = __double_as_longlong(x);
            const uint64_t lo = op((uint32_t)b), hi = op((uint32_t)(b >> 32));
            return __longlong_as_double((int64_t)((hi << 32) | lo));
        } else {
            return __uint_as_float(op(__float_as_uint(x)));
        }
    };
    if constexpr (L <= 4) v += move(v, [](uint32_t x) { return dpp_u<dpp_row_ror(4)>(x); });
    if constexpr (L <= 8) v += move(v, [](uint32_t x) { return dpp_u<dpp_row_ror(8)>(x); });
    auto swap_sum = [&](auto swap) {  // the pair (lane & ~m, lane | m) in that order, for both lanes
        if constexpr (sizeof(V) == 8) {
            const uint64_t b = __double_as_longlong(v);
            const auto lo = swap((uint32_t)b), hi = swap((uint32_t)(b >> 32));
            const double a = __longlong_as_double((int64_t)(((uint64_t)hi[0] << 32) | lo[0]));
            const double c = __longlong_as_double((int64_t)(((uint64_t)hi[1] << 32) | lo[1]));
            return (V)(a + c);
        } else {
            const auto r = swap(__float_as_uint(v));
            return (V)(__uint_as_float(r[0]) + __uint_as_float(r[1]));
        }
    };
    if constexpr (L <= 16)
        v = swap_sum([](uint32_t x) { return __builtin_amdgcn_permlane16_swap(x, x, false, false); });
    v = swap_sum([](uint32_t x) { return __builtin_amdgcn_permlane32_swap(x, x, false, false); });
    return v;
}
constexpr int64_t kEpsMinPos = int64_t(1) << 26;
constexpr int64_t kDirectMinPos = int64_t(1) << 42;

// eps = (a_t - a_0) - t f with each product rounded on its own, as the angle
// a_t = (p0 + t) f is defined (a fused multiply-add would skip a rounding)
__device__ inline float rope_eps(int64_t p0, int t, double f) {
#pragma clang fp contract(off)
    const double at = (double)(p0 + t) * f, a0 = (double)p0 * f, tf = (double)t * f;
    return (float)((at - a0) - tf);
}

// EPS: compile the loop that corrects for the rounding of the angle products
// (blocks at positions of 2^26 or more); it holds about 90 more VGPRs than the
// plain loop, so launches whose positions are known to stay below 2^26 leave
// it out.  With ROPE the (cos, sin) table of t * f_j takes block_tokens * D/2
// float2 of dynamic LDS.
template <typename T, int D, bool ROPE, bool EPS>
__global__ __launch_bounds__(kWaves *kWave) void build_index_kernel(
    const T *__restrict__ k_pool, int64_t n_pages, const int32_t *__restrict__ block_to_page,
    int32_t first_block, int32_t n_blocks, int n_kv_heads, int block_tokens, float k_scale,
    float *__restrict__ index, const int64_t *__restrict__ block_pos, RopeFreqs fr) {
    constexpr bool F8 = sizeof(T) == 1;
    // elements per lane per row.  FP8 keys take 8 (as bf16 does), not the 16
    // of a 16-byte load: the sums of a lane's elements are then exchanged
    // between 4 lanes of a row group instead of 8, over half as many elements
    // (a third of the cross-lane work)
    constexpr int VEC = F8 ? 8 : Vec16<T>::N;
    constexpr int LPR = D / VEC;      // lanes per token row
    constexpr int TG = kWave / LPR;   // token rows per wave instruction
    constexpr int NI = 16 / TG;       // instructions per 16 tokens
    static_assert(NI * TG == 16, "16 tokens split over whole instructions");
    constexpr int PAD = D + 4;        // LDS row stride (floats): conflict-free column reads
    // exact sums: fp32 for unrotated FP8 codes, fp64 otherwise
    using Acc = typename std::conditional<F8 && !ROPE, float, double>::type;
    // blocks per step.  Without RoPE two (8 loads of 16 bytes in flight per
    // lane for bf16 at d = 128, occupancy 4; four blocks held 168 VGPRs at
    // occupancy 3 and were 2-4% slower, eight were slower still).  The
    // rotation's per-block cos/sin take registers, so with RoPE one block per
    // step (at d = 128 the bf16 kernel then holds 83 VGPRs against 181 with
    // two blocks, and the 1M index takes 0.66 ms against 0.84), except in the
    // kernel with the rounding correction
    constexpr int BPS0 = !ROPE ? 2 : (16 / NI > 4 ? 4 : 16 / NI);
    constexpr int BPS = !ROPE || BPS0 == 1 ? BPS0 : (!EPS ? 1 : BPS0 / 2);
    constexpr int RB = ROPE ? BPS : 1, RV = ROPE ? VEC / 2 : 1;  // sizes of the per-block rotation
    constexpr int kPart = part_blocks<ROPE>();
    __shared__ float tile_buf[kPart * PAD];
    // RoPE: (cos, sin) of t * f_j, row t at pitch RP: a wave's reads (rows
    // tg, pairs lp * VEC/2 + e) then fall on distinct banks two lanes at a time
    extern __shared__ float2 rot_t[];
    constexpr int RP = D / 2 + 1;
    // RoPE: (cos, sin) of p0 * f_j for every pair of the wave's current
    // blocks, computed one pair per lane and read back by the TG lanes that
    // hold the pair on their rows (each of which computed it before)
    __shared__ float2 rot_0[ROPE ? kWaves * BPS * (D / 2) : 1];

    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int tg = lane / LPR, lp = lane % LPR;
    const int g = blockIdx.y;
    const int64_t part = first_block / kPart + blockIdx.x;  // this workgroup's kPart blocks
    const int64_t tile = part / (kIndexTile / kPart);
    const int64_t b_tile0 = part * kPart;  // first block of the part
    const int64_t b_lo = b_tile0 > first_block ? b_tile0 : first_block;
    const int64_t b_end = (int64_t)first_block + n_blocks;
    const int64_t b_hi = b_tile0 + kPart < b_end ? b_tile0 + kPart : b_end;
    const double inv = 1.0 / (double)block_tokens, ks = (double)k_scale;
    constexpr int HV = VEC / 2;           // RoPE: pairs per lane
    const int j0 = lp * HV;               // RoPE: the lane's first pair
    if constexpr (ROPE) {
        for (int i = threadIdx.x; i < block_tokens * (D / 2); i += kWaves * kWave) {
            float c, sn;
            rope_cos_sin(i / (D / 2), fr.f[i % (D / 2)], &c, &sn);
            rot_t[(i / (D / 2)) * RP + i % (D / 2)] = make_float2(c, sn);
        }
        __syncthreads();
    }

    // The page (and RoPE position) of each of the wave's kPart / kWaves
    // slots, one clamped load per lane up front: the steps below take them
    // from this lane instead of a dependent memory round trip each.
    constexpr int kSlots = kPart / kWaves;
    static_assert(kSlots <= kWave, "one slot per lane");
    int32_t slot_page = -1;
    int64_t slot_pos = 0;
    {
        const int64_t b = b_tile0 + wave + (int64_t)kWaves * lane;
        const bool in = lane < kSlots && b >= b_lo && b < b_hi;
        const int64_t bc = in ? b : b_lo;
        const int32_t pg = block_to_page[bc];
        slot_page = in ? pg : -1;
        if constexpr (ROPE) slot_pos = block_pos ? block_pos[bc] : b * (int64_t)block_tokens;
    }
    // wave w reduces the part's slots w, w+4, w+8, ... (BPS at a time)
    for (int s0 = wave; s0 < kPart; s0 += kWaves * BPS) {
        Acc acc[BPS][VEC];
        double mean[VEC];
        bool ok[BPS];
        const T *base[BPS];
        float c0[RB][RV], s0v[RB][RV];  // cos, sin of a_0 = p0 * f_j for the lane's pairs
        int64_t p0[RB];
        bool far[RB];   // positions reach kEpsMinPos: correct for the rounding of the products
        bool vfar[RB];  // positions reach kDirectMinPos: every token's own cos/sin
#pragma unroll
        for (int k = 0; k < BPS; ++k) {
            const int64_t b = b_tile0 + s0 + k * kWaves;
            const int m = (s0 - wave) / kWaves + k;  // the block's slot (wave-uniform)
            const bool in = b >= b_lo && b < b_hi;
            const int64_t page = in ? __builtin_amdgcn_readlane(slot_page, m) : -1;
            ok[k] = in && page >= 0 && page < n_pages;
            // a block outside the range or without a valid page reads page 0
            // (in bounds) and is written as NaN
            base[k] = k_pool + ((ok[k] ? page : 0) * n_kv_heads + g) * (int64_t)block_tokens * D +
                      (ROPE ? j0 : lp * VEC);
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[k][e] = 0;
            if constexpr (ROPE) {
                const int64_t pm = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(slot_pos >> 32), m) << 32) |
                                             (uint32_t)__builtin_amdgcn_readlane((int)slot_pos, m));
                p0[k] = block_pos && ok[k] ? pm : b * (int64_t)block_tokens;
                far[k] = !(p0[k] > -kEpsMinPos && p0[k] + block_tokens <= kEpsMinPos);
                vfar[k] = !(p0[k] > -kDirectMinPos && p0[k] + block_tokens <= kDirectMinPos);
                float2 *r0 = rot_0 + (wave * BPS + k) * (D / 2);
                for (int j = lane; j < D / 2; j += kWave) {
                    float c, sn;
                    rope_cos_sin(p0[k], fr.f[j], &c, &sn);
                    r0[j] = make_float2(c, sn);
                }
#pragma unroll
                for (int e = 0; e < HV; ++e) {
                    const float2 cs = r0[j0 + e];
                    c0[k][e] = cs.x;
                    s0v[k][e] = cs.y;
                }
            }
        }
        // the token loop, compiled without and with the rounding correction
        // (mode 0, 1) and with every token's own cos/sin (mode 2)
        auto sum_tokens = [&](auto mode) {
            for (int t0 = 0; t0 < block_tokens; t0 += 16) {
                uint4 raw[BPS][NI];
#pragma unroll
                for (int k = 0; k < BPS; ++k)
#pragma unroll
                    for (int i = 0; i < NI; ++i) {
                        const T *row = base[k] + (int64_t)(t0 + tg + TG * i) * D;
                        if constexpr (ROPE && F8) {
                            raw[k][i] = make_uint4(load_stream4(row), load_stream4(row + D / 2), 0u, 0u);
                        } else if constexpr (F8) {
                            const uint2 w = load_stream8(row);
                            raw[k][i] = make_uint4(w.x, w.y, 0u, 0u);
                        } else if constexpr (ROPE) {
                            const uint2 lo = load_stream8(row), hi = load_stream8(row + D / 2);
                            raw[k][i] = make_uint4(lo.x, lo.y, hi.x, hi.y);
                        } else {
                            raw[k][i] = load_stream16(row);
                        }
                    }
#pragma unroll
                for (int i = 0; i < NI; ++i) {
                    const int t = t0 + tg + TG * i;
                    float2 rt[RV];
                    if constexpr (ROPE) {
#pragma unroll
                        for (int e = 0; e < HV; ++e) rt[e] = rot_t[t * RP + j0 + e];
                    }
#pragma unroll
                    for (int k = 0; k < BPS; ++k) {
                        float v[VEC];
                        if constexpr (F8) {  // 8 codes in two words (RoPE: 4 of each half)
                            const uint32_t w[2] = {raw[k][i].x, raw[k][i].y};
#pragma unroll
                            for (int h = 0; h < 2; ++h) {
                                const f32x2_t lo = __builtin_amdgcn_cvt_pk_f32_fp8(w[h], false);
                                const f32x2_t hi = __builtin_amdgcn_cvt_pk_f32_fp8(w[h], true);
                                v[4 * h] = lo[0]; v[4 * h + 1] = lo[1];
                                v[4 * h + 2] = hi[0]; v[4 * h + 3] = hi[1];
                            }
                        } else {
                            Vec16<T>::decode(raw[k][i], v);
                        }
                        if constexpr (ROPE) {
#pragma unroll
                            for (int e = 0; e < HV; ++e) {  // pair j0 + e: v[e] and v[HV + e]
                                // with the correction: the token's whole turn by
                                // (p0 + t) f_j; without it only the turn by t f_j,
                                // the block's common turn by p0 f_j being applied
                                // to the sum afterwards (rotations compose)
                                float c = rt[e].x, sn = rt[e].y;
                                if constexpr (decltype(mode)::value == 2) {
                                    rope_cos_sin(p0[k] + t, fr.f[j0 + e], &c, &sn);
                                } else if constexpr (decltype(mode)::value == 1) {
                                    const float ct = c;
                                    c = c0[k][e] * ct - s0v[k][e] * sn;
                                    sn = s0v[k][e] * ct + c0[k][e] * sn;
                                    const float eps = rope_eps(p0[k], t, fr.f[j0 + e]);
                                    const float cc = c;
                                    c = cc - sn * eps;
                                    sn = sn + cc * eps;
                                }
                                // turn by -angle: x_j c + x_{j+h} s, -x_j s + x_{j+h} c
                                const float lo = v[e], hi = v[HV + e];
                                v[e] = lo * c + hi * sn;
                                v[HV + e] = hi * c - lo * sn;
                            }
                        }
#pragma unroll
                        for (int e = 0; e < VEC; ++e) acc[k][e] += (Acc)v[e];
                    }
                }
            }
        };
        bool any_far = false, any_vfar = false;
        if constexpr (ROPE) {
#pragma unroll
            for (int k = 0; k < BPS; ++k) {
                any_far |= far[k];
                any_vfar |= vfar[k];
            }
        }
        using Plain = std::integral_constant<int, 0>;
        if constexpr (EPS) {
            if (any_vfar)  // wave-uniform
                sum_tokens(std::integral_constant<int, 2>{});
            else if (any_far)
                sum_tokens(std::integral_constant<int, 1>{});
            else
                sum_tokens(Plain{});
        } else {
            sum_tokens(Plain{});
        }
        const bool turn_sum = !(EPS && any_far);  // RoPE: the sums still owe the turn by p0 f_j
#pragma unroll
        for (int k = 0; k < BPS; ++k) {
#pragma unroll
            for (int e = 0; e < VEC; ++e) acc[k][e] = sum_lanes_mod<LPR>(acc[k][e]);
#pragma unroll
            for (int e = 0; e < VEC; ++e) mean[e] = (double)acc[k][e] * ks * inv;
            if constexpr (ROPE) {
                if (turn_sum) {
#pragma unroll
                    for (int e = 0; e < HV; ++e) {
                        const double lo = mean[e], hi = mean[HV + e], c = c0[k][e], sn = s0v[k][e];
                        mean[e] = lo * c + hi * sn;
                        mean[HV + e] = hi * c - lo * sn;
                    }
                }
            }
            if (tg == 0) {
                float *dst = tile_buf + (s0 + k * kWaves) * PAD;
                if constexpr (ROPE) {  // dims j0 + e and D/2 + j0 + e
#pragma unroll
                    for (int e = 0; e < VEC; ++e)
                        dst[e < HV ? j0 + e : D / 2 + j0 + e - HV] = ok[k] ? (float)mean[e] : __builtin_nanf("");
                } else {
#pragma unroll
                    for (int e = 0; e < VEC; e += 4)
                        *reinterpret_cast<float4 *>(dst + lp * VEC + e) = ok[k]
                            ? make_float4((float)mean[e], (float)mean[e + 1], (float)mean[e + 2], (float)mean[e + 3])
                            : make_float4(__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""),
                                          __builtin_nanf(""));
                }
            }
        }
    }
    __syncthreads();
    // write the part into its tile: for each 4-float column j4, kPart
    // consecutive blocks (512-byte runs)
    float *out = index + ((tile * n_kv_heads + g) * (D / 4)) * (kIndexTile * 4) +
                 (part % (kIndexTile / kPart)) * kPart * 4;
    for (int i = threadIdx.x; i < (D / 4) * kPart; i += kWaves * kWave) {
        const int j4 = i / kPart, slot = i % kPart;
        const int64_t b = b_tile0 + slot;
        if (b < b_lo || b >= b_hi) continue;
        const float4 v = *reinterpret_cast<const float4 *>(tile_buf + slot * PAD + j4 * 4);
        *reinterpret_cast<float4 *>(out + ((int64_t)j4 * kIndexTile + slot) * 4) = v;
    }
}

template <typename T, int D>
hipError_t launch_t(int n_kv_heads, int block_tokens, float k_scale, const void *k_pool, int64_t n_pages,
                    const int32_t *block_to_page, int32_t first_block, int32_t n_blocks,
                    float *index, hipStream_t stream, bool rope, const int64_t *block_pos,
                    const RopeFreqs *fr) {
    const int part = rope ? part_blocks<true>() : part_blocks<false>();
    const int64_t t0 = first_block / part;
    const int64_t t1 = ((int64_t)first_block + n_blocks + part - 1) / part;
    dim3 grid((unsigned)(t1 - t0), (unsigned)n_kv_heads);
    RopeFreqs f{};
    if (rope) {
        f = *fr;
        const size_t lds = sizeof(float2) * (size_t)block_tokens * (D / 2 + 1);
        // default positions b * block_tokens all below 2^26: the rounding
        // correction is never taken, so leave it out of the kernel
        const bool near = block_pos == nullptr && ((int64_t)first_block + n_blocks) * block_tokens <= kEpsMinPos;
        if (near)
            hipLaunchKernelGGL((build_index_kernel<T, D, true, false>), grid, dim3(kWaves * kWave), lds, stream,
                               static_cast<const T *>(k_pool), n_pages, block_to_page, first_block, n_blocks,
                               n_kv_heads, block_tokens, k_scale, index, block_pos, f);
        else
            hipLaunchKernelGGL((build_index_kernel<T, D, true, true>), grid, dim3(kWaves * kWave), lds, stream,
                               static_cast<const T *>(k_pool), n_pages, block_to_page, first_block, n_blocks,
                               n_kv_heads, block_tokens, k_scale, index, block_pos, f);
    } else {
        hipLaunchKernelGGL((build_index_kernel<T, D, false, false>), grid, dim3(kWaves * kWave), 0, stream,
                           static_cast<const T *>(k_pool), n_pages, block_to_page, first_block, n_blocks,
                           n_kv_heads, block_tokens, k_scale, index, block_pos, f);
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_build_index(int kv_dtype, int head_dim, int n_kv_heads, int block_tokens, float k_scale,
                              const void *k_pool, int64_t n_pages, const int32_t *block_to_page,
                              int32_t first_block, int32_t n_blocks, float *index,
                              hipStream_t stream, bool rope, const int64_t *block_pos, const RopeFreqs *fr) {
    if (n_blocks == 0) return hipSuccess;
    auto go = [&](auto elem, auto dim) {
        using T = decltype(elem);
        return launch_t<T, decltype(dim)::value>(n_kv_heads, block_tokens, k_scale, k_pool, n_pages,
                                                 block_to_page, first_block, n_blocks, index, stream, rope,
                                                 block_pos, fr);
    };
    using D64 = std::integral_constant<int, 64>;
    using D128 = std::integral_constant<int, 128>;
    if (kv_dtype == 2) return head_dim == 128 ? go(uint8_t{}, D128{}) : go(uint8_t{}, D64{});
    if (kv_dtype == 1) return head_dim == 128 ? go(uint16_t{}, D128{}) : go(uint16_t{}, D64{});
    return head_dim == 128 ? go(float{}, D128{}) : go(float{}, D64{});
}

}  // namespace kvmem
