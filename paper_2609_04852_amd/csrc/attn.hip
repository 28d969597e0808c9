// Decode attention over the execution view through its page table (Sec. 4.4,
// Sec. 5.3): split-K flash-decode plus an exact log-sum-exp merge.
//
// Kernels, by shape (launch_bt picks one; every one writes the same partials):
//   attn_mfma16        bf16 K/V with 3 to 47 query rows per KV head, and FP8
//                      below 48 rows: both products on the matrix cores
//   attn_mfma_rows     48 or more rows (bf16, FP8): groups of 16-row waves
//                      share each K/V tile through LDS
//   attn_splitk_row16  fp32 K/V at d = 64 with a multiple of 4 rows (a token
//                      row is one 16-lane DPP row), vector units
//   attn_splitk        every other shape, vector units
//   attn_combine       the exact merge of a (KV head, row)'s split partials
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

// Stages the n_pp (>= 1) page ids of a split into LDS: every thread's loads
// are issued together (clamped indexes, no branch), so the prologue takes one
// memory round trip instead of one per id a thread holds.  An id outside
// [0, n_pages) is stored as page 0 (never read: the caller's partial becomes
// NaN); returns whether this thread saw one.
template <int NT>
__device__ inline bool stage_page_ids(const int32_t *__restrict__ vpages, int p_begin, int n_pp, int64_t n_pages,
                                      int32_t *sm_pg) {
    constexpr int PER = (kAttnMaxPages + NT - 1) / NT;
    int32_t v[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) v[u] = vpages[p_begin + min((int)threadIdx.x + NT * u, n_pp - 1)];
    bool bad = false;
#pragma unroll
    for (int u = 0; u < PER; ++u) {
        const int i = threadIdx.x + NT * u;
        if (i < n_pp) {
            const bool ok = v[u] >= 0 && (int64_t)v[u] < n_pages;
            sm_pg[i] = ok ? v[u] : 0;
            bad |= !ok;
        }
    }
    return bad;
}

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
        float *dst = part + (((int64_t)g * n_splits + split) * rows_total + row0 + r) * (D + kPartStride);
        dst[d] = any_bad ? __builtin_nanf("") : acc;
        if (d == 0) {
            dst[D] = mx;
            dst[D + 1] = l;
        }
    }
}

// Fast path for 16-lane token rows (bf16 with d = 128, or f32 with d = 64) and
// RH >= 4 query rows per KV head.  Work goes in units of 16 tokens of a page:
// lane group lg (a 16-lane DPP row) takes tokens 4i + lg, i < 4.  The 4*RH
// partial logits of a lane are summed over its row with row_transpose_reduce16,
// after which lane lp owns query row r = lp % RH for RH/4 token slots; it alone
// exponentiates those scores, keeps the running max and sum of its row, and
// the probabilities reach the other 15 lanes through row_newbcast.  Rescaling
// of the accumulators is skipped unless some running max grew.  The next
// unit's K and V are loaded (non-temporal) while the current one is processed.
template <typename T, int D, int BT, int RH>
__global__ __launch_bounds__(kAttnThreads) void attn_splitk_row16_kernel(
    const float *__restrict__ q, const T *__restrict__ k_pool, const T *__restrict__ v_pool,
    int64_t n_pages, const int32_t *__restrict__ view_pages, int n_sel, int n_view,
    int last_page_tokens, int n_kv_heads, int n_q_heads, int group, int rows_total,
    int pages_per_split, int n_splits, float qscale, float *__restrict__ part) {
    constexpr int VEC = Vec16<T>::N;
    static_assert(D / VEC == 16, "one token row per 16-lane DPP row");
    static_assert(RH >= 4 && RH <= 16 && BT % 16 == 0, "shape of the fast path");
    constexpr int NV = 4 * RH;         // partial logits per lane per unit
    constexpr int NC = NV / 16;        // finished logits per lane per unit
    constexpr int UNITS = BT / 16;     // 16-token units per page
    __shared__ float sm_o[kAttnWaves][RH][D];
    __shared__ float sm_m[kAttnWaves][RH], sm_l[kAttnWaves][RH];
    __shared__ int sm_bad;
    __shared__ int32_t sm_pg[kAttnMaxPages];

    const int split = blockIdx.x, g = blockIdx.y, row0 = blockIdx.z * RH;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int lg = lane / 16, lp = lane % 16;
    const int my_r = lp % RH;
    const int32_t *vpages = view_pages + (int64_t)(n_sel == 1 ? 0 : g) * n_view;
    const int p_begin = split * pages_per_split;
    const int p_end = min(n_view, p_begin + pages_per_split);
    // the split's page ids, staged once (invalid ones are never read: they
    // become page 0 and make this split's partial NaN)
    if (threadIdx.x == 0) sm_bad = 0;
    __syncthreads();
    if (stage_page_ids<kAttnThreads>(vpages, p_begin, p_end - p_begin, n_pages, sm_pg)) sm_bad = 1;
    __syncthreads();

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
    float o[RH][VEC];
#pragma unroll
    for (int r = 0; r < RH; ++r)
#pragma unroll
        for (int e = 0; e < VEC; ++e) o[r][e] = 0.f;
    float m_own = -INFINITY, l_own = 0.f;

    // unit u of this wave: page p_begin + wave + 4*(u / UNITS), tokens 16*(u % UNITS) ...
    const int n_my_pages = p_end - p_begin - wave > 0 ? (p_end - p_begin - wave + kAttnWaves - 1) / kAttnWaves : 0;
    const int n_units = n_my_pages * UNITS;
    // Loads are unconditional (all in flight together): a token past the
    // page's valid ones reads token 0 of the page and is zeroed afterwards, so
    // whatever the pool holds there never reaches the sums.
    auto fetch = [&](int u, uint4 (&kr)[4], uint4 (&vr)[4], int &ntok_out) {
        const int pi = p_begin + wave + kAttnWaves * (u / UNITS);
        const int t0 = 16 * (u % UNITS);
        const int64_t page = sm_pg[pi - p_begin];
        const int ntok = (pi == n_view - 1 ? last_page_tokens : BT) - t0;
        ntok_out = ntok;
        const int64_t off = (page * n_kv_heads + g) * (int64_t)BT * D + (int64_t)t0 * D + lp * VEC;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int t = 4 * i + lg;
            const int64_t to = (int64_t)(t < ntok ? t : -t0) * D;
            kr[i] = load_stream16(k_pool + off + to);
            vr[i] = load_stream16(v_pool + off + to);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            if (4 * i + lg >= ntok) {
                kr[i] = make_uint4(0u, 0u, 0u, 0u);
                vr[i] = make_uint4(0u, 0u, 0u, 0u);
            }
        }
    };
    auto widen = [](const uint4 &w, float (&out)[VEC]) {
        if constexpr (VEC == 8) {
            const uint32_t x[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                out[2 * i] = __uint_as_float(x[i] << 16);
                out[2 * i + 1] = __uint_as_float(x[i] & 0xffff0000u);
            }
        } else {
            out[0] = __uint_as_float(w.x); out[1] = __uint_as_float(w.y);
            out[2] = __uint_as_float(w.z); out[3] = __uint_as_float(w.w);
        }
    };
    auto process = [&](const uint4 (&kr)[4], const uint4 (&vr)[4], int ntok) {
        // partial logits: value v = i*RH + r
        float part[NV];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float kx[VEC];
            widen(kr[i], kx);
#pragma unroll
            for (int r = 0; r < RH; ++r) {
                float acc = 0.f;
#pragma unroll
                for (int e = 0; e < VEC; ++e) acc += qr[r][e] * kx[e];
                part[i * RH + r] = acc;
            }
        }
        // finished logits: slot c holds value c*16 + lp, i.e. token slot
        // (c*16 + lp) / RH of row my_r
        float sc[NC];
        float pm = -INFINITY;
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            float chunk[16];
#pragma unroll
            for (int k = 0; k < 16; ++k) chunk[k] = part[c * 16 + k];
            const float sv = row_transpose_reduce16(chunk, lp);
            const int t = 4 * ((c * 16 + lp) / RH) + lg;
            sc[c] = t < ntok ? sv : -INFINITY;
            pm = fmaxf(pm, sc[c]);
        }
        // row maximum over the lanes that share my_r
        if constexpr (RH < 16) pm = fmaxf(pm, dpp_f<dpp_row_ror(RH)>(pm));
        if constexpr (RH < 8) pm = fmaxf(pm, dpp_f<dpp_row_ror(2 * RH)>(pm));
        if constexpr (RH < 4) pm = fmaxf(pm, dpp_f<dpp_row_ror(4 * RH)>(pm));
        const float mn = fmaxf(m_own, pm);
        const float msafe = mn == -INFINITY ? 0.f : mn;
        if (__any(mn > m_own)) {
            const float alpha = exp2f(m_own - msafe);  // 0 while m_own is -inf
            l_own *= alpha;
            float al[RH];
            static_for<RH>([&](auto r) { al[r] = dpp_f<dpp_row_bcast(r)>(alpha); });
#pragma unroll
            for (int r = 0; r < RH; ++r)
#pragma unroll
                for (int e = 0; e < VEC; ++e) o[r][e] *= al[r];
        }
        m_own = mn;
        float pc[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            pc[c] = exp2f(sc[c] - msafe);
            l_own += pc[c];
        }
        // p for every (token slot i, row r): value i*RH + r lives in lane
        // (i*RH + r) % 16, slot (i*RH + r) / 16
        static_for<4>([&](auto i) {
            float vx[VEC];
            widen(vr[i], vx);
            static_for<RH>([&](auto r) {
                constexpr int v = i * RH + r;
                const float p = dpp_f<dpp_row_bcast(v % 16)>(pc[v / 16]);
#pragma unroll
                for (int e = 0; e < VEC; ++e) o[r][e] += p * vx[e];
            });
        });
    };

    // two statically named buffers: unit u+1 loads while unit u is processed
    uint4 ka[4], va[4], kb[4], vb[4];
    int na = 0, nb = 0;
    if (n_units > 0) fetch(0, ka, va, na);
    for (int u = 0; u < n_units; u += 2) {
        if (u + 1 < n_units) fetch(u + 1, kb, vb, nb);
        process(ka, va, na);
        if (u + 1 >= n_units) break;
        if (u + 2 < n_units) fetch(u + 2, ka, va, na);
        process(kb, vb, nb);
    }

    // per lane group: row sums over the lanes sharing a row, then broadcast
    float lsum = l_own;
    if constexpr (RH < 16) lsum += dpp_f<dpp_row_ror(RH)>(lsum);
    if constexpr (RH < 8) lsum += dpp_f<dpp_row_ror(2 * RH)>(lsum);
    float mrow[RH], lrow[RH];
    static_for<RH>([&](auto r) {
        mrow[r] = dpp_f<dpp_row_bcast(r)>(m_own);
        lrow[r] = dpp_f<dpp_row_bcast(r)>(lsum);
    });
    // merge the 4 lane groups of the wave (lanes lp, lp+16, lp+32, lp+48)
#pragma unroll
    for (int r = 0; r < RH; ++r) {
        float mx = mrow[r];
        mx = fmaxf(mx, shfl_xor_f(mx, 16));
        mx = fmaxf(mx, shfl_xor_f(mx, 32));
        const float f = mrow[r] == -INFINITY ? 0.f : exp2f(mrow[r] - mx);
        float l = lrow[r] * f;
        l += shfl_xor_f(l, 16);
        l += shfl_xor_f(l, 32);
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
            float x = o[r][e] * f;
            x += shfl_xor_f(x, 16);
            x += shfl_xor_f(x, 32);
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
    __syncthreads();
    const bool any_bad = sm_bad != 0;
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
        float *dst = part + (((int64_t)g * n_splits + split) * rows_total + row0 + r) * (D + kPartStride);
        dst[d] = any_bad ? __builtin_nanf("") : acc;
        if (d == 0) {
            dst[D] = mx;
            dst[D + 1] = l;
        }
    }
}

// MFMA path for bf16 K/V with 3 or more query rows per KV head (e.g. 4 GQA
// heads x 4 query tokens), in tiles of 16 rows (a partial last tile is padded
// with zero queries that are never written).  At 16 rows the step does 16
// flops per K/V byte, more than the vector units sustain at full HBM rate, so
// both products run on the matrix cores (v_mfma_f32_16x16x32_bf16); with
// fewer rows the matrix cores still leave the vector units freer than the
// vector kernel does.  Lane l of a wave works on query row l % 16;
// kg = l / 16 picks its 8-element slice of each 32-long contraction.
//   scores  S^T = K Q^T per 16 tokens: K (A operand, lane: token l%16, 8
//           dims) is read from a per-wave LDS copy of the tile, which is loaded
//           like V with whole rows per load instruction (the operand layout
//           itself would touch 16 rows and half a cache line of each per
//           instruction); Q^T is the B operand kept in registers.  Q is split as hi + lo bf16 (q = hi + lo to 2^-16),
//           so the logits keep fp32 accuracy at twice the (cheap) MFMA count.
//           Lane l receives S[row l%16][tokens 4kg .. 4kg+3] of the 16.
//   softmax online per row in base 2; each lane holds 8 scores of its row per
//           32-token tile, the row max is completed over the 4 kg lanes.
//   output  O^T = V^T P^T per 32 tokens and 16 dims: P^T (B operand) is the
//           lane's own 8 probabilities, split hi + lo; V^T (A operand) comes
//           from a per-wave LDS copy of the tile through two transposing reads
//           (ds_read_b64_tr_b16) per 16 dims.  The contraction order of tokens
//           is the same permutation on both sides.
// Waves take the split's 32-token tiles in turn and are merged in LDS; one
// partial (O, max, sum) per row is written in the format attn_combine reads.
// FP8 K/V (E4M3 codes): every code is exactly a bf16 value, so the same MFMA
// products run on codes widened in registers (v_cvt_scalef32_pk_bf16_fp8, two
// codes per instruction); k_scale is folded into Q and v_scale into the
// partial output.  One 16-byte K load then holds 16 dims, which feed two
// 32-long contractions: chunk 2c+u takes dims 64c + 16kg + 8u + [0, 8), and Q
// is laid out the same way.  K codes stay codes in LDS and are widened after
// the operand read; V codes are widened before they go to LDS.
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
constexpr int kMfmaRows = 16;
constexpr int kMfmaTile = 32;  // tokens per tile

// hi + lo bf16 split of 8 floats: hi = bf16(x), lo = bf16(x - hi), both rounded
// to nearest even by the conversion instruction (v_cvt_pk_bf16_f32)
__device__ inline void split_bf16x8(const float (&x)[8], bf16x8_t &hi, bf16x8_t &lo) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        const __bf16 h = (__bf16)x[j];
        hi[j] = h;
        lo[j] = (__bf16)(x[j] - (float)h);
    }
}

// The LDS transposing read: within each group of 16 lanes, lane i receives
// element i % 4 of the 4-element (8-byte) chunks addressed by lanes i/4 + 4j,
// j = 0..3.
typedef short i16x4_t __attribute__((ext_vector_type(4)));
__device__ inline uint2 lds_read_tr16(const uint16_t *p) {
    const i16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4_t *)(p));
    return __builtin_bit_cast(uint2, v);
}

__device__ inline bf16x8_t as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8_t, v); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
// 4 E4M3 codes -> 4 bf16 (exact), as two dwords of bf16 pairs in code order
__device__ inline uint2 fp8x4_to_bf16x4(uint32_t w) {
    return make_uint2(__builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, false)),
                      __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, true)));
}
// 8 codes (two dwords) -> one bf16x8 operand
__device__ inline bf16x8_t fp8x8_to_bf16x8(uint32_t w0, uint32_t w1) {
    const uint2 a = fp8x4_to_bf16x4(w0), b = fp8x4_to_bf16x4(w1);
    return as_bf16x8(make_uint4(a.x, a.y, b.x, b.y));
}

// T = uint16_t (bf16 bits) or uint8_t (FP8 E4M3 codes)
template <typename T, int D, int BT>
__global__ __launch_bounds__(kAttnThreads, 2) void attn_mfma16_kernel(
    const float *__restrict__ q, const T *__restrict__ k_pool, const T *__restrict__ v_pool,
    int64_t n_pages, const int32_t *__restrict__ view_pages, int n_sel, int n_view, int last_page_tokens,
    int n_kv_heads, int n_q_heads, int group, int rows_total, int pages_per_split, int n_splits,
    float qscale, float v_scale, float *__restrict__ part) {
    constexpr bool F8 = sizeof(T) == 1;
    constexpr int EPL = 16 / sizeof(T);  // elements per 16-byte load
    constexpr int KC = D / 32;           // 32-long chunks of the head dimension (scores)
    constexpr int KL = F8 ? KC / 2 : KC; // 16-byte K operand reads per lane per 16-token half
    constexpr int MB = D / 16;           // 16-dim blocks of the output
    constexpr int VP = D + 16;           // LDS row pitch of the V tile, in halves (rows 8 banks apart)
    constexpr int VL = kMfmaTile * D / EPL / kWave;  // 16-byte loads per lane per tile, of K and of V
    static_assert(VL * kWave * EPL == kMfmaTile * D, "K and V tiles split over the wave");
    // K is loaded the way V is (each load instruction covers whole rows, 1 KB
    // contiguous) and read back in the A-operand layout from a per-wave LDS
    // tile of raw elements (FP8 codes are widened after that read)
    constexpr int KPB = D * (int)sizeof(T) + 16;  // LDS row pitch of the K tile, in bytes
    static_assert(2 * KL == VL, "K and V tiles take the same loads");
    // first dim of the lane's 8-long slice of contraction chunk c (Q and K alike)
    auto chunk_dim = [&](int c, int kg) { return F8 ? 64 * (c / 2) + 16 * kg + 8 * (c % 2) : 32 * c + 8 * kg; };
    __shared__ uint16_t sm_v[kAttnWaves][kMfmaTile * VP];
    __shared__ __attribute__((aligned(16))) uint8_t sm_k[kAttnWaves][kMfmaTile * KPB];
    __shared__ float sm_m[kAttnWaves][kMfmaRows], sm_l[kAttnWaves][kMfmaRows];
    __shared__ int sm_bad[kAttnWaves];

    __shared__ int32_t sm_pg[kAttnMaxPages];
    const int split = blockIdx.x, g = blockIdx.y, row0 = blockIdx.z * kMfmaRows;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int r16 = lane % 16, kg = lane / 16;
    const int32_t *vpages = view_pages + (int64_t)(n_sel == 1 ? 0 : g) * n_view;
    const int p_begin = split * pages_per_split;
    const int p_end = min(n_view, p_begin + pages_per_split);
    // tokens of the split, page-major; the view's last page may be partial
    const int n_tok = (p_end - p_begin) * BT - (p_end == n_view ? BT - last_page_tokens : 0);
    const int n_tiles = (n_tok + kMfmaTile - 1) / kMfmaTile;
    // the split's page ids, staged once (invalid ones are never read: they
    // become page 0 and make this split's partial NaN)
    if (threadIdx.x < kAttnWaves) sm_bad[threadIdx.x] = 0;
    __syncthreads();
    if (stage_page_ids<kAttnThreads>(vpages, p_begin, p_end - p_begin, n_pages, sm_pg)) sm_bad[0] = 1;
    __syncthreads();
    const bool any_bad = sm_bad[0] != 0;

    // Q^T operand: lane holds q[row r16][chunk_dim(c, kg) + j] * qscale as hi + lo
    // (rows past rows_total pad the 16-row tile with zeros and are not written)
    bf16x8_t qhi[KC], qlo[KC];
    {
        const int row = min(row0 + r16, rows_total - 1), m = row / group, hh = row % group;
        const float qs = row0 + r16 < rows_total ? qscale : 0.f;
        const float *qp = q + ((int64_t)m * n_q_heads + g * group + hh) * D;
#pragma unroll
        for (int c = 0; c < KC; ++c) {
            const float4 a = *reinterpret_cast<const float4 *>(qp + chunk_dim(c, kg));
            const float4 b = *reinterpret_cast<const float4 *>(qp + chunk_dim(c, kg) + 4);
            const float x[8] = {a.x * qs, a.y * qs, a.z * qs, a.w * qs, b.x * qs, b.y * qs, b.z * qs, b.w * qs};
            split_bf16x8(x, qhi[c], qlo[c]);
        }
    }
    f32x4_t acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float mrun = -INFINITY, lpart = 0.f;

    // K and V of tile t (16 tokens of a half never cross a page): load i ->
    // token (lane + 64 i) / (D/EPL), 16 bytes at dim EPL * ((lane + 64 i) %
    // (D/EPL)), for K and V alike.  Tokens past the split read the split's
    // last token again (in bounds) and are masked out of the softmax.
    // A full tile takes the fast path: each half's page base is wave-uniform
    // (scalar registers) and load i adds lane * EPL plus a constant (it covers
    // 64 / (D/EPL) whole tokens, all in one half).  Only the split's last tile
    // clamps per lane.
    const uint32_t v_lane = (uint32_t)(lane * EPL);
    constexpr int TPI = kWave / (D / EPL);  // tokens per load instruction
    static_assert(16 % TPI == 0, "a load instruction stays inside one half");
    auto half_base = [&](int s0) -> int64_t {  // s0: first token of a half, wave-uniform, < n_tok
        const int64_t pg = __builtin_amdgcn_readfirstlane(sm_pg[s0 / BT]);
        return (pg * n_kv_heads + g) * (int64_t)BT * D + (int64_t)(s0 % BT) * D;
    };
    auto load_tile = [&](int t, uint4 (&kb)[VL], uint4 (&vb)[VL]) {
        if (t * kMfmaTile + kMfmaTile <= n_tok) {
            int64_t base[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) base[h] = half_base(t * kMfmaTile + 16 * h);
#pragma unroll
            for (int i = 0; i < VL; ++i) {
                const int h = i * TPI / 16;
                kb[i] = load_stream16(k_pool + base[h] + v_lane + (i * TPI - 16 * h) * D);
                vb[i] = load_stream16(v_pool + base[h] + v_lane + (i * TPI - 16 * h) * D);
            }
            return;
        }
        const T *kbase[2], *vbase[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int s0 = min(t * kMfmaTile + 16 * h, n_tok - 1);
            const int64_t off = ((int64_t)sm_pg[s0 / BT] * n_kv_heads + g) * (int64_t)BT * D +
                                (int64_t)(s0 % BT) * D;
            kbase[h] = k_pool + off;
            vbase[h] = v_pool + off;
        }
#pragma unroll
        for (int i = 0; i < VL; ++i) {
            const int idx = lane + kWave * i, x = idx / (D / EPL), ch = idx % (D / EPL);
            const int h = x / 16;
            const int64_t off = (int64_t)(min(x, n_tok - 1 - t * kMfmaTile) - 16 * h) * D + EPL * ch;
            kb[i] = load_stream16(kbase[h] + off);
            vb[i] = load_stream16(vbase[h] + off);
        }
    };
    uint16_t *my_v = sm_v[wave];
    uint8_t *my_k = sm_k[wave];
    // K tile to LDS as loaded: row x at pitch KPB, 16 bytes at 16*ch (the 16
    // rows of an operand read then start 4 banks apart at d = 128 bf16 and
    // at 16 distinct 4-bank offsets for FP8)
    auto stage_k = [&](const uint4 (&kb)[VL]) {
#pragma unroll
        for (int i = 0; i < VL; ++i) {
            const int idx = lane + kWave * i, x = idx / (D / EPL), ch = idx % (D / EPL);
            *reinterpret_cast<uint4 *>(my_k + x * KPB + 16 * ch) = kb[i];
        }
    };
    // V tile to LDS as bf16 (row x, EPL values at EPL*ch); a wave reads only its own tile
    auto stage_v = [&](const uint4 (&vb)[VL]) {
#pragma unroll
        for (int i = 0; i < VL; ++i) {
            const int idx = lane + kWave * i, x = idx / (D / EPL), ch = idx % (D / EPL);
            uint2 *dst = reinterpret_cast<uint2 *>(my_v + x * VP + EPL * ch);
            if constexpr (F8) {
                dst[0] = fp8x4_to_bf16x4(vb[i].x);
                dst[1] = fp8x4_to_bf16x4(vb[i].y);
                dst[2] = fp8x4_to_bf16x4(vb[i].z);
                dst[3] = fp8x4_to_bf16x4(vb[i].w);
            } else {
                dst[0] = make_uint2(vb[i].x, vb[i].y);
                dst[1] = make_uint2(vb[i].z, vb[i].w);
            }
        }
    };
    auto process = [&](int t) {
        // scores of the 32 tokens: lane gets row r16, tokens 16h + 4kg + i
        float sc[8];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            f32x4_t st = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < KC; ++c) {
                // the lane's 16 bytes of K row 16h + r16 (FP8: two chunks' codes)
                const uint4 w = *reinterpret_cast<const uint4 *>(
                    my_k + (16 * h + r16) * KPB + (int)sizeof(T) * chunk_dim(F8 ? c & ~1 : c, kg));
                bf16x8_t kk;
                if constexpr (F8) kk = c % 2 == 0 ? fp8x8_to_bf16x8(w.x, w.y) : fp8x8_to_bf16x8(w.z, w.w);
                else kk = as_bf16x8(w);
                st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, qhi[c], st, 0, 0, 0);
                st = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, qlo[c], st, 0, 0, 0);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) sc[4 * h + i] = st[i];
        }
        if (t * kMfmaTile + kMfmaTile > n_tok) {  // the split's last tile: mask tokens past its end
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (t * kMfmaTile + 16 * (j / 4) + 4 * kg + j % 4 >= n_tok) sc[j] = -INFINITY;
        }
        // online softmax of row r16 (replicated over the 4 kg lanes)
        float cm = sc[0];
#pragma unroll
        for (int j = 1; j < 8; ++j) cm = fmaxf(cm, sc[j]);
        cm = fmaxf(cm, shfl_xor_f(cm, 16));
        cm = fmaxf(cm, shfl_xor_f(cm, 32));
        const float mn = fmaxf(mrun, cm);
        const float msafe = mn == -INFINITY ? 0.f : mn;
        if (__any(mn > mrun)) {
            const float alpha = exp2_hw(mrun - msafe);
            lpart *= alpha;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) acc[mb] *= alpha;
        }
        mrun = mn;
        float pr[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            pr[j] = exp2_hw(sc[j] - msafe);
            lpart += pr[j];
        }
        bf16x8_t phi, plo;
        split_bf16x8(pr, phi, plo);
        // output: A = V^T, lane (r16, kg) needs dims 16mb + r16 of tokens
        // 16(j/4) + 4kg + j%4.  Lane r16 of group kg addresses token
        // 4kg + r16/4 (+16 for the second read), dims 16mb + 4(r16 % 4) .. +3;
        // the transposing read then hands each lane its dim of the 4 tokens.
        const uint16_t *vrow = my_v + (4 * kg + r16 / 4) * VP + 4 * (r16 % 4);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const uint2 a = lds_read_tr16(vrow + 16 * mb);
            const uint2 b = lds_read_tr16(vrow + 16 * VP + 16 * mb);
            const bf16x8_t va = as_bf16x8(make_uint4(a.x, a.y, b.x, b.y));
            acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, phi, acc[mb], 0, 0, 0);
            acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, plo, acc[mb], 0, 0, 0);
        }
    };
    // wave w takes tiles w, w + 4, ...: the tile's K and V go to LDS, the
    // next tile's loads are issued into the same registers, then the tile is
    // processed from LDS while they are in flight
    {
        uint4 kx[VL], vx[VL];
        int t = wave;
        if (t < n_tiles) load_tile(t, kx, vx);
        while (t < n_tiles) {
            stage_k(kx);
            stage_v(vx);
            const int t1 = t + kAttnWaves;
            if (t1 < n_tiles) load_tile(t1, kx, vx);
            process(t);
            t = t1;
        }
    }
    // row sums over the 4 kg lanes
    float lrun = lpart + shfl_xor_f(lpart, 16);
    lrun += shfl_xor_f(lrun, 32);
    // merge the waves: O^T in LDS as [wave][row][D] floats (reuses the V tiles)
    __syncthreads();
    float *sm_o = reinterpret_cast<float *>(&sm_v[0][0]);
    static_assert(sizeof(float) * kAttnWaves * kMfmaRows * D <= sizeof(uint16_t) * kAttnWaves * kMfmaTile * VP,
                  "merge buffer fits the V tiles");
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) sm_o[(wave * kMfmaRows + r16) * D + 16 * mb + 4 * kg + i] = acc[mb][i];
    if (kg == 0) {
        sm_m[wave][r16] = mrun;
        sm_l[wave][r16] = lrun;
    }
    __syncthreads();
    const int rows_here = min(kMfmaRows, rows_total - row0);
    for (int idx = threadIdx.x; idx < rows_here * D; idx += kAttnThreads) {
        const int r = idx / D, d = idx % D;
        float mx = sm_m[0][r];
#pragma unroll
        for (int w = 1; w < kAttnWaves; ++w) mx = fmaxf(mx, sm_m[w][r]);
        float o = 0.f, l = 0.f;
#pragma unroll
        for (int w = 0; w < kAttnWaves; ++w) {
            const float f = sm_m[w][r] == -INFINITY ? 0.f : exp2f(sm_m[w][r] - mx);
            o += sm_o[(w * kMfmaRows + r) * D + d] * f;
            l += sm_l[w][r] * f;
        }
        float *dst = part + (((int64_t)g * n_splits + split) * rows_total + row0 + r) * (D + kPartStride);
        dst[d] = any_bad ? __builtin_nanf("") : o * v_scale;
        if (d == 0) {
            dst[D] = mx;
            dst[D + 1] = l;
        }
    }
}

// Many query rows per KV head (a step's prefill replayed over the view: e.g.
// 128 tokens x 4 GQA heads = 512 rows).  The workgroup's NW waves each own 16
// rows and share every 32-token K/V tile: the whole workgroup loads it once
// into one of two LDS stages (K and V as bf16; FP8 codes widened on the way
// in), so K/V is read from memory once per 16 NW rows instead of once per 16
// (at 512 rows: 466 us with 4 waves, 300 with 8, 288 with 16 over a 64K view).
// Per tile each wave runs the products of attn_mfma16 with its K operand read
// from LDS (row pitch D + 8 halves: the 16 rows of one read sit 4 banks apart)
// and V^T by the transposing reads; each wave keeps its rows' running softmax
// and writes their partials itself (no merge across waves).
// NW waves (16 rows each) share one K/V tile: 4, 8 or 16 by the row count
template <typename T, int D, int BT, int NW>
__global__ __launch_bounds__(NW * kWave) void attn_mfma_rows_kernel(
    const float *__restrict__ q, const T *__restrict__ k_pool, const T *__restrict__ v_pool,
    int64_t n_pages, const int32_t *__restrict__ view_pages, int n_sel, int n_view, int last_page_tokens,
    int n_kv_heads, int n_q_heads, int group, int rows_total, int pages_per_split, int n_splits,
    float qscale, float v_scale, float *__restrict__ part) {
    constexpr bool F8 = sizeof(T) == 1;
    constexpr int EPL = 16 / sizeof(T);               // elements per 16-byte load
    constexpr int KC = D / 32, MB = D / 16;
    constexpr int KP = D + 8, VP = D + 16;            // LDS row pitches, in halves
    constexpr int UPR = D / EPL;                      // 16-byte units per token row
    constexpr int LPT = kMfmaTile * UPR;              // units per tile, K or V
    constexpr int NT = NW * kWave;
    constexpr int LPL = (LPT + NT - 1) / NT;          // per thread
    __shared__ __attribute__((aligned(16))) uint16_t sm_k[2][kMfmaTile * KP];
    __shared__ __attribute__((aligned(16))) uint16_t sm_v[2][kMfmaTile * VP];
    __shared__ int32_t sm_pg[kAttnMaxPages];
    const int split = blockIdx.x, g = blockIdx.y;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const int r16 = lane % 16, kg = lane / 16;
    const int row0 = blockIdx.z * (NW * kMfmaRows) + wave * kMfmaRows;
    const int32_t *vpages = view_pages + (int64_t)(n_sel == 1 ? 0 : g) * n_view;
    const int p_begin = split * pages_per_split;
    const int p_end = min(n_view, p_begin + pages_per_split);
    const int n_tok = (p_end - p_begin) * BT - (p_end == n_view ? BT - last_page_tokens : 0);
    const int n_tiles = (n_tok + kMfmaTile - 1) / kMfmaTile;
    // an invalid id is never read; the split's partial becomes NaN
    const bool bad = stage_page_ids<NT>(vpages, p_begin, p_end - p_begin, n_pages, sm_pg);
    const bool any_bad = __syncthreads_or(bad) != 0;

    // Q^T operand of this wave's 16 rows, hi + lo bf16 (padding rows are zero)
    bf16x8_t qhi[KC], qlo[KC];
    {
        const int row = min(row0 + r16, rows_total - 1), m = row / group, hh = row % group;
        const float qs = row0 + r16 < rows_total ? qscale : 0.f;
        const float *qp = q + ((int64_t)m * n_q_heads + g * group + hh) * D + 8 * kg;
#pragma unroll
        for (int c = 0; c < KC; ++c) {
            const float4 a = *reinterpret_cast<const float4 *>(qp + 32 * c);
            const float4 b = *reinterpret_cast<const float4 *>(qp + 32 * c + 4);
            const float x[8] = {a.x * qs, a.y * qs, a.z * qs, a.w * qs, b.x * qs, b.y * qs, b.z * qs, b.w * qs};
            split_bf16x8(x, qhi[c], qlo[c]);
        }
    }
    f32x4_t acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float mrun = -INFINITY, lpart = 0.f;

    // unit u of tile t: token u / UPR, EPL elements at dim EPL * (u % UPR); tokens
    // past the split read its last token again and are masked out of the softmax
    auto load = [&](int t, uint4 (&kr)[LPL], uint4 (&vr)[LPL]) {
#pragma unroll
        for (int i = 0; i < LPL; ++i) {
            const int u = threadIdx.x + NT * i;
            if (LPT % NT == 0 || u < LPT) {
                const int tok = min(t * kMfmaTile + u / UPR, n_tok - 1);
                const int64_t off = ((int64_t)sm_pg[tok / BT] * n_kv_heads + g) * (int64_t)BT * D +
                                    (int64_t)(tok % BT) * D + EPL * (u % UPR);
                kr[i] = load_stream16(k_pool + off);
                vr[i] = load_stream16(v_pool + off);
            }
        }
    };
    auto put = [&](uint16_t *dst, const uint4 &x) {
        if constexpr (F8) {
            uint2 *d2 = reinterpret_cast<uint2 *>(dst);
            d2[0] = fp8x4_to_bf16x4(x.x);
            d2[1] = fp8x4_to_bf16x4(x.y);
            d2[2] = fp8x4_to_bf16x4(x.z);
            d2[3] = fp8x4_to_bf16x4(x.w);
        } else {
            *reinterpret_cast<uint4 *>(dst) = x;
        }
    };
    auto stage = [&](int st, const uint4 (&kr)[LPL], const uint4 (&vr)[LPL]) {
#pragma unroll
        for (int i = 0; i < LPL; ++i) {
            const int u = threadIdx.x + NT * i;
            if (LPT % NT == 0 || u < LPT) {
                const int x = u / UPR, col = EPL * (u % UPR);
                put(&sm_k[st][x * KP + col], kr[i]);
                put(&sm_v[st][x * VP + col], vr[i]);
            }
        }
    };
    auto process = [&](int t, int st) {
        const uint16_t *kt = sm_k[st];
        float sc[8];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            f32x4_t s4 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c = 0; c < KC; ++c) {
                const bf16x8_t kk =
                    as_bf16x8(*reinterpret_cast<const uint4 *>(kt + (16 * h + r16) * KP + 32 * c + 8 * kg));
                s4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, qhi[c], s4, 0, 0, 0);
                s4 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kk, qlo[c], s4, 0, 0, 0);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) sc[4 * h + i] = s4[i];
        }
        if (t * kMfmaTile + kMfmaTile > n_tok) {
#pragma unroll
            for (int j = 0; j < 8; ++j)
                if (t * kMfmaTile + 16 * (j / 4) + 4 * kg + j % 4 >= n_tok) sc[j] = -INFINITY;
        }
        float cm = sc[0];
#pragma unroll
        for (int j = 1; j < 8; ++j) cm = fmaxf(cm, sc[j]);
        cm = fmaxf(cm, shfl_xor_f(cm, 16));
        cm = fmaxf(cm, shfl_xor_f(cm, 32));
        const float mn = fmaxf(mrun, cm);
        const float msafe = mn == -INFINITY ? 0.f : mn;
        if (__any(mn > mrun)) {
            const float alpha = exp2_hw(mrun - msafe);
            lpart *= alpha;
#pragma unroll
            for (int mb = 0; mb < MB; ++mb) acc[mb] *= alpha;
        }
        mrun = mn;
        float pr[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            pr[j] = exp2_hw(sc[j] - msafe);
            lpart += pr[j];
        }
        bf16x8_t phi, plo;
        split_bf16x8(pr, phi, plo);
        const uint16_t *vrow = sm_v[st] + (4 * kg + r16 / 4) * VP + 4 * (r16 % 4);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const uint2 a = lds_read_tr16(vrow + 16 * mb);
            const uint2 b = lds_read_tr16(vrow + 16 * VP + 16 * mb);
            const bf16x8_t va = as_bf16x8(make_uint4(a.x, a.y, b.x, b.y));
            acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, phi, acc[mb], 0, 0, 0);
            acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, plo, acc[mb], 0, 0, 0);
        }
    };
    {
        uint4 kr[LPL], vr[LPL];
        if (n_tiles > 0) {
            load(0, kr, vr);
            stage(0, kr, vr);
        }
        __syncthreads();
        for (int t = 0; t < n_tiles; ++t) {
            const int st = t & 1;
            if (t + 1 < n_tiles) load(t + 1, kr, vr);
            process(t, st);
            // the other stage was last read in iteration t - 1, before the barrier
            if (t + 1 < n_tiles) stage(st ^ 1, kr, vr);
            __syncthreads();
        }
    }
    float lrun = lpart + shfl_xor_f(lpart, 16);
    lrun += shfl_xor_f(lrun, 32);
    if (row0 + r16 < rows_total) {
        float *dst = part + (((int64_t)g * n_splits + split) * rows_total + row0 + r16) * (D + kPartStride);
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
            const float4 o = any_bad ? make_float4(__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""),
                                                   __builtin_nanf(""))
                                     : make_float4(acc[mb][0] * v_scale, acc[mb][1] * v_scale, acc[mb][2] * v_scale,
                                                   acc[mb][3] * v_scale);
            *reinterpret_cast<float4 *>(dst + 16 * mb + 4 * kg) = o;
        }
        if (kg == 0) {
            dst[D] = mrun;
            dst[D + 1] = lrun;
        }
    }
}

constexpr int kCombineThreads = 256;

// One workgroup per (KV head, row).  The split weights 2^(m_s - M) are formed
// once into LDS; then D/4 lanes read one split's partial row as float4s and the
// workgroup walks kCombineThreads/(D/4) splits at a time, so every thread keeps
// many independent loads in flight.
template <int D>
__global__ __launch_bounds__(kCombineThreads) void attn_combine_kernel(
    const float *__restrict__ part, int n_splits, int rows_total, int n_q_heads, int group,
    float *__restrict__ out, float *__restrict__ lse) {
    constexpr int LPS = D / 4;                     // lanes per split row
    constexpr int SPI = kCombineThreads / LPS;     // splits per iteration
    extern __shared__ float sm_w[];                // [n_splits] weights
    __shared__ float sm_red[kCombineThreads / kWave];
    __shared__ float4 sm_acc[SPI][LPS];
    const int g = blockIdx.x / rows_total, r = blockIdx.x % rows_total;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const int64_t stride = (int64_t)rows_total * (D + kPartStride);
    const float *pr = part + ((int64_t)g * n_splits * rows_total + r) * (D + kPartStride);
    const int sl = tid / LPS, dq = tid % LPS;

    // one round trip for what most launches need: the thread's first PRE
    // partial-row slices and (m, l) of split tid; later ones are read as used
    constexpr int PRE = 8;
    float4 held[PRE];
#pragma unroll
    for (int k = 0; k < PRE; ++k) {
        const int s = sl + k * SPI;
        held[k] = s < n_splits ? *reinterpret_cast<const float4 *>(pr + s * stride + dq * 4)
                               : make_float4(0.f, 0.f, 0.f, 0.f);
    }
    const float m0 = tid < n_splits ? pr[tid * stride + D] : -INFINITY;
    const float l0 = tid < n_splits ? pr[tid * stride + D + 1] : 0.f;
    float mx = m0;
    for (int s = tid + kCombineThreads; s < n_splits; s += kCombineThreads) mx = fmaxf(mx, pr[s * stride + D]);
    mx = wave_max(mx);
    if (lane == 0) sm_red[wave] = mx;
    __syncthreads();
    mx = sm_red[0];
#pragma unroll
    for (int w = 1; w < kCombineThreads / kWave; ++w) mx = fmaxf(mx, sm_red[w]);
    __syncthreads();
    float l = 0.f;
    for (int s = tid; s < n_splits; s += kCombineThreads) {
        const float ms = s == tid ? m0 : pr[s * stride + D];
        const float f = ms == -INFINITY ? 0.f : exp2f(ms - mx);
        sm_w[s] = f;
        l += (s == tid ? l0 : pr[s * stride + D + 1]) * f;
    }
    l = wave_sum_f(l);
    if (lane == 0) sm_red[wave] = l;
    __syncthreads();
    l = 0.f;
#pragma unroll
    for (int w = 0; w < kCombineThreads / kWave; ++w) l += sm_red[w];

    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int k = 0; k < PRE; ++k) {
        const int s = sl + k * SPI;
        if (s < n_splits) {
            const float f = sm_w[s];
            acc.x += held[k].x * f; acc.y += held[k].y * f; acc.z += held[k].z * f; acc.w += held[k].w * f;
        }
    }
#pragma unroll 8
    for (int s = sl + PRE * SPI; s < n_splits; s += SPI) {
        const float4 v = *reinterpret_cast<const float4 *>(pr + s * stride + dq * 4);
        const float f = sm_w[s];
        acc.x += v.x * f; acc.y += v.y * f; acc.z += v.z * f; acc.w += v.w * f;
    }
    sm_acc[sl][dq] = acc;
    __syncthreads();
    if (tid < LPS) {
        float4 t = sm_acc[0][tid];
        for (int i = 1; i < SPI; ++i) {
            const float4 u = sm_acc[i][tid];
            t.x += u.x; t.y += u.y; t.z += u.z; t.w += u.w;
        }
        const float inv = 1.f / l;
        const int m = r / group, h = g * group + r % group;
        *reinterpret_cast<float4 *>(out + ((int64_t)m * n_q_heads + h) * D + tid * 4) =
            make_float4(t.x * inv, t.y * inv, t.z * inv, t.w * inv);
        if (lse && tid == 0) lse[(int64_t)m * n_q_heads + h] = (mx + log2f(l)) * kLn2;
    }
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

template <typename T, int D, int BT, int RH>
hipError_t launch_row16(const AttnPlan &p, const float *q, const void *k_pool, const void *v_pool,
                        int64_t n_pages, const int32_t *view_pages, float qscale, float *part,
                        hipStream_t stream) {
    dim3 grid(p.n_splits, p.n_kv_heads, p.rows_per_head / RH);
    hipLaunchKernelGGL((attn_splitk_row16_kernel<T, D, BT, RH>), grid, dim3(kAttnThreads), 0, stream, q,
                       static_cast<const T *>(k_pool), static_cast<const T *>(v_pool), n_pages,
                       view_pages, p.n_sel, p.n_view, p.last_page_tokens, p.n_kv_heads, p.n_q_heads,
                       p.group, p.rows_per_head, p.pages_per_split, p.n_splits, qscale, part);
    return hipGetLastError();
}

template <typename T, int D, int BT>
hipError_t launch_mfma16(const AttnPlan &p, const float *q, const void *k_pool, const void *v_pool,
                         int64_t n_pages, const int32_t *view_pages, float qscale, float *part,
                         hipStream_t stream) {
    dim3 grid(p.n_splits, p.n_kv_heads, (p.rows_per_head + kMfmaRows - 1) / kMfmaRows);
    hipLaunchKernelGGL((attn_mfma16_kernel<T, D, BT>), grid, dim3(kAttnThreads), 0, stream, q,
                       static_cast<const T *>(k_pool), static_cast<const T *>(v_pool), n_pages,
                       view_pages, p.n_sel, p.n_view, p.last_page_tokens, p.n_kv_heads, p.n_q_heads,
                       p.group, p.rows_per_head, p.pages_per_split, p.n_splits, qscale, p.v_scale, part);
    return hipGetLastError();
}

// rows per KV head from which K/V tiles are shared through LDS by 64-row groups
constexpr int kRowsLds = 48;

template <typename T, int D, int BT, int NW>
hipError_t launch_mfma_rows_nw(const AttnPlan &p, const float *q, const void *k_pool, const void *v_pool,
                               int64_t n_pages, const int32_t *view_pages, float qscale, float *part,
                               hipStream_t stream) {
    dim3 grid(p.n_splits, p.n_kv_heads, (p.rows_per_head + NW * kMfmaRows - 1) / (NW * kMfmaRows));
    hipLaunchKernelGGL((attn_mfma_rows_kernel<T, D, BT, NW>), grid, dim3(NW * kWave), 0, stream, q,
                       static_cast<const T *>(k_pool), static_cast<const T *>(v_pool), n_pages, view_pages, p.n_sel,
                       p.n_view, p.last_page_tokens, p.n_kv_heads, p.n_q_heads, p.group, p.rows_per_head,
                       p.pages_per_split, p.n_splits, qscale, p.v_scale, part);
    return hipGetLastError();
}

template <typename T, int D, int BT>
hipError_t launch_mfma_rows(const AttnPlan &p, const float *q, const void *k_pool, const void *v_pool,
                            int64_t n_pages, const int32_t *view_pages, float qscale, float *part,
                            hipStream_t stream) {
    if (p.rows_per_head <= 64)
        return launch_mfma_rows_nw<T, D, BT, 4>(p, q, k_pool, v_pool, n_pages, view_pages, qscale, part, stream);
    if (p.rows_per_head <= 128)
        return launch_mfma_rows_nw<T, D, BT, 8>(p, q, k_pool, v_pool, n_pages, view_pages, qscale, part, stream);
    return launch_mfma_rows_nw<T, D, BT, 16>(p, q, k_pool, v_pool, n_pages, view_pages, qscale, part, stream);
}

template <typename T, int D, int BT>
hipError_t launch_bt(const AttnPlan &p, const float *q, const void *k, const void *v, int64_t n_pages,
                     const int32_t *vp, float qscale, float *part, hipStream_t stream) {
    const int rows = p.rows_per_head;
    if constexpr (std::is_same<T, uint8_t>::value) {
        // FP8: always the matrix cores (rows padded to 16)
        if (rows >= kRowsLds) return launch_mfma_rows<T, D, BT>(p, q, k, v, n_pages, vp, qscale, part, stream);
        return launch_mfma16<T, D, BT>(p, q, k, v, n_pages, vp, qscale, part, stream);
    } else {
        if constexpr (std::is_same<T, uint16_t>::value) {
            // bf16 with 3 or more rows per KV head: matrix cores (rows padded to 16)
            if (rows >= kRowsLds) return launch_mfma_rows<T, D, BT>(p, q, k, v, n_pages, vp, qscale, part, stream);
            if (rows >= 3) return launch_mfma16<T, D, BT>(p, q, k, v, n_pages, vp, qscale, part, stream);
        }
        if constexpr (D / Vec16<T>::N == 16) {
            if (rows % 8 == 0) return launch_row16<T, D, BT, 8>(p, q, k, v, n_pages, vp, qscale, part, stream);
            if (rows % 4 == 0) return launch_row16<T, D, BT, 4>(p, q, k, v, n_pages, vp, qscale, part, stream);
        }
        // 8 rows per workgroup, except fp32 K/V with d = 128 and 64-token pages, whose
        // 8-row kernel does not fit the registers
        if constexpr (!(std::is_same<T, float>::value && D == 128 && BT == 64)) {
            if (rows % 8 == 0) return launch_rh<T, D, BT, 8>(p, q, k, v, n_pages, vp, qscale, part, stream);
        }
        if (rows % 4 == 0) return launch_rh<T, D, BT, 4>(p, q, k, v, n_pages, vp, qscale, part, stream);
        if (rows % 2 == 0) return launch_rh<T, D, BT, 2>(p, q, k, v, n_pages, vp, qscale, part, stream);
        return launch_rh<T, D, BT, 1>(p, q, k, v, n_pages, vp, qscale, part, stream);
    }
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
    const float qscale = scale * kLog2e * p.k_scale;  // k_scale is 1 unless the pools are FP8
    hipError_t e;
    auto go = [&](auto elem, auto dim) {
        return launch_d<decltype(elem), decltype(dim)::value>(p, q, k_pool, v_pool, n_pages, view_pages, qscale,
                                                              part, stream);
    };
    using D64 = std::integral_constant<int, 64>;
    using D128 = std::integral_constant<int, 128>;
    if (p.kv_dtype == 2)
        e = p.head_dim == 128 ? go(uint8_t{}, D128{}) : go(uint8_t{}, D64{});
    else if (p.kv_dtype == 1)
        e = p.head_dim == 128 ? go(uint16_t{}, D128{}) : go(uint16_t{}, D64{});
    else
        e = p.head_dim == 128 ? go(float{}, D128{}) : go(float{}, D64{});
    if (e != hipSuccess) return e;
    const dim3 grid(p.n_kv_heads * p.rows_per_head);
    const size_t lds = sizeof(float) * (size_t)p.n_splits;
    if (p.head_dim == 128)
        hipLaunchKernelGGL((attn_combine_kernel<128>), grid, dim3(kCombineThreads), lds, stream, part,
                           p.n_splits, p.rows_per_head, p.n_q_heads, p.group, out, lse);
    else
        hipLaunchKernelGGL((attn_combine_kernel<64>), grid, dim3(kCombineThreads), lds, stream, part,
                           p.n_splits, p.rows_per_head, p.n_q_heads, p.group, out, lse);
    return hipGetLastError();
}

}  // namespace kvmem
