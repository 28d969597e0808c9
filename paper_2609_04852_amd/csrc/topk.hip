// Selector (Sec. 4.3, default selector; Sec. 5.2): pick the k_eff candidates
// with the largest fp32 score R (ties: lower block id), and write the view
// [sink blocks] ++ [selected, ascending] ++ [recent blocks] with its pages.
//
// R >= 0, so key = bits(R) + 1 orders like R (and 0 is free for "absent");
// bit 31 of a key is always 0.  The selection is a two-level radix select
// followed by an exact finish, spread over one workgroup per chunk of
// kSelChunk candidates:
//
//   score reduction  histograms every candidate's key by bits 30..19
//                    (kSelBins bins) into a per-selection global histogram.
//   sel_refine       every workgroup finds the pivot bin -- the bin holding
//                    the k-th largest key -- from that histogram, counts its
//                    keys above the pivot bin, appends its pivot-bin keys (with
//                    their candidate index) to the row's pivot-bin array, and
//                    adds them to a second global histogram by bits 18..8
//                    (kSelBins2).
//   sel_finish       every workgroup finds the sub-pivot bin in the second
//                    histogram, passes once over the pivot-bin keys to collect
//                    the few keys of the sub-pivot bin in LDS, and ranks those
//                    exactly by (key desc, candidate asc).  That gives the
//                    threshold key T and the tie cut c_T of the k-th key: a
//                    candidate is selected iff key > T or (key == T and
//                    c <= c_T).  The workgroup counts the selections of the
//                    chunks before its own for its output offset, and a
//                    block-wide prefix sum puts each selected id of its chunk
//                    at its place, so the view comes out in chronological
//                    order without a sort; pages are looked up as ids are
//                    written.  Every workgroup takes the same small decision
//                    itself instead of waiting for one to broadcast it.
//
// When the sub-pivot bin holds many keys (near-equal scores), the finish falls
// back to an MSB-first radix select over them (in LDS, or from the pivot-bin
// array when they do not fit).  All counts are integers, so the selection is exact
// and deterministic.
#include "kvmem_device.h"
#include "kvmem_internal.h"

namespace kvmem {
namespace {

constexpr int kChunkThreads = kSelChunk / 4;  // 4 candidates per thread
constexpr int kFinishThreads = kChunkThreads;
constexpr int kDigitBits = 11;
constexpr int kSubShift = kSelShift1 - 11;  // second-level digit: the 11 key bits below the first
constexpr int kWindowCap = 8192;        // sub-pivot keys kept in LDS
constexpr int kBruteMax = kFinishThreads;  // sub-pivot sets ranked pairwise
static_assert(kSelBins2 << kSubShift == 1 << kSelShift1, "second level = the bits below the first");

enum { kCtrlPivot = 0, kCtrlRank = 3 };

__device__ inline uint32_t mask_above(int bit) { return bit >= 31 ? 0u : (~0u << (bit + 1)); }
__device__ inline uint32_t bin1(uint32_t key) { return (key >> kSelShift1) & (kSelBins - 1); }
__device__ inline uint32_t bin2(uint32_t key) { return (key >> kSubShift) & (kSelBins2 - 1); }

// The bin holding rank k (1-based, descending) of histogram gh and the number
// of items in the bins above it (all threads of the workgroup get the values).
// gh may hold COPIES copies of the histogram, copy_stride words apart, whose
// counts add up.
template <int NT, int NBINS, int COPIES = 1>
__device__ void find_pivot(const uint32_t *__restrict__ gh, uint32_t k, uint32_t *scratch,
                           uint32_t *s_out, uint32_t *pivot, uint32_t *above, int64_t copy_stride = 0) {
    constexpr int PER = NBINS / NT;  // bins per thread, descending
    static_assert(PER * NT == NBINS, "bins divide evenly");
    uint32_t cnt[PER];
    uint32_t mine = 0u;
    uint32_t part[COPIES][PER];
#pragma unroll
    for (int c = 0; c < COPIES; ++c)
#pragma unroll
        for (int i = 0; i < PER; ++i) part[c][i] = gh[c * copy_stride + NBINS - 1 - (threadIdx.x * PER + i)];
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        cnt[i] = 0u;
#pragma unroll
        for (int c = 0; c < COPIES; ++c) cnt[i] += part[c][i];
        mine += cnt[i];
    }
    uint32_t total;
    uint32_t run = block_exclusive_scan<NT>(mine, scratch, &total);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        if (run < k && run + cnt[i] >= k) {
            s_out[0] = (uint32_t)(NBINS - 1 - (threadIdx.x * PER + i));
            s_out[1] = run;
        }
        run += cnt[i];
    }
    __syncthreads();
    *pivot = s_out[0];
    *above = s_out[1];
    __syncthreads();
}

// Loads candidates 4t..4t+3 of chunk `chunk` (keys; 0 past n_cand >= 1).
// Score rows are padded to a multiple of 64 floats, so a float4 slot that
// starts below n_cand is in bounds.
__device__ inline void load_chunk_keys(const float *R, int chunk, int n_cand, uint32_t (&k)[4], int &c0) {
    c0 = chunk * kSelChunk + 4 * threadIdx.x;
    // clamped rather than skipped: a load under a per-lane condition becomes a
    // branch of its own, and the compiler then waits for each such load alone
    const float4 x = *reinterpret_cast<const float4 *>(R + min(c0, (n_cand - 1) & ~3));
    const float v[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) k[e] = c0 + e < n_cand ? __float_as_uint(v[e]) + 1u : 0u;
}

// Pointers into the histogram area of the workspace (n_sel rows).
struct SelHist {
    uint32_t *h1, *h2, *count;
    int64_t h1_stride;  // words between the copies of the first-level histogram
    __device__ SelHist(uint32_t *hist, int sel, int n_sel)
        : h1(hist + (int64_t)sel * kSelBins),
          h2(hist + (int64_t)kHistCopies * n_sel * kSelBins + (int64_t)sel * kSelBins2),
          count(hist + (int64_t)n_sel * (kHistCopies * kSelBins + kSelBins2) + sel),
          h1_stride((int64_t)n_sel * kSelBins) {}
};

__global__ __launch_bounds__(kChunkThreads) void sel_refine_kernel(
    const float *__restrict__ r32, int64_t r_stride, uint32_t *__restrict__ hist, int n_cand, int k_eff,
    int n_chunks, uint32_t *__restrict__ ctrl, uint32_t *__restrict__ above_cnt, uint2 *__restrict__ seg) {
    __shared__ uint32_t scratch[kChunkThreads / kWave + 1];
    __shared__ uint32_t s_out[2];
    __shared__ uint32_t s_base;
    __shared__ uint32_t lh[kSelBins2];
    if (k_eff <= 0) return;
    const int chunk = blockIdx.x, sel = blockIdx.y;
    const SelHist h(hist, sel, gridDim.y);
    for (int i = threadIdx.x; i < kSelBins2; i += kChunkThreads) lh[i] = 0u;
    // the chunk's keys do not depend on the pivot: read them with the histogram
    uint32_t k[4];
    int c0;
    load_chunk_keys(r32 + (int64_t)sel * r_stride, chunk, n_cand, k, c0);
    uint32_t pivot, above_all;
    find_pivot<kChunkThreads, kSelBins, kHistCopies>(h.h1, (uint32_t)k_eff, scratch, s_out, &pivot, &above_all,
                                                     h.h1_stride);
    if (chunk == 0 && threadIdx.x == 0) {
        ctrl[sel * 8 + kCtrlPivot] = pivot;
        ctrl[sel * 8 + kCtrlRank] = (uint32_t)k_eff - above_all;  // rank inside the pivot bin
    }
    uint32_t n_above = 0u, n_in = 0u;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (k[e] == 0u) continue;
        n_above += bin1(k[e]) > pivot ? 1u : 0u;
        n_in += bin1(k[e]) == pivot ? 1u : 0u;
    }
    uint32_t tot_above, tot_in;
    block_exclusive_scan<kChunkThreads>(n_above, scratch, &tot_above);
    uint32_t pos = block_exclusive_scan<kChunkThreads>(n_in, scratch, &tot_in);
    if (threadIdx.x == 0) {
        above_cnt[sel * n_chunks + chunk] = tot_above;
        // this chunk's place in the row's pivot-bin array (chunks in any order)
        if (tot_in) s_base = atomicAdd(h.count, tot_in);
    }
    if (tot_in == 0u) return;
    __syncthreads();
    pos += s_base;
    uint2 *row = seg + (int64_t)sel * n_chunks * kSelChunk;
#pragma unroll
    for (int e = 0; e < 4; ++e)
        if (k[e] != 0u && bin1(k[e]) == pivot) {
            row[pos++] = make_uint2(k[e], (uint32_t)(c0 + e));
            atomicAdd(&lh[bin2(k[e])], 1u);
        }
    __syncthreads();
    // the thread's bins read from LDS at once, then the non-empty ones added
    constexpr int PER = kSelBins2 / kChunkThreads;
    static_assert(PER * kChunkThreads == kSelBins2, "bins split evenly");
    uint32_t cnt[PER];
#pragma unroll
    for (int u = 0; u < PER; ++u) cnt[u] = lh[threadIdx.x + kChunkThreads * u];
#pragma unroll
    for (int u = 0; u < PER; ++u)
        if (cnt[u]) atomicAdd(&h.h2[threadIdx.x + kChunkThreads * u], cnt[u]);
}

struct FinishShared {
    uint32_t hist[1 << kDigitBits];
    uint32_t scratch[kFinishThreads / kWave + 1];
    uint32_t red_a[kFinishThreads / kWave], red_b[kFinishThreads / kWave];
    uint32_t s_out[2];
    uint32_t s_digit, s_krem;
    uint32_t s_thr, s_cut;
    uint32_t wcnt[kFinishThreads / kWave];  // sub-pivot keys found by each wave
    // sub-pivot (key, candidate), in no particular order: wave w fills
    // window[w * kWaveCap ...]
    uint2 window[kWindowCap];
};
constexpr int kWaveCap = kWindowCap / (kFinishThreads / kWave);

__device__ inline void block_and_or(uint32_t &a, uint32_t &o, FinishShared &sh) {
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
#pragma unroll
    for (int s = kWave / 2; s >= 1; s >>= 1) {
        a &= __shfl_xor(a, s, kWave);
        o |= __shfl_xor(o, s, kWave);
    }
    if (lane == 0) { sh.red_a[wave] = a; sh.red_b[wave] = o; }
    __syncthreads();
    a = ~0u; o = 0u;
#pragma unroll
    for (int w = 0; w < kFinishThreads / kWave; ++w) { a &= sh.red_a[w]; o |= sh.red_b[w]; }
    __syncthreads();
}

// Key of rank k (1-based, descending) among the items get(i, &key), i < nmax,
// of every thread (get returns false for an absent item).  Returns the key;
// *k_rem receives how many items equal to it are needed to reach rank k.
// Requires 1 <= k <= number of items.  Called by the whole workgroup.  The
// bits shared by all keys are skipped, then each pass histograms the next 11
// bits of the keys that still match the resolved prefix.
template <typename Get>
__device__ uint32_t exact_rank(Get get, int nmax, uint32_t k, FinishShared &sh, uint32_t *k_rem) {
    constexpr int NT = kFinishThreads;
    const int tid = threadIdx.x;
    uint32_t a = ~0u, o = 0u;
    for (int i = 0; i < nmax; ++i) {
        uint32_t key;
        if (get(i, &key)) { a &= key; o |= key; }
    }
    block_and_or(a, o, sh);
    const uint32_t diff = a ^ o;
    uint32_t prefix = a, krem = k;
    if (diff != 0u) {
        int bit = 31 - __clz(diff);
        prefix = a & mask_above(bit);
        while (bit >= 0) {
            const int nb = bit + 1 < kDigitBits ? bit + 1 : kDigitBits;
            const int shift = bit + 1 - nb;
            const int nbins = 1 << nb;
            const uint32_t dmask = (uint32_t)nbins - 1u, above = mask_above(bit);
            for (int i = tid; i < nbins; i += NT) sh.hist[i] = 0u;
            __syncthreads();
            for (int i = 0; i < nmax; ++i) {
                uint32_t key;
                if (get(i, &key) && (key & above) == prefix) atomicAdd(&sh.hist[(key >> shift) & dmask], 1u);
            }
            __syncthreads();
            constexpr int kPerMax = (1 << kDigitBits) / NT;
            const int per = (nbins + NT - 1) / NT;
            uint32_t cnt[kPerMax] = {};
            uint32_t mine = 0u;
            for (int i = 0; i < per; ++i) {
                const int rank = tid * per + i;
                if (rank < nbins) cnt[i] = sh.hist[nbins - 1 - rank];
                mine += cnt[i];
            }
            uint32_t total;
            uint32_t run = block_exclusive_scan<NT>(mine, sh.scratch, &total);
            for (int i = 0; i < per; ++i) {
                const int rank = tid * per + i;
                if (rank < nbins && run < krem && run + cnt[i] >= krem) {
                    sh.s_digit = (uint32_t)(nbins - 1 - rank);
                    sh.s_krem = krem - run;
                }
                run += cnt[i];
            }
            __syncthreads();
            prefix |= sh.s_digit << shift;
            krem = sh.s_krem;
            bit -= nb;
            __syncthreads();
        }
    }
    *k_rem = krem;
    return prefix;
}

__global__ __launch_bounds__(kFinishThreads) void sel_finish_kernel(
    const float *__restrict__ r32, int64_t r_stride, int n_cand, int k_eff, int n_sink, int n_recent,
    int n_blocks, int n_view, int n_chunks, uint32_t *__restrict__ hist, const uint32_t *__restrict__ ctrl,
    const uint32_t *__restrict__ above_cnt, const uint2 *__restrict__ seg,
    const int32_t *__restrict__ block_to_page, int32_t *__restrict__ view_blocks,
    int32_t *__restrict__ view_pages) {
    constexpr int NT = kFinishThreads, NW = NT / kWave;
    __shared__ FinishShared sh;
    const int chunk = blockIdx.x, sel = blockIdx.y;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    int32_t *vb = view_blocks + (int64_t)sel * n_view;
    int32_t *vp = view_pages + (int64_t)sel * n_view;
    if (chunk == 0) {
        for (int i = tid; i < n_sink; i += NT) {
            vb[i] = i;
            vp[i] = block_to_page[i];
        }
        for (int i = tid; i < n_recent; i += NT) {
            const int b = n_blocks - n_recent + i;
            vb[n_sink + k_eff + i] = b;
            vp[n_sink + k_eff + i] = block_to_page[b];
        }
    }
    if (k_eff <= 0) return;
    const SelHist h(hist, sel, gridDim.y);
    const uint2 *row = seg + (int64_t)sel * n_chunks * kSelChunk;
    // Everything that does not depend on this kernel's decisions is read up
    // front, in one round trip: the first U pivot-bin items of each thread
    // (read before their count is known; the array holds n_chunks * kSelChunk
    // items, those past the count are ignored), the chunk's keys and their
    // pages, and the selections above the pivot bin in the chunks before it.
    constexpr int U = 8;  // pivot-bin items per thread in flight
    const uint32_t cap = (uint32_t)n_chunks * kSelChunk;
    uint2 first[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const uint32_t i = (uint32_t)(tid + u * NT);
        first[u] = row[min(i, cap - 1u)];
    }
    uint32_t k[4];
    int c0;
    load_chunk_keys(r32 + (int64_t)sel * r_stride, chunk, n_cand, k, c0);
    int32_t pg[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) pg[e] = block_to_page[n_sink + min(c0 + e, n_cand - 1)];
    uint32_t before = 0u;  // selections of the chunks before this one
    for (int i = tid; i < chunk; i += NT) before += above_cnt[(int64_t)sel * n_chunks + i];
    const uint32_t k_in = ctrl[sel * 8 + kCtrlRank];  // rank inside the pivot bin
    const uint32_t n_b = min(*h.count, (uint32_t)n_cand);  // keys in the pivot bin (<= n_cand)
    // sub-pivot bin and the rank inside it (its barriers also publish `above`)
    uint32_t sub, above_sub;
    find_pivot<NT, kSelBins2>(h.h2, k_in, sh.scratch, sh.s_out, &sub, &above_sub);
    const uint32_t k_sub = k_in - above_sub;
    const uint32_t c_start = (uint32_t)chunk * kSelChunk;
    // one pass over the pivot-bin keys: those above the sub-pivot bin are
    // selected (count the ones of earlier chunks), the sub-pivot ones go to
    // this wave's part of the LDS window (no atomics: ballot + popcount)
    uint32_t wn = 0u;
    const uint64_t lt_mask = (1ull << lane) - 1ull;
    auto visit = [&](bool valid, uint2 it) {
        const uint32_t b2 = bin2(it.x);
        before += (valid && b2 > sub && it.y < c_start) ? 1u : 0u;
        const bool in = valid && b2 == sub;
        const uint64_t m = __ballot(in);
        const uint32_t idx = wn + (uint32_t)__popcll(m & lt_mask);
        if (in && idx < (uint32_t)kWaveCap) sh.window[wave * kWaveCap + idx] = it;
        wn += (uint32_t)__popcll(m);
    };
    {
        const int n_iter = (int)((n_b + NT - 1) / NT);
#pragma unroll
        for (int u = 0; u < U; ++u) visit((uint32_t)(tid + u * NT) < n_b, first[u]);
        for (int j0 = U; j0 < n_iter; j0 += U) {
            uint2 it[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const uint32_t i = (uint32_t)(tid + (j0 + u) * NT);
                it[u] = row[min(i, n_b - 1u)];  // n_b >= 1 here
            }
#pragma unroll
            for (int u = 0; u < U; ++u) visit((uint32_t)(tid + (j0 + u) * NT) < n_b, it[u]);
        }
    }
    if (lane == 0) sh.wcnt[wave] = wn;
    __syncthreads();
    uint32_t wc[NW], wp[NW + 1];  // per-wave counts and their prefix
    bool overflow = false;
    wp[0] = 0u;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
        wc[w] = sh.wcnt[w];
        overflow |= wc[w] > (uint32_t)kWaveCap;
        wp[w + 1] = wp[w] + wc[w];
    }
    const uint32_t n_sub = wp[NW];  // 1 <= k_sub <= n_sub
    // item i < n_sub of the sub-pivot set in LDS
    auto win = [&](uint32_t i) {
        int w = 0;
#pragma unroll
        for (int v = 1; v < NW; ++v) w += i >= wp[v] ? 1 : 0;
        return sh.window[w * kWaveCap + (i - wp[w])];
    };
    if (n_sub <= (uint32_t)kBruteMax) {
        // rank of each sub-pivot key by (key desc, candidate asc) by comparing
        // it with all others; the k_sub-th one gives T and c_T
        const uint2 mine = tid < (int)n_sub ? win((uint32_t)tid) : make_uint2(0u, 0u);
        uint32_t rank = 0u;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const uint2 *part = sh.window + w * kWaveCap;
#pragma unroll 4
            for (uint32_t j = 0; j < wc[w]; ++j) {
                const uint2 o = part[j];
                rank += (o.x > mine.x || (o.x == mine.x && o.y < mine.y)) ? 1u : 0u;
            }
        }
        if (tid < (int)n_sub) {
            if (rank == k_sub - 1u) { sh.s_thr = mine.x; sh.s_cut = mine.y; }
            before += (rank < k_sub && mine.y < c_start) ? 1u : 0u;
        }
        __syncthreads();
    } else {
        // many near-equal keys: radix select over the sub-pivot set, in LDS when
        // it fits, else filtered again from the pivot-bin array
        const uint32_t n_items = overflow ? n_b : n_sub;
        auto get_item = [&](int j, uint2 *it) {
            const uint32_t i = (uint32_t)(tid + j * NT);
            if (i >= n_items) return false;
            if (!overflow) {
                *it = win(i);
                return true;
            }
            *it = row[i];
            return bin2(it->x) == sub;
        };
        const int nmax = (int)((n_items + NT - 1) / NT);
        uint32_t k_rem;
        const uint32_t thr = exact_rank([&](int j, uint32_t *key) {
            uint2 it;
            if (!get_item(j, &it)) return false;
            *key = it.x;
            return true;
        }, nmax, k_sub, sh, &k_rem);
        // among keys equal to thr, the k_rem lowest candidate ids: rank k_rem
        // of ~c, which is larger for lower c
        uint32_t n_tie = 0u;
        for (int j = 0; j < nmax; ++j) {
            uint2 it;
            if (get_item(j, &it) && it.x == thr) ++n_tie;
        }
        uint32_t n_tie_all;
        block_exclusive_scan<NT>(n_tie, sh.scratch, &n_tie_all);
        uint32_t cut = 0xFFFFFFFFu;
        if (k_rem < n_tie_all) {
            uint32_t dummy;
            const uint32_t kk = exact_rank([&](int j, uint32_t *key) {
                uint2 it;
                if (!get_item(j, &it) || it.x != thr) return false;
                *key = ~it.y;
                return true;
            }, nmax, k_rem, sh, &dummy);
            cut = ~kk;
        }
        for (int j = 0; j < nmax; ++j) {
            uint2 it;
            if (get_item(j, &it) && it.y < c_start && (it.x > thr || (it.x == thr && it.y <= cut))) ++before;
        }
        if (tid == 0) { sh.s_thr = thr; sh.s_cut = cut; }
        __syncthreads();
    }
    const uint32_t thr = sh.s_thr, cut = sh.s_cut;
    // output offset of this chunk: every selection in the chunks before it
    uint32_t base;
    block_exclusive_scan<NT>(before, sh.scratch, &base);
    // emit this chunk's selected candidates in order
    bool take[4];
    uint32_t n_take = 0u;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        take[e] = k[e] != 0u && (k[e] > thr || (k[e] == thr && (uint32_t)(c0 + e) <= cut));
        n_take += take[e] ? 1u : 0u;
    }
    uint32_t tot;
    uint32_t pos = base + block_exclusive_scan<NT>(n_take, sh.scratch, &tot);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (!take[e] || pos >= (uint32_t)k_eff) continue;  // pos < k_eff by construction
        vb[n_sink + pos] = n_sink + c0 + e;
        vp[n_sink + pos] = pg[e];
        ++pos;
    }
}

}  // namespace

hipError_t launch_topk(const SelectPlan &p, const int32_t *b2p, int32_t *vb, int32_t *vp, char *ws,
                       hipStream_t stream) {
    const float *r32 = reinterpret_cast<const float *>(ws + p.off_r32);
    uint32_t *hist = reinterpret_cast<uint32_t *>(ws + p.off_hist);
    uint32_t *ctrl = reinterpret_cast<uint32_t *>(ws + p.off_ctrl);
    uint32_t *above = reinterpret_cast<uint32_t *>(ws + p.off_above);
    uint2 *seg = reinterpret_cast<uint2 *>(ws + p.off_seg);
    // one workgroup per chunk (at least one per row: it writes sink and recent)
    const dim3 chunks(p.n_chunks > 0 ? p.n_chunks : 1, p.n_sel);
    hipLaunchKernelGGL(sel_refine_kernel, chunks, dim3(kChunkThreads), 0, stream, r32, (int64_t)p.cand_stride,
                       hist, p.n_cand, p.k_eff, p.n_chunks, ctrl, above, seg);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sel_finish_kernel, chunks, dim3(kFinishThreads), 0, stream, r32, (int64_t)p.cand_stride,
                       p.n_cand, p.k_eff, p.n_sink, p.n_recent, p.n_blocks, p.n_view, p.n_chunks, hist, ctrl,
                       above, seg, b2p, vb, vp);
    return hipGetLastError();
}

}  // namespace kvmem
