// Selector (Sec. 4.3, default selector; Sec. 5.2): pick the k_eff candidates
// with the largest fp32 score R (ties: lower block id), and write the view
// [sink blocks] ++ [selected, ascending] ++ [recent blocks] with its pages.
//
// R >= 0, so key = bits(R) + 1 orders like R (and 0 is free for "absent").
// The score reduction has already histogrammed every candidate's key by bits
// 30..19 (kSelBins bins) into a per-selection global histogram.  Three stages
// follow, so that the memory traffic is spread over many workgroups and only
// a small decision runs in a single one:
//
//   sel_refine  (one workgroup per chunk of kSelChunk candidates): every
//               workgroup finds the pivot bin -- the bin holding the k-th
//               largest key -- from the histogram, counts its keys above the
//               pivot bin, and writes its pivot-bin keys (with their candidate
//               index) to its own segment, in index order.
//   sel_decide  (one workgroup per selection row): gathers the pivot-bin keys
//               (usually a few thousand) into LDS and runs an exact MSB-first
//               radix select on them for the remaining rank: threshold key T
//               and k_rem = how many keys equal to T are taken.  Among those,
//               the k_rem lowest candidate ids win (a second radix select on
//               the ids gives the cut c_T).  It then counts the selected keys
//               per chunk and turns the counts into output offsets.
//   sel_emit    (one workgroup per chunk): selected = key > T or (key == T and
//               c <= c_T); a block-wide prefix sum plus the chunk's offset puts
//               each id at its place, so the view comes out in chronological
//               order without a sort; the page of each block is looked up as
//               it is written.
//
// All counts are integers, so the selection is exact and deterministic.
#include "kvmem_device.h"
#include "kvmem_internal.h"

namespace kvmem {
namespace {

constexpr int kChunkThreads = kSelChunk / 4;  // 4 candidates per thread
constexpr int kDecideThreads = 1024;
constexpr int kDigitBits = 11;
constexpr int kWindowCap = 8192;  // pivot-bin keys kept in LDS by sel_decide

enum { kCtrlPivot = 0, kCtrlThr = 1, kCtrlTieCut = 2, kCtrlRank = 3 };

__device__ inline uint32_t mask_above(int bit) { return bit >= 31 ? 0u : (~0u << (bit + 1)); }

// The pivot bin and the number of keys above it, from the descending
// histogram scan (all threads of the workgroup return the same values).
template <int NT>
__device__ void find_pivot(const uint32_t *__restrict__ gh, uint32_t k, uint32_t *scratch,
                           uint32_t *s_out, uint32_t *pivot, uint32_t *above) {
    constexpr int PER = kSelBins / NT;  // bins per thread, descending
    uint32_t cnt[PER];
    uint32_t mine = 0u;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        cnt[i] = gh[kSelBins - 1 - (threadIdx.x * PER + i)];
        mine += cnt[i];
    }
    uint32_t total;
    uint32_t run = block_exclusive_scan<NT>(mine, scratch, &total);
#pragma unroll
    for (int i = 0; i < PER; ++i) {
        if (run < k && run + cnt[i] >= k) {
            s_out[0] = (uint32_t)(kSelBins - 1 - (threadIdx.x * PER + i));
            s_out[1] = run;
        }
        run += cnt[i];
    }
    __syncthreads();
    *pivot = s_out[0];
    *above = s_out[1];
    __syncthreads();
}

// Loads candidates 4t..4t+3 of chunk `chunk` (keys; 0 past n_cand).  Score
// rows are padded to a multiple of 64 floats, so a float4 slot that starts
// below n_cand is in bounds.
__device__ inline void load_chunk_keys(const float *R, int chunk, int n_cand, uint32_t (&k)[4], int &c0) {
    c0 = chunk * kSelChunk + 4 * threadIdx.x;
    const float4 x = c0 < n_cand ? *reinterpret_cast<const float4 *>(R + c0) : make_float4(0.f, 0.f, 0.f, 0.f);
    const float v[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) k[e] = c0 + e < n_cand ? __float_as_uint(v[e]) + 1u : 0u;
}

__global__ __launch_bounds__(kChunkThreads) void sel_refine_kernel(
    const float *__restrict__ r32, int64_t r_stride, const uint32_t *__restrict__ hist, int n_cand,
    int k_eff, int n_chunks, uint32_t *__restrict__ ctrl, uint32_t *__restrict__ above_cnt,
    uint32_t *__restrict__ seg_cnt, uint2 *__restrict__ seg) {
    __shared__ uint32_t scratch[kChunkThreads / kWave + 1];
    __shared__ uint32_t s_out[2];
    if (k_eff <= 0) return;
    const int chunk = blockIdx.x, sel = blockIdx.y;
    uint32_t pivot, above_all;
    find_pivot<kChunkThreads>(hist + (int64_t)sel * kSelBins, (uint32_t)k_eff, scratch, s_out, &pivot,
                              &above_all);
    if (chunk == 0 && threadIdx.x == 0) {
        ctrl[sel * 8 + kCtrlPivot] = pivot;
        ctrl[sel * 8 + kCtrlRank] = (uint32_t)k_eff - above_all;  // rank inside the pivot bin
    }
    uint32_t k[4];
    int c0;
    load_chunk_keys(r32 + (int64_t)sel * r_stride, chunk, n_cand, k, c0);
    uint32_t n_above = 0u, n_in = 0u;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (k[e] == 0u) continue;
        const uint32_t d = (k[e] >> 19) & (kSelBins - 1);
        n_above += d > pivot ? 1u : 0u;
        n_in += d == pivot ? 1u : 0u;
    }
    uint32_t tot_above, tot_in;
    block_exclusive_scan<kChunkThreads>(n_above, scratch, &tot_above);
    uint32_t pos = block_exclusive_scan<kChunkThreads>(n_in, scratch, &tot_in);
    uint2 *my_seg = seg + ((int64_t)sel * n_chunks + chunk) * kSelChunk;
#pragma unroll
    for (int e = 0; e < 4; ++e)
        if (k[e] != 0u && ((k[e] >> 19) & (kSelBins - 1)) == pivot)
            my_seg[pos++] = make_uint2(k[e], (uint32_t)(c0 + e));
    if (threadIdx.x == 0) {
        above_cnt[sel * n_chunks + chunk] = tot_above;
        seg_cnt[sel * n_chunks + chunk] = tot_in;
    }
}

struct DecideShared {
    uint32_t hist[1 << kDigitBits];
    uint32_t scratch[kDecideThreads / kWave + 1];
    uint32_t red_a[kDecideThreads / kWave], red_b[kDecideThreads / kWave];
    uint32_t s_digit, s_krem;
    uint32_t seg_base[kTopkMaxCand / kSelChunk + 1];
    uint32_t sel_cnt[kTopkMaxCand / kSelChunk];
    uint2 window[kWindowCap];  // pivot-bin (key, candidate)
};

__device__ inline void block_and_or(uint32_t &a, uint32_t &o, DecideShared &sh) {
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
    for (int w = 0; w < kDecideThreads / kWave; ++w) { a &= sh.red_a[w]; o |= sh.red_b[w]; }
    __syncthreads();
}

// Key of rank k (1-based, descending) among the items get(i, &key), i < nmax,
// of every thread (get returns false for an absent item).  Returns the key;
// *k_rem receives how many items equal to it are needed to reach rank k.
// Requires 1 <= k <= number of items.  Called by the whole workgroup.  The
// bits shared by all keys are skipped, then each pass histograms the next 11
// bits of the keys that still match the resolved prefix.
template <typename Get>
__device__ uint32_t exact_rank(Get get, int nmax, uint32_t k, DecideShared &sh, uint32_t *k_rem) {
    constexpr int NT = kDecideThreads;
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

__global__ __launch_bounds__(kDecideThreads) void sel_decide_kernel(
    int k_eff, int n_chunks, uint32_t *__restrict__ ctrl, const uint32_t *__restrict__ above_cnt,
    const uint32_t *__restrict__ seg_cnt, const uint2 *__restrict__ seg,
    uint32_t *__restrict__ chunk_off) {
    __shared__ DecideShared sh;
    if (k_eff <= 0) return;
    const int sel = blockIdx.x, tid = threadIdx.x;
    const uint32_t k_in = ctrl[sel * 8 + kCtrlRank];  // rank inside the pivot bin
    const uint2 *my_seg = seg + (int64_t)sel * n_chunks * kSelChunk;
    // segment bases (n_chunks <= 64: one wave scans them)
    if (tid < kWave) {
        const uint32_t c = tid < n_chunks ? seg_cnt[sel * n_chunks + tid] : 0u;
        uint32_t incl = c;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const uint32_t y = __shfl_up(incl, o, kWave);
            if (tid >= o) incl += y;
        }
        if (tid < n_chunks) sh.seg_base[tid] = incl - c;
        if (tid == kWave - 1) sh.seg_base[kTopkMaxCand / kSelChunk] = incl;
    }
    if (tid < n_chunks) sh.sel_cnt[tid] = 0u;
    __syncthreads();
    const uint32_t n_b = sh.seg_base[kTopkMaxCand / kSelChunk];
    const bool in_lds = n_b <= (uint32_t)kWindowCap;
    // item i of the pivot bin, in candidate order: its chunk by binary search
    auto item = [&](uint32_t i) {
        int lo = 0, hi = n_chunks - 1;
        while (lo < hi) {
            const int mid = (lo + hi + 1) / 2;
            if (sh.seg_base[mid] <= i) lo = mid; else hi = mid - 1;
        }
        return my_seg[(int64_t)lo * kSelChunk + (i - sh.seg_base[lo])];
    };
    if (in_lds) {
        for (uint32_t i = tid; i < n_b; i += kDecideThreads) sh.window[i] = item(i);
        __syncthreads();
    }
    const int nmax = (int)((n_b + kDecideThreads - 1) / kDecideThreads);
    auto get_item = [&](int j, uint2 *it) {
        const uint32_t i = (uint32_t)(tid + j * kDecideThreads);
        if (i >= n_b) return false;
        *it = in_lds ? sh.window[i] : item(i);
        return true;
    };
    // threshold key and how many keys equal to it are taken
    uint32_t k_rem;
    const uint32_t thr = exact_rank([&](int j, uint32_t *key) {
        uint2 it;
        if (!get_item(j, &it)) return false;
        *key = it.x;
        return true;
    }, nmax, k_in, sh, &k_rem);
    // among keys equal to thr, the k_rem lowest candidate ids: rank k_rem of
    // (2^16 - c), which is larger for lower c (c < 2^16)
    uint32_t n_tie = 0u;
    for (int j = 0; j < nmax; ++j) {
        uint2 it;
        if (get_item(j, &it) && it.x == thr) ++n_tie;
    }
    uint32_t n_tie_all;
    block_exclusive_scan<kDecideThreads>(n_tie, sh.scratch, &n_tie_all);
    uint32_t cut = 0xFFFFFFFFu;
    if (k_rem < n_tie_all) {
        uint32_t dummy;
        const uint32_t kk = exact_rank([&](int j, uint32_t *key) {
            uint2 it;
            if (!get_item(j, &it) || it.x != thr) return false;
            *key = 0x10000u - it.y;
            return true;
        }, nmax, k_rem, sh, &dummy);
        cut = 0x10000u - kk;
    }
    // selected pivot-bin keys per chunk, then the chunks' output offsets
    for (int j = 0; j < nmax; ++j) {
        uint2 it;
        if (get_item(j, &it) && (it.x > thr || (it.x == thr && it.y <= cut)))
            atomicAdd(&sh.sel_cnt[it.y / kSelChunk], 1u);
    }
    __syncthreads();
    if (tid < kWave) {
        const uint32_t c = tid < n_chunks ? above_cnt[sel * n_chunks + tid] + sh.sel_cnt[tid] : 0u;
        uint32_t incl = c;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const uint32_t y = __shfl_up(incl, o, kWave);
            if (tid >= o) incl += y;
        }
        if (tid < n_chunks) chunk_off[sel * n_chunks + tid] = incl - c;
    }
    if (tid == 0) {
        ctrl[sel * 8 + kCtrlThr] = thr;
        ctrl[sel * 8 + kCtrlTieCut] = cut;
    }
}

__global__ __launch_bounds__(kChunkThreads) void sel_emit_kernel(
    const float *__restrict__ r32, int64_t r_stride, int n_cand, int k_eff, int n_sink, int n_recent,
    int n_blocks, int n_view, int n_chunks, const uint32_t *__restrict__ ctrl,
    const uint32_t *__restrict__ chunk_off, const int32_t *__restrict__ block_to_page,
    int32_t *__restrict__ view_blocks, int32_t *__restrict__ view_pages) {
    __shared__ uint32_t scratch[kChunkThreads / kWave + 1];
    const int chunk = blockIdx.x, sel = blockIdx.y;
    int32_t *vb = view_blocks + (int64_t)sel * n_view;
    int32_t *vp = view_pages + (int64_t)sel * n_view;
    if (chunk == 0) {
        for (int i = threadIdx.x; i < n_sink; i += kChunkThreads) {
            vb[i] = i;
            vp[i] = block_to_page[i];
        }
        for (int i = threadIdx.x; i < n_recent; i += kChunkThreads) {
            const int b = n_blocks - n_recent + i;
            vb[n_sink + k_eff + i] = b;
            vp[n_sink + k_eff + i] = block_to_page[b];
        }
    }
    if (k_eff <= 0) return;
    const uint32_t thr = ctrl[sel * 8 + kCtrlThr], cut = ctrl[sel * 8 + kCtrlTieCut];
    uint32_t k[4];
    int c0;
    load_chunk_keys(r32 + (int64_t)sel * r_stride, chunk, n_cand, k, c0);
    bool take[4];
    uint32_t n_take = 0u;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        take[e] = k[e] != 0u && (k[e] > thr || (k[e] == thr && (uint32_t)(c0 + e) <= cut));
        n_take += take[e] ? 1u : 0u;
    }
    uint32_t tot;
    uint32_t pos = chunk_off[sel * n_chunks + chunk] + block_exclusive_scan<kChunkThreads>(n_take, scratch, &tot);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        if (!take[e] || pos >= (uint32_t)k_eff) continue;  // pos < k_eff by construction
        const int b = n_sink + c0 + e;
        vb[n_sink + pos] = b;
        vp[n_sink + pos] = block_to_page[b];
        ++pos;
    }
}

}  // namespace

hipError_t launch_topk(const SelectPlan &p, const int32_t *b2p, int32_t *vb, int32_t *vp, char *ws,
                       hipStream_t stream) {
    const float *r32 = reinterpret_cast<const float *>(ws + p.off_r32);
    const uint32_t *hist = reinterpret_cast<const uint32_t *>(ws + p.off_hist);
    uint32_t *ctrl = reinterpret_cast<uint32_t *>(ws + p.off_ctrl);
    uint32_t *above = reinterpret_cast<uint32_t *>(ws + p.off_above);
    uint32_t *segcnt = reinterpret_cast<uint32_t *>(ws + p.off_segcnt);
    uint32_t *chunkoff = reinterpret_cast<uint32_t *>(ws + p.off_chunkoff);
    uint2 *seg = reinterpret_cast<uint2 *>(ws + p.off_seg);
    const dim3 chunks(p.n_chunks, p.n_sel);
    hipLaunchKernelGGL(sel_refine_kernel, chunks, dim3(kChunkThreads), 0, stream, r32, (int64_t)p.cand_stride,
                       hist, p.n_cand, p.k_eff, p.n_chunks, ctrl, above, segcnt, seg);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(sel_decide_kernel, dim3(p.n_sel), dim3(kDecideThreads), 0, stream, p.k_eff,
                       p.n_chunks, ctrl, above, segcnt, seg, chunkoff);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(sel_emit_kernel, chunks, dim3(kChunkThreads), 0, stream, r32, (int64_t)p.cand_stride,
                       p.n_cand, p.k_eff, p.n_sink, p.n_recent, p.n_blocks, p.n_view, p.n_chunks, ctrl,
                       chunkoff, b2p, vb, vp);
    return hipGetLastError();
}

}  // namespace kvmem
