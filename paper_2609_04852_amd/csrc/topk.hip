// Selector (Sec. 4.3, default selector; Sec. 5.2): pick the k_eff candidates
// with the largest fp32 score R (ties: lower block id), and write the view
// [sink blocks] ++ [selected, ascending] ++ [recent blocks] with its pages.
//
// One workgroup of 1024 threads per selection row.  Thread t keeps the keys of
// candidates [t*IPT, (t+1)*IPT) in registers.  R >= 0, so the fp32 bit pattern
// read as uint32 orders like the value.  An MSB-first radix select finds the
// exact key T of the k_eff-th largest score: the bits common to every key are
// skipped (one AND/OR reduction), then each pass histograms the next 11 bits of
// the keys that still match the resolved prefix in LDS and picks the digit
// holding the k-th item.  With T known, and k_rem = how many of the items equal
// to T must be taken, one ordered pass selects key > T, plus the first k_rem
// items with key == T in block order -- the lower ids -- and block-wide prefix
// sums give each thread its output offset, so the selected ids come out already
// in chronological order with no sort.
#include "kvmem_device.h"
#include "kvmem_internal.h"

namespace kvmem {
namespace {

constexpr int kTopkThreads = 1024;
constexpr int kDigitBits = 11;

__device__ inline uint32_t mask_above(int bit) { return bit >= 31 ? 0u : (~0u << (bit + 1)); }

template <int IPT>
__global__ __launch_bounds__(kTopkThreads) void topk_select_kernel(
    const float *__restrict__ r32, int n_cand, int k_eff, int n_sink, int n_recent, int n_blocks,
    int n_view, const int32_t *__restrict__ block_to_page, int32_t *__restrict__ view_blocks,
    int32_t *__restrict__ view_pages) {
    __shared__ uint32_t hist[1 << kDigitBits];
    __shared__ uint32_t scratch[kTopkThreads / kWave + 1];
    __shared__ uint32_t red_and[kTopkThreads / kWave], red_or[kTopkThreads / kWave];
    __shared__ uint32_t s_digit, s_krem;

    const int sel = blockIdx.x;
    const int tid = threadIdx.x, lane = tid % kWave, wave = tid / kWave;
    const float *R = r32 + (int64_t)sel * n_cand;
    int32_t *vb = view_blocks + (int64_t)sel * n_view;
    int32_t *vp = view_pages + (int64_t)sel * n_view;
    const int c_begin = tid * IPT;

    uint32_t key[IPT];
#pragma unroll
    for (int j = 0; j < IPT; ++j) {
        const int c = c_begin + j;
        key[j] = c < n_cand ? __float_as_uint(R[c]) : 0u;
    }

    const bool take_all = k_eff >= n_cand;
    uint32_t thr = 0, k_rem = 0;
    if (!take_all && k_eff > 0) {
        uint32_t a = ~0u, o = 0u;
#pragma unroll
        for (int j = 0; j < IPT; ++j)
            if (c_begin + j < n_cand) { a &= key[j]; o |= key[j]; }
#pragma unroll
        for (int s = kWave / 2; s >= 1; s >>= 1) {
            a &= __shfl_xor(a, s, kWave);
            o |= __shfl_xor(o, s, kWave);
        }
        if (lane == 0) { red_and[wave] = a; red_or[wave] = o; }
        __syncthreads();
        a = ~0u; o = 0u;
        for (int w = 0; w < kTopkThreads / kWave; ++w) { a &= red_and[w]; o |= red_or[w]; }
        const uint32_t diff = a ^ o;
        uint32_t prefix = a;
        k_rem = (uint32_t)k_eff;
        if (diff != 0u) {
            int bit = 31 - __clz(diff);
            prefix = a & mask_above(bit);
            while (bit >= 0) {
                const int nb = bit + 1 < kDigitBits ? bit + 1 : kDigitBits;
                const int shift = bit + 1 - nb;
                const int nbins = 1 << nb;
                const uint32_t dmask = (uint32_t)nbins - 1u, above = mask_above(bit);
                for (int i = tid; i < nbins; i += kTopkThreads) hist[i] = 0u;
                __syncthreads();
#pragma unroll
                for (int j = 0; j < IPT; ++j)
                    if (c_begin + j < n_cand && (key[j] & above) == prefix)
                        atomicAdd(&hist[(key[j] >> shift) & dmask], 1u);
                __syncthreads();
                // bins in descending order; thread t owns `per` consecutive ones
                const int per = (nbins + kTopkThreads - 1) / kTopkThreads;
                uint32_t cnt[2] = {0u, 0u};
                uint32_t mine = 0u;
                for (int i = 0; i < per; ++i) {
                    const int rank = tid * per + i;
                    if (rank < nbins) cnt[i] = hist[nbins - 1 - rank];
                    mine += cnt[i];
                }
                uint32_t total;
                uint32_t run = block_exclusive_scan<kTopkThreads>(mine, scratch, &total);
                for (int i = 0; i < per; ++i) {
                    const int rank = tid * per + i;
                    if (rank < nbins && run < k_rem && run + cnt[i] >= k_rem) {
                        s_digit = (uint32_t)(nbins - 1 - rank);
                        s_krem = k_rem - run;
                    }
                    run += cnt[i];
                }
                __syncthreads();
                prefix |= s_digit << shift;
                k_rem = s_krem;
                bit -= nb;
                __syncthreads();
            }
        }
        thr = prefix;
    }

    // ordered compaction of the selected candidates
    if (k_eff > 0) {
        uint32_t n_gt = 0u, n_eq = 0u;
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            if (c_begin + j >= n_cand) continue;
            if (take_all || key[j] > thr) ++n_gt;
            else if (key[j] == thr) ++n_eq;
        }
        uint32_t tot;
        const uint32_t base_gt = block_exclusive_scan<kTopkThreads>(n_gt, scratch, &tot);
        const uint32_t base_eq = block_exclusive_scan<kTopkThreads>(n_eq, scratch, &tot);
        uint32_t pos = base_gt + (base_eq < k_rem ? base_eq : k_rem);
        uint32_t eq_seen = base_eq;
#pragma unroll
        for (int j = 0; j < IPT; ++j) {
            const int c = c_begin + j;
            if (c >= n_cand) continue;
            bool take = take_all || key[j] > thr;
            if (!take && key[j] == thr) {
                take = eq_seen < k_rem;
                ++eq_seen;
            }
            if (take && pos < (uint32_t)k_eff) {  // pos < k_eff by construction; never write past it
                const int b = n_sink + c;
                vb[n_sink + pos] = b;
                vp[n_sink + pos] = block_to_page[b];
                ++pos;
            }
        }
    }
    for (int i = tid; i < n_sink; i += kTopkThreads) {
        vb[i] = i;
        vp[i] = block_to_page[i];
    }
    for (int i = tid; i < n_recent; i += kTopkThreads) {
        const int b = n_blocks - n_recent + i;
        vb[n_sink + k_eff + i] = b;
        vp[n_sink + k_eff + i] = block_to_page[b];
    }
}

template <int IPT>
hipError_t launch_ipt(const SelectPlan &p, const float *r32, const int32_t *b2p, int32_t *vb,
                      int32_t *vp, hipStream_t stream) {
    hipLaunchKernelGGL((topk_select_kernel<IPT>), dim3(p.n_sel), dim3(kTopkThreads), 0, stream, r32,
                       p.n_cand, p.k_eff, p.n_sink, p.n_recent, p.n_blocks, p.n_view, b2p, vb, vp);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_topk(const SelectPlan &p, const float *r32, const int32_t *b2p, int32_t *vb,
                       int32_t *vp, hipStream_t stream) {
    const int need = (p.n_cand + kTopkThreads - 1) / kTopkThreads;
    if (need <= 1) return launch_ipt<1>(p, r32, b2p, vb, vp, stream);
    if (need <= 2) return launch_ipt<2>(p, r32, b2p, vb, vp, stream);
    if (need <= 4) return launch_ipt<4>(p, r32, b2p, vb, vp, stream);
    if (need <= 8) return launch_ipt<8>(p, r32, b2p, vb, vp, stream);
    if (need <= 16) return launch_ipt<16>(p, r32, b2p, vb, vp, stream);
    if (need <= 32) return launch_ipt<32>(p, r32, b2p, vb, vp, stream);
    if (need <= 64) return launch_ipt<64>(p, r32, b2p, vb, vp, stream);
    return hipErrorInvalidValue;
}

}  // namespace kvmem
