// Working-set update at a recall point (Sec. 4.4 "Retrieval-Aware Hierarchical
// Reuse", Eq. 11 and Eq. 12) over a bounded execution page pool.
//
// The repository view of the pool lives in caller-owned device arrays: the page
// of each resident block (G), the step that last selected each block (W of the
// previous recall), and per page its block, the position its K is encoded at and
// the number of in-place delta re-encodings since K was last built from raw K.
// One update, all on the stream with no host round trip:
//
//   ws_clear     zero the page marks
//   ws_classify  per view block: GPU hit or miss (Eq. 12), retained or not
//                (Eq. 11); a hit marks its page kept and is sorted into
//                "unchanged", "delta" (its compact position moved and its page
//                has had fewer than max_deltas delta steps) or "rebuild"
//   ws_assign    one workgroup: prefix sums give each view block its rank in
//                its category; the pages holding no selected block are taken in
//                clock order from the hand, one per miss in view order; the
//                counts and the header (previous step, |W|, hand) are written
//   ws_apply     per view block: misses take their page (evicting its previous
//                block from G), every page's position and delta counter are
//                updated, and the build list (misses and rebuilds: raw K
//                re-encoded, V copied) and the delta list are filled
//
// The build and delta lists then run through the re-encoding kernels of
// rope.hip, whose grids are sized for the whole view and stop at the lists'
// device-side lengths.
#include "kvmem_device.h"
#include "kvmem_internal.h"

namespace kvmem {
namespace {

constexpr int kWsThreads = 256;
constexpr int kAssignThreads = 1024;

enum : int32_t { kUnchanged = 0, kDelta = 1, kRebuild = 2, kLoad = 3, kInvalid = 4 };

__global__ __launch_bounds__(kWsThreads) void ws_reset_kernel(WorkingSetState s) {
    const int64_t n = (int64_t)(s.n_blocks > s.n_pages ? s.n_blocks : s.n_pages);
    for (int64_t i = (int64_t)blockIdx.x * kWsThreads + threadIdx.x; i < n; i += (int64_t)gridDim.x * kWsThreads) {
        if (i < s.n_blocks) {
            s.block_page[i] = -1;
            s.block_last_step[i] = -1;
        }
        if (i < s.n_pages) {
            s.page_block[i] = -1;
            s.page_pos[i] = 0;
            s.page_deltas[i] = 0;
        }
        if (i < kWsHeaderWords) s.header[i] = i == 0 ? -1 : 0;  // no previous step, |W| = 0, hand 0
    }
}

__global__ __launch_bounds__(kWsThreads) void ws_clear_kernel(int32_t *__restrict__ kept, int n_pages) {
    for (int i = blockIdx.x * kWsThreads + threadIdx.x; i < n_pages; i += gridDim.x * kWsThreads) kept[i] = 0;
}

__global__ __launch_bounds__(kWsThreads) void ws_classify_kernel(WorkingSetState s, const int32_t *__restrict__ view,
                                                                 int n_view, int64_t first_pos, int block_tokens,
                                                                 int max_deltas, WsScratch w) {
    const int i = blockIdx.x * kWsThreads + threadIdx.x;
    if (i >= n_view) return;
    const int32_t b = view[i];
    int32_t kind = kInvalid, ret = 0;
    if (b >= 0 && b < s.n_blocks) {
        const int32_t prev = s.header[0];
        ret = prev >= 0 && s.block_last_step[b] == prev;
        const int32_t p = s.block_page[b];
        if (p >= 0 && p < s.n_pages) {
            w.kept[p] = 1;
            const int64_t shift = first_pos + (int64_t)i * block_tokens - s.page_pos[p];
            kind = shift == 0 ? kUnchanged : (s.page_deltas[p] < max_deltas ? kDelta : kRebuild);
        } else {
            kind = kLoad;
        }
    }
    w.kind[i] = kind;
    w.retained[i] = ret;
}

// Exclusive scan of `flag` over the view by the one workgroup; returns the total.
template <int NT>
__device__ int32_t scan_view(const int32_t *kind, int n_view, int32_t want, int32_t *rank, uint32_t *sc) {
    int32_t base = 0;
    for (int c0 = 0; c0 < n_view; c0 += NT) {
        const int i = c0 + (int)threadIdx.x;
        const uint32_t f = i < n_view && kind[i] == want;
        uint32_t tot;
        const uint32_t ex = block_exclusive_scan<NT>(f, sc, &tot);
        if (f) rank[i] = base + (int32_t)ex;
        base += (int32_t)tot;
    }
    return base;
}

__global__ __launch_bounds__(kAssignThreads) void ws_assign_kernel(WorkingSetState s, int n_view, int step,
                                                                   WsScratch w, int32_t *__restrict__ counts) {
    constexpr int NT = kAssignThreads;
    __shared__ uint32_t sc[NT / kWave + 1];
    __shared__ int32_t sm_evicted;
    const int tid = threadIdx.x;
    // ranks inside each category (view order)
    const int32_t n_load = scan_view<NT>(w.kind, n_view, kLoad, w.rank, sc);
    const int32_t n_delta = scan_view<NT>(w.kind, n_view, kDelta, w.rank, sc);
    const int32_t n_rebuild = scan_view<NT>(w.kind, n_view, kRebuild, w.rank, sc);
    const int32_t n_invalid = scan_view<NT>(w.kind, n_view, kInvalid, w.rank, sc);
    int32_t n_ret = 0;
    for (int c0 = 0; c0 < n_view; c0 += NT) {
        const int i = c0 + tid;
        uint32_t tot;
        block_exclusive_scan<NT>(i < n_view ? (uint32_t)w.retained[i] : 0u, sc, &tot);
        n_ret += (int32_t)tot;
    }
    // pages holding no selected block, in clock order from the hand
    const int P = s.n_pages;
    const int hand = s.header[2];
    if (tid == 0) sm_evicted = 0;
    __syncthreads();
    int32_t found = 0, evicted = 0;
    for (int c0 = 0; c0 < P && found < n_load; c0 += NT) {
        const int j = c0 + tid;
        const int p = j < P ? (hand + j) % P : 0;
        const uint32_t f = j < P && w.kept[p] == 0;
        uint32_t tot;
        const uint32_t ex = block_exclusive_scan<NT>(f, sc, &tot);
        if (f && found + (int32_t)ex < n_load) {
            w.taken[found + ex] = p;
            if (s.page_block[p] >= 0) evicted++;
        }
        found += (int32_t)tot;
    }
    if (evicted) atomicAdd(&sm_evicted, evicted);
    __syncthreads();
    if (tid == 0) {
        const int32_t n_prev = s.header[1];
        counts[0] = n_view - n_invalid;          // |W_t|
        counts[1] = n_ret;                       // |R_t|
        counts[2] = n_view - n_invalid - n_ret;  // |L_t|
        counts[3] = n_prev - n_ret;              // |E_t|
        counts[4] = n_load;                      // |L_t^physical|
        counts[5] = n_delta;                     // K re-encoded in place
        counts[6] = n_rebuild;                   // K rebuilt from raw K (delta bound reached)
        counts[7] = sm_evicted;                  // resident blocks that left the pool
        counts[8] = n_invalid;                   // view ids outside [0, M) (ignored)
        w.lists[0] = n_load + n_rebuild;         // build list length
        w.lists[1] = n_delta;                    // delta list length
        w.lists[2] = n_load;                     // rebuilds follow the loads in the build list
        s.header[0] = step;
        s.header[1] = n_view - n_invalid;
        if (n_load > 0) s.header[2] = (w.taken[n_load - 1] + 1) % P;
    }
}

__global__ __launch_bounds__(kWsThreads) void ws_apply_kernel(WorkingSetState s, const int32_t *__restrict__ view,
                                                              const int32_t *__restrict__ block_to_page, int n_view,
                                                              int64_t first_pos, int block_tokens, int step,
                                                              WsScratch w, int32_t *__restrict__ exec_pages) {
    const int i = blockIdx.x * kWsThreads + threadIdx.x;
    if (i >= n_view) return;
    const int32_t kind = w.kind[i];
    if (kind == kInvalid) {
        exec_pages[i] = -1;
        return;
    }
    const int32_t b = view[i];
    const int64_t pos = first_pos + (int64_t)i * block_tokens;
    int32_t p;
    if (kind == kLoad) {
        p = w.taken[w.rank[i]];
        const int32_t old = s.page_block[p];
        if (old >= 0 && old < s.n_blocks) s.block_page[old] = -1;  // not selected: no other thread touches it
        s.page_block[p] = b;
        s.block_page[b] = p;
    } else {
        p = s.block_page[b];
    }
    if (kind == kLoad || kind == kRebuild) {
        const int k = kind == kLoad ? w.rank[i] : w.lists[2] + w.rank[i];
        w.build_src[k] = block_to_page[b];
        w.build_dst[k] = p;
        w.build_pos[k] = pos;
        s.page_deltas[p] = 0;
    } else if (kind == kDelta) {
        const int k = w.rank[i];
        w.delta_page[k] = p;
        w.delta_shift[k] = pos - s.page_pos[p];
        s.page_deltas[p] += 1;
    }
    s.page_pos[p] = pos;
    s.block_last_step[b] = step;
    exec_pages[i] = p;
}

}  // namespace

hipError_t launch_ws_reset(const WorkingSetState &s, hipStream_t stream) {
    const int64_t n = s.n_blocks > s.n_pages ? s.n_blocks : s.n_pages;
    const int grid = (int)((n + kWsThreads - 1) / kWsThreads < 4096 ? (n + kWsThreads - 1) / kWsThreads : 4096);
    hipLaunchKernelGGL(ws_reset_kernel, dim3(grid > 0 ? grid : 1), dim3(kWsThreads), 0, stream, s);
    return hipGetLastError();
}

hipError_t launch_ws_update(const WorkingSetState &s, const WsScratch &w, int kv_dtype, int head_dim, int n_kv_heads,
                            int block_tokens, const RopeFreqs &fr, int step, const int32_t *view, int n_view,
                            int64_t first_pos, int max_deltas, const int32_t *block_to_page, const void *raw_k,
                            const void *v_src, int64_t n_src_pages, void *k_exec, void *v_exec,
                            int32_t *exec_pages, int32_t *counts, hipStream_t stream) {
    const int gp = (s.n_pages + kWsThreads - 1) / kWsThreads;
    hipLaunchKernelGGL(ws_clear_kernel, dim3(gp < 1024 ? gp : 1024), dim3(kWsThreads), 0, stream, w.kept, s.n_pages);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int gv = (n_view + kWsThreads - 1) / kWsThreads;
    if (n_view > 0) {
        hipLaunchKernelGGL(ws_classify_kernel, dim3(gv), dim3(kWsThreads), 0, stream, s, view, n_view, first_pos,
                           block_tokens, max_deltas, w);
        if ((e = hipGetLastError()) != hipSuccess) return e;
    }
    // an empty view still ends the previous working set (counts and header)
    hipLaunchKernelGGL(ws_assign_kernel, dim3(1), dim3(kAssignThreads), 0, stream, s, n_view, step, w, counts);
    if ((e = hipGetLastError()) != hipSuccess || n_view == 0) return e;
    hipLaunchKernelGGL(ws_apply_kernel, dim3(gv), dim3(kWsThreads), 0, stream, s, view, block_to_page, n_view,
                       first_pos, block_tokens, step, w, exec_pages);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    e = launch_materialize(kv_dtype, head_dim, n_kv_heads, block_tokens, fr, raw_k, v_src, n_src_pages, w.build_src,
                           w.build_pos, w.build_dst, n_view, k_exec, v_exec, s.n_pages, stream, w.lists);
    if (e != hipSuccess) return e;
    return launch_rope_delta(kv_dtype, head_dim, n_kv_heads, block_tokens, fr, k_exec, s.n_pages, w.delta_page,
                             w.delta_shift, n_view, stream, w.lists + 1);
}

}  // namespace kvmem
