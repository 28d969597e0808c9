"""Working-set update at a recall point -- TEST INFRASTRUCTURE ONLY.

Part of the CPU oracle (only tests/, the smoke check and the benchmark's CPU
baseline use it; it never touches the HIP library).  Plain Python and numpy,
written from the paper's Sec. 4.4 "Retrieval-Aware Hierarchical Reuse":

  Eq. 11   R_t = W_t & W_{t-1} (retained), L_t = W_t - W_{t-1} (incoming),
           E_t = W_{t-1} - W_t (outgoing)
  Eq. 12   L_t^physical = W_t - G_{t-1}: the selected blocks not resident in
           the bounded GPU page pool, the only ones that need a stage-in

A GPU hit keeps its page.  Its V is valid as is; its K is valid only at the
position it was encoded for, so when the block's compact position moves, K is
re-encoded in place by the difference (a delta re-encoding), at most
`max_deltas` times between rebuilds from the position-independent raw K (the
paper bounds the number of in-place adjustments, Sec. 4.4).

Readings (the paper leaves them open):
  * view block i (view_blocks ascending) sits at compact position
    first_position + i * Bt;
  * the pages that receive L^physical are the pages holding no block of W_t,
    taken in clock order from a hand (pages hand, hand + 1, ... modulo P), one
    per incoming block in view order; the hand then moves past the last page
    taken.  A taken page's previous block leaves G (an eviction);
  * a hit whose page has had max_deltas delta re-encodings is rebuilt from raw
    K instead (its counter restarts at 0), as is every incoming block.
"""
import numpy as np


class WorkingSet:
    """Repository-view state of the execution pool (all replaced by update())."""

    def __init__(self, n_blocks: int, n_pages: int):
        self.n_blocks, self.n_pages = int(n_blocks), int(n_pages)
        self.block_page = np.full(n_blocks, -1, np.int64)       # G membership: page of each block
        self.block_last_step = np.full(n_blocks, -1, np.int64)  # last recall step selecting the block
        self.page_block = np.full(n_pages, -1, np.int64)
        self.page_pos = np.zeros(n_pages, np.int64)             # position the page's K is encoded at
        self.page_deltas = np.zeros(n_pages, np.int64)          # delta re-encodings since the last rebuild
        self.prev_step = -1                                     # step of the previous update
        self.n_prev = 0                                         # |W_{t-1}|
        self.hand = 0

    def update(self, step, view_blocks, first_position, block_tokens, max_deltas):
        """One recall point.  Returns a dict:
          exec_pages [n_view]          page of each view block
          counts                       [|W_t|, |R_t|, |L_t|, |E_t|, |L_phys|, n_delta, n_rebuild, n_evicted]
          build  list of (i, block, page, position): K rebuilt from raw K (and V copied)
          delta  list of (i, page, shift): K re-encoded in place by shift positions"""
        view = [int(b) for b in view_blocks]
        n = len(view)
        if n > self.n_pages:
            raise ValueError("the execution pool is smaller than the view")
        if any(b < 0 or b >= self.n_blocks for b in view) or any(view[i] >= view[i + 1] for i in range(n - 1)):
            raise ValueError("view blocks must be ascending block ids")
        pos = [int(first_position) + i * int(block_tokens) for i in range(n)]
        retained = sum(1 for b in view if self.block_last_step[b] == self.prev_step and self.prev_step >= 0)
        hits = [self.block_page[b] >= 0 for b in view]
        kept = set(int(self.block_page[b]) for b, h in zip(view, hits) if h)
        # pages for the misses, in clock order from the hand
        misses = [i for i in range(n) if not hits[i]]
        free = [(self.hand + j) % self.n_pages for j in range(self.n_pages)
                if (self.hand + j) % self.n_pages not in kept]
        taken = free[:len(misses)]
        exec_pages = [-1] * n
        build, delta = [], []
        evicted = 0
        for i, p in zip(misses, taken):
            old = int(self.page_block[p])
            if old >= 0:
                self.block_page[old] = -1
                evicted += 1
            b = view[i]
            self.page_block[p] = b
            self.block_page[b] = p
            self.page_pos[p] = pos[i]
            self.page_deltas[p] = 0
            exec_pages[i] = p
            build.append((i, b, p, pos[i]))
        for i in range(n):
            if not hits[i]:
                continue
            p = int(self.block_page[view[i]])
            exec_pages[i] = p
            shift = pos[i] - int(self.page_pos[p])
            if shift != 0:
                if self.page_deltas[p] < max_deltas:
                    delta.append((i, p, shift))
                    self.page_deltas[p] += 1
                else:
                    build.append((i, view[i], p, pos[i]))
                    self.page_deltas[p] = 0
                self.page_pos[p] = pos[i]
        if taken:
            self.hand = (taken[-1] + 1) % self.n_pages
        for b in view:
            self.block_last_step[b] = step
        counts = [n, retained, n - retained, self.n_prev - retained, len(misses), len(delta),
                  len(build) - len(misses), evicted]
        self.prev_step, self.n_prev = int(step), n
        build.sort()
        return {"exec_pages": np.array(exec_pages, np.int64), "counts": np.array(counts, np.int64),
                "build": build, "delta": delta}
