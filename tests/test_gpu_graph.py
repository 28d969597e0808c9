"""Decode steps captured in a HIP graph (as bench.py replays them) give, on every
replay, exactly what the same steps give when launched eagerly: the library's
kernels clear their own scratch (no memset nodes), and each replay must match
bitwise, with eager work and synchronizations between the replays."""
import numpy as np
import pytest
import torch

from paper_2609_04852_amd import kvmem as K
from paper_2609_04852_amd import workload as W
from paper_2609_04852_amd.step import LayerState
from parity import log

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    K.lib()
    yield
    torch.cuda.synchronize()


def snapshot(st):
    return [t.cpu().numpy().copy() for t in (st.view_blocks, st.view_pages, st.out, st.lse)]


@pytest.mark.parametrize("name", ["64k", "1m_fp8"])
def test_graph_replays_match_eager(name):
    cfg = W.CONFIGS[name]
    log(f"[case] graph replay {name}")
    w = W.generate(cfg, cfg.seed, n_query_sets=3)
    st = LayerState(cfg, w.k_pool[0], w.v_pool[0], w.block_to_page)
    st.build_index()
    q = torch.from_numpy(np.ascontiguousarray(w.q[:, :1])).cuda()  # [sets][1][n_q][Hq][d]

    def step(i):
        st.select(q[i], with_scores=False)
        st.attend(q[i][0])

    eager = []
    for i in range(3):
        step(i)
        torch.cuda.synchronize()
        eager.append(snapshot(st))
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(0)
        step(1)  # the buffers end with set 1's results
    for rep in range(4):
        step(2)  # eager work between replays
        torch.cuda.synchronize()
        got = snapshot(st)
        for a, b in zip(got, eager[2]):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"eager step after replay {rep}"
        graph.replay()
        torch.cuda.synchronize()
        got = snapshot(st)
        for a, b in zip(got, eager[1]):
            assert np.array_equal(a.view(np.uint8), b.view(np.uint8)), f"replay {rep}"
