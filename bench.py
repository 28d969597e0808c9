"""Benchmark of the KVMem decode step on one MI355X.

One step = kvmem_select (score every candidate block, top-k under the budget,
view tables) + kvmem_sparse_attn (split-K attention over the selected pages and
the recent window), for every layer of the workload.  Inputs are synthetic
(seeded generator), resident in HBM before timing starts, and the Mean-K index
is built (and timed) beforehand.  Steps rotate over several query sets so
consecutive steps select different views, as consecutive decode steps would.

Prints one JSON line.  `value` is decode steps/s; `roofline` covers the
dominant call (sparse attention) measured with HIP events on its stream;
`cpu_baseline` is the fp64 CPU oracle timed on a bounded sample.
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
PEAK_HBM_GBPS = 8000.0  # MI355X HBM3E
ATTN_SOURCES = ["paper_2609_04852_amd/csrc/attn.hip", "paper_2609_04852_amd/csrc/kvmem_device.h",
                "paper_2609_04852_amd/csrc/kvmem_internal.h"]
TRAFFIC_FILE = os.path.join(HERE, "profiles", "sparse_attn_1m_traffic.json")


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--config", default="1m", help="workload name (see workload.CONFIGS)")
    p.add_argument("--seed", type=int, default=None)
    p.add_argument("--query-sets", type=int, default=8)
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="time budget of the CPU-oracle baseline sample (0 disables it)")
    p.add_argument("--graph", action="store_true", help="replay the steps from a captured HIP graph")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run 5 device-to-device copies of MIB MiB (known bytes, for scaling "
                        "rocprofv3 FETCH_SIZE / WRITE_SIZE) and exit")
    return p.parse_args()


def copy_calibration(mib):
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": n * 4, "copies": 5}), flush=True)


def source_digest(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(HERE, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def algorithmic_bytes(cfg):
    """Bytes the method must move per layer-step (each read or written once)."""
    hkv, d, bt = cfg.n_kv_heads, cfg.head_dim, cfg.block_tokens
    n_sel = cfg.n_sel
    q = cfg.n_q * cfg.n_q_heads * d * 4
    index = cfg.n_candidates * hkv * d * 4
    kv = cfg.n_view * bt * hkv * d * cfg.elem_bytes * 2  # K and V of every view page, per KV head
    tables = n_sel * cfg.n_view * 4 * 2
    out = cfg.n_q * cfg.n_q_heads * (d + 1) * 4
    select = q + index + tables
    attn = q + kv + n_sel * cfg.n_view * 4 + out
    return select, attn


def cpu_oracle_baseline(w, seconds):
    """fp64 oracle on the same workload: relevance + selection + attention per step.
    FP8 pools are decoded by the oracle's decoder: for the index in chunks of
    blocks beforehand, and inside every timed step for the view's pages."""
    import oracle
    cfg = w.cfg
    mode = oracle.MEAN_ALL if cfg.mode == "mean_all" else oracle.MAX_GROUP
    fp8 = cfg.kv_dtype == "fp8"

    def index_of(pool):
        if not fp8:
            return oracle.mean_k(pool, w.block_to_page)
        rows = []
        for b0 in range(0, cfg.n_blocks, 4096):
            pages = w.block_to_page[b0:b0 + 4096]
            sub = oracle.decode_fp8(pool[pages], cfg.kv_scale)
            rows.append(oracle.mean_k(sub, np.arange(len(pages), dtype=np.int32)))
        return np.concatenate(rows, 0)

    def attend(q, kp, vp_pool, vp):
        if not fp8:
            return oracle.view_attention(q, kp, vp_pool, vp)
        pages, local = np.unique(vp, return_inverse=True)
        local = local.reshape(vp.shape).astype(np.int32)
        return oracle.view_attention(q, oracle.decode_fp8(kp[pages], cfg.kv_scale),
                                     oracle.decode_fp8(vp_pool[pages], cfg.kv_scale), local)

    index = [index_of(w.k_pool[l]) for l in range(len(w.k_pool))]
    n = 0
    t0 = time.perf_counter()
    while True:
        qs = w.q[n % w.q.shape[0]]
        for l in range(len(w.k_pool)):
            rel = oracle.block_relevance(qs[l:l + 1], index[l][None], cfg.sink_blocks, cfg.n_recent, mode)
            k = oracle.k_eff(cfg.budget_tokens, cfg.budget_tokens, cfg.block_tokens, cfg.n_blocks,
                             cfg.sink_blocks, cfg.n_recent)
            _, vp = oracle.select(rel, cfg.sink_blocks, cfg.n_recent, k, w.block_to_page)
            attend(qs[l], w.k_pool[l], w.v_pool[l], vp)
        n += 1
        el = time.perf_counter() - t0
        if el >= seconds or n >= 50:
            break
    return n, el, oracle.num_threads()


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): the "
              "KVMem decode step here has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_04852_amd import kvmem as K
    from paper_2609_04852_amd import workload as W
    from paper_2609_04852_amd.step import LayerState

    K.lib()  # fail loudly if the HIP library is not built
    cfg = W.CONFIGS[args.config]
    seed = cfg.seed if args.seed is None else args.seed
    print(f"[bench] generating {cfg.name} seed={seed}", file=sys.stderr, flush=True)
    t = time.perf_counter()
    w = W.generate(cfg, seed, n_query_sets=args.query_sets)
    print(f"[bench] generated in {time.perf_counter() - t:.1f}s; uploading", file=sys.stderr, flush=True)
    dev = torch.device("cuda", 0)
    layers = [LayerState(cfg, w.k_pool[l], w.v_pool[l], w.block_to_page, dev) for l in range(cfg.n_layers)]
    qdev = torch.from_numpy(w.q).to(dev)  # [sets][L][n_q][Hq][d]
    torch.cuda.synchronize()

    # Mean-K index build (off the per-step path), timed separately
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for st in layers:
        st.build_index()
    e0.record()
    for st in layers:
        st.build_index()
    e1.record()
    torch.cuda.synchronize()
    build_ms = e0.elapsed_time(e1)
    build_bytes = cfg.n_layers * (cfg.n_blocks * cfg.n_kv_heads * cfg.block_tokens * cfg.head_dim *
                                  cfg.elem_bytes + cfg.n_blocks * cfg.n_kv_heads * cfg.head_dim * 4)

    stream = torch.cuda.current_stream()
    n_sets = qdev.shape[0]

    def step(i, ev=None):
        qs = qdev[i % n_sets]
        for l, st in enumerate(layers):
            st.select(qs[l:l + 1], with_scores=False)
            if ev is not None:
                ev[0].record(stream)
            st.attend(qs[l])
            if ev is not None:
                ev[1].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()

    graph = None
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(n_sets):
                step(i)
        graph.replay()
        torch.cuda.synchronize()

    # attention-call events, one pair per (step, layer)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps * cfg.n_layers)] if graph is None else []
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    if graph is None:
        for i in range(args.steps):
            for l, st in enumerate(layers):
                qs = qdev[i % n_sets]
                st.select(qs[l:l + 1], with_scores=False)
                a, b = evs[i * cfg.n_layers + l]
                a.record(stream)
                st.attend(qs[l])
                b.record(stream)
    else:
        reps = max(1, args.steps // n_sets)
        for _ in range(reps):
            graph.replay()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    n_steps = args.steps if graph is None else max(1, args.steps // n_sets) * n_sets
    ms_per_step = (t1 - t0) * 1000.0 / n_steps

    sel_bytes, attn_bytes = algorithmic_bytes(cfg)
    step_bytes = cfg.n_layers * (sel_bytes + attn_bytes)
    roofline = None
    dist = None
    if evs:
        attn_all = np.array([a.elapsed_time(b) for a, b in evs])
        attn_ms = float(np.mean(attn_all))
        # one step = between the starts of consecutive first-layer attention calls
        starts = [evs[i * cfg.n_layers][0] for i in range(args.steps)]
        step_all = np.array([starts[i].elapsed_time(starts[i + 1]) for i in range(len(starts) - 1)])
        dist = {"step_ms_p10_p50_p90": [round(float(np.percentile(step_all, p)), 5) for p in (10, 50, 90)]
                if step_all.size else None,
                "attn_ms_p10_p50_p90": [round(float(np.percentile(attn_all, p)), 5) for p in (10, 50, 90)]}
        achieved = attn_bytes / (attn_ms * 1e-3) / 1e9
        traffic = None
        if os.path.exists(TRAFFIC_FILE):
            with open(TRAFFIC_FILE) as f:
                tr = json.load(f)
            if tr.get("source_digest") == source_digest(ATTN_SOURCES) and tr.get("config") == cfg.name:
                traffic = tr.get("hbm_bytes_per_launch")
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                    "frac": round(achieved / PEAK_HBM_GBPS, 4), "traffic": traffic,
                    "kernel": "kvmem_sparse_attn (split-K attention + attn_combine)",
                    "bytes_per_launch": attn_bytes, "avg_launch_ms": round(attn_ms, 5)}

    # position handling (Sec. 4.4, Sec. 5.3), on the last step's view of layer 0:
    # re-encode every view block's K at compact positions from the raw keys and
    # copy V (kvmem_materialize), move them all by one block (kvmem_rerope), and
    # build the index from RoPE-encoded keys (kvmem_build_index_rope).  Values do
    # not matter for the timing; the bytes are those of the whole view.
    st = layers[0]
    n_view = st.view_pages.shape[1]
    page_bytes = cfg.n_kv_heads * cfg.block_tokens * cfg.head_dim * cfg.elem_bytes
    kx = torch.empty((n_view,) + tuple(st.k_pool.shape[1:]), dtype=st.k_pool.dtype, device=dev)
    vx = torch.empty_like(kx)
    src = st.view_pages[0].contiguous()
    dst = torch.arange(n_view, dtype=torch.int32, device=dev)
    cpos = torch.arange(n_view, dtype=torch.int64, device=dev) * cfg.block_tokens
    shift = torch.full((n_view,), cfg.block_tokens, dtype=torch.int64, device=dev)
    rope_base = 1e6

    def timed(fn, reps=10):
        fn()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / reps

    fp8 = cfg.kv_dtype == "fp8"  # FP8 pools are not re-encoded (that would quantise K again)
    mat_ms = None if fp8 else timed(
        lambda: K.kvmem_materialize(st.geom, rope_base, st.k_pool, st.v_pool, src, cpos, dst, kx, vx))
    rer_ms = None if fp8 else timed(lambda: K.kvmem_rerope(st.geom, rope_base, kx, dst, shift))
    irope_ms = timed(lambda: K.kvmem_build_index_rope(st.geom, st.k_pool, st.block_to_page, 0, cfg.n_blocks,
                                                      st.index, rope_base), reps=3)
    st.build_index()  # restore the position-independent index
    torch.cuda.synchronize()
    mat_bytes = 4 * n_view * page_bytes  # read K and V, write K and V
    rer_bytes = 2 * n_view * page_bytes  # read and write K
    irope_bytes = build_bytes // cfg.n_layers
    def rate(ms, nbytes):
        if ms is None:
            return "not applicable to FP8 pools"
        return {"ms": round(ms, 4), "bytes": nbytes, "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
                "frac_of_peak": round(nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 4)}

    position = {"view_blocks": n_view,
                "materialize": rate(mat_ms, mat_bytes),
                "rerope": rate(rer_ms, rer_bytes),
                "index_from_encoded_keys": {"ms": round(irope_ms, 4), "bytes": irope_bytes,
                                            "GBps": round(irope_bytes / (irope_ms * 1e-3) / 1e9, 1)}}
    del kx, vx

    # attainable-bandwidth reference: a plain 2 GiB device-to-device copy
    # (2 GiB read + 2 GiB written per copy), timed with events
    src = torch.empty(1 << 29, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record()
    for _ in range(5):
        dst.copy_(src)
    c1.record()
    torch.cuda.synchronize()
    copy_ref = round(5 * 2 * src.numel() * 4 / (c0.elapsed_time(c1) * 1e-3) / 1e9, 1)
    del src, dst

    cpu = None
    if args.cpu_seconds > 0:
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        n, el, cores = cpu_oracle_baseline(w, args.cpu_seconds)
        cpu = {"value": round(n / el, 4), "unit": "steps/s", "cores": cores, "kind": "oracle",
               "sample": f"{n} full decode steps of the same workload (fp64 relevance, selection and "
                         f"attention for every layer; index built beforehand), {el:.1f}s"}

    gbps = step_bytes / (ms_per_step * 1e-3) / 1e9
    out = {
        "metric": "decode steps/s + achieved HBM GB/s (% peak) for score+top-k+sparse attn @1M-token history",
        "value": round(1000.0 / ms_per_step, 2),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": n_steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": cfg.description, "name": cfg.name, "history_tokens": cfg.history_tokens,
                   "layers": cfg.n_layers, "kv_heads": cfg.n_kv_heads, "q_heads": cfg.n_q_heads,
                   "head_dim": cfg.head_dim, "block_tokens": cfg.block_tokens, "kv_dtype": cfg.kv_dtype,
                   "top_k": cfg.top_k, "recent_tokens": cfg.recent_tokens,
                   "view_tokens": cfg.n_view * cfg.block_tokens, "query_tokens": cfg.n_q,
                   "selection": cfg.mode, "seed": seed, "query_sets": n_sets,
                   "hip_graph": graph is not None},
        "step_bytes": step_bytes,
        "step_GBps": round(gbps, 1),
        "step_frac_of_peak": round(gbps / PEAK_HBM_GBPS, 4),
        "index_build_GBps": round(build_bytes / (build_ms * 1e-3) / 1e9, 1),
        "timing_distribution": dist,
        "position_handling": position,
        "attainable_copy_GBps": copy_ref,
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
