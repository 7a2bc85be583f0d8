"""Serving-style use of the library: the whole path (select, plan, run, merge; and the 3-D path)
captured in one HIP graph, where every replay equals the eager result bit for bit (the calls
record only kernel launches: no memset, copy, allocation or synchronisation; the replays
alternate with eager work that clears the outputs, as a serving loop would), and two problems in
flight at once on two streams, each equal to its sequential run (no shared state)."""
import numpy as np
import pytest
import torch

from paper_2605_31158_amd import la
from paper_2605_31158_amd.workloads import WORKLOADS, make_inputs, make_clustered
from helpers import say, to_gpu

pytestmark = pytest.mark.gpu


def bound_step(q, k, v, block, tau, mask, counts, idx, o, lse, ws):
    select = la.bind_select(q, k, block, tau, mask, counts, idx, ws)
    plan, run, merge = la.bind_attn_steps(q, k, v, counts, idx, block, o, ws, lse=lse)
    return select, plan, run, merge


CASES = [
    ("tiny", None),
    ("random b64", (1, 6, 1000, 5000, 128, 64, 0.9, 21)),
    ("random b128", (2, 3, 700, 4000, 64, 128, 0.8, 22)),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_step_graph_replays_equal_eager(case):
    label, spec = case
    if spec is None:
        wl = WORKLOADS["tiny"]
        inp = make_inputs(wl)
        block, tau = wl.block, wl.tau
    else:
        B, H, Lq, Lk, d, block, tau, seed = spec
        inp = make_clustered(B, H, Lq, Lk, d, block, seed)
    g = to_gpu(inp)
    q, k, v = g["q"], g["k"], g["v"]
    B, H, Lq, d = q.shape
    Lk = k.shape[2]
    NQ, NK = la.nblocks(Lq, block), la.nblocks(Lk, block)
    say(f"[graph] {label}: B={B} H={H} Lq={Lq} Lk={Lk} d={d} block={block} tau={tau}")
    shape = la.make_shape(B, H, Lq, Lk, d, block)
    ws = torch.empty(la.workspace_bytes(shape), dtype=torch.uint8, device="cuda")
    mask = torch.empty((B, H, NQ, NK), dtype=torch.uint8, device="cuda")
    counts = torch.empty((B, H, NQ), dtype=torch.int32, device="cuda")
    idx = torch.empty((B, H, NQ, NK), dtype=torch.int32, device="cuda")
    o = torch.empty_like(q)
    lse = torch.empty((B, H, Lq), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        steps = bound_step(q, k, v, block, tau, mask, counts, idx, o, lse, ws)
        for _ in range(2):
            for f in steps:
                f()
    s.synchronize()
    ref = [t.clone() for t in (mask, counts, o, lse)]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        for f in steps:
            f()
    s.synchronize()
    for r in range(4):
        with torch.cuda.stream(s):
            for t in (mask, counts, o, lse):
                t.zero_()
            graph.replay()
        s.synchronize()
        same = [torch.equal(a, b) for a, b in zip((mask, counts, o, lse), ref)]
        say(f"[graph] {label}: replay {r}: mask/counts/o/lse equal {same}")
        assert all(same)
    # eager calls after the replays still agree
    with torch.cuda.stream(s):
        o.zero_()
        for f in steps:
            f()
    s.synchronize()
    assert torch.equal(o, ref[2])


def test_3d_path_graph_replays_equal_eager():
    # the 3-D path: Q-Prep, KV-Prep, selection from the pooled means, plan, run, merge, Untile
    # Scatter, captured together (the tiny 3-D workload: text, ragged grid edges, padding slots)
    from paper_2605_31158_amd.workloads import WORKLOADS_3D, make_inputs_3d
    wl = WORKLOADS_3D["tiny_3d"]
    inp = make_inputs_3d(wl)
    g = to_gpu(inp)
    grid = la.grid3d(wl.B, wl.H, wl.d, wl.n_text, wl.T_ctx, wl.T_q, wl.Hs, wl.Ws, wl.bt, wl.bh, wl.bw, wl.block)
    shape = la.grid3d_shape(grid)
    kvalid = torch.from_numpy(la.grid3d_valid(grid)[1]).cuda()
    B, H, d, blk = wl.B, wl.H, wl.d, wl.block
    NQ, NK = shape.Lq // blk, shape.Lk // blk
    say(f"[graph] 3-D tiny: NQ={NQ} NK={NK}")
    dev = "cuda"
    q_t = torch.empty((B, H, shape.Lq, d), dtype=torch.bfloat16, device=dev)
    k_t = torch.empty((B, H, shape.Lk, d), dtype=torch.bfloat16, device=dev)
    v_t = torch.empty_like(k_t)
    qbar = torch.empty((B, H, NQ, d), dtype=torch.float32, device=dev)
    kbar = torch.empty((B, H, NK, d), dtype=torch.float32, device=dev)
    mask = torch.empty((B, H, NQ, NK), dtype=torch.uint8, device=dev)
    counts = torch.empty((B, H, NQ), dtype=torch.int32, device=dev)
    idx = torch.empty((B, H, NQ, NK), dtype=torch.int32, device=dev)
    o_t = torch.empty_like(q_t)
    lse_t = torch.empty((B, H, shape.Lq), dtype=torch.float32, device=dev)
    o = torch.empty_like(g["q"])
    lse = torch.empty((B, H, g["q"].shape[2]), dtype=torch.float32, device=dev)
    ws = torch.empty(la.workspace_bytes(shape), dtype=torch.uint8, device=dev)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        steps = la.bind_3d(grid, g["q"], g["k"], g["v"], q_t, k_t, v_t, qbar, kbar, mask, counts, idx, kvalid, o_t,
                           lse_t, o, lse, ws, tau=wl.tau)
        for _ in range(2):
            for f in steps:
                f()
    s.synchronize()
    ref = [t.clone() for t in (mask, o, lse)]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        for f in steps:
            f()
    s.synchronize()
    for r in range(3):
        with torch.cuda.stream(s):
            for t in (mask, o, lse, o_t, q_t):
                t.zero_()
            graph.replay()
        s.synchronize()
        same = [torch.equal(a, b) for a, b in zip((mask, o, lse), ref)]
        say(f"[graph] 3-D tiny: replay {r}: mask/o/lse equal {same}")
        assert all(same)


def test_two_streams_concurrently_equal_sequential():
    # two different problems in flight at once on two streams (default priority), each with its
    # own workspace: the library keeps no shared state, so each result equals its sequential run
    probs = []
    for spec in ((1, 4, 900, 4000, 128, 64, 0.9, 31), (2, 3, 600, 3000, 64, 128, 0.85, 32)):
        B, H, Lq, Lk, d, block, tau, seed = spec
        inp = make_clustered(B, H, Lq, Lk, d, block, seed)
        g = to_gpu(inp)
        NQ, NK = la.nblocks(Lq, block), la.nblocks(Lk, block)
        shape = la.make_shape(B, H, Lq, Lk, d, block)
        bufs = dict(ws=torch.empty(la.workspace_bytes(shape), dtype=torch.uint8, device="cuda"),
                    mask=torch.empty((B, H, NQ, NK), dtype=torch.uint8, device="cuda"),
                    counts=torch.empty((B, H, NQ), dtype=torch.int32, device="cuda"),
                    idx=torch.empty((B, H, NQ, NK), dtype=torch.int32, device="cuda"),
                    o=torch.empty_like(g["q"]),
                    lse=torch.empty((B, H, Lq), dtype=torch.float32, device="cuda"))
        probs.append((g, block, tau, bufs, torch.cuda.Stream()))
    steps = []
    for g, block, tau, b, s in probs:
        with torch.cuda.stream(s):
            steps.append(bound_step(g["q"], g["k"], g["v"], block, tau, b["mask"], b["counts"], b["idx"], b["o"],
                                    b["lse"], b["ws"]))
    refs = []
    for (g, block, tau, b, s), st in zip(probs, steps):      # one after the other
        with torch.cuda.stream(s):
            for f in st:
                f()
        s.synchronize()
        refs.append((b["mask"].clone(), b["o"].clone(), b["lse"].clone()))
    for rep in range(3):                                      # both in flight, interleaved launches
        for (g, block, tau, b, s) in probs:
            with torch.cuda.stream(s):
                b["o"].zero_()
                b["mask"].zero_()
        torch.cuda.synchronize()
        for j in range(4):
            for st in steps:
                st[j]()
        torch.cuda.synchronize()
        for (g, block, tau, b, s), (rm, ro, rl) in zip(probs, refs):
            assert torch.equal(b["mask"], rm) and torch.equal(b["o"], ro) and torch.equal(b["lse"], rl)
    say("[streams] two problems in flight on two streams: equal to their sequential runs")
