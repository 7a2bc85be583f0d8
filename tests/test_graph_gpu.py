"""The whole path (select, plan, run, merge) captured in one HIP graph: every replay equals the
eager result bit for bit.  The calls record only kernel launches (no memset, copy, allocation or
synchronisation), so a caller can capture them; the replays alternate with eager work that
clears the outputs, as a serving loop would."""
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
