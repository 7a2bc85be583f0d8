"""GPU block-sparse attention vs the fp64 oracle evaluated on the GPU's own block mask.

Bar: max-abs <= 2e-2 and mean-abs <= 2e-3 on the bf16 output; lse within 1e-3.
"""
import math

import numpy as np
import pytest
import torch

from oracle import la_oracle as O
from paper_2605_31158_amd import la
from paper_2605_31158_amd.workloads import WORKLOADS, CONFIG_ORDER, make_inputs, make_clustered
from helpers import (say, tau32, to_gpu, check_list, check_selection, check_schedule, assert_attn_close,
                     bf16_tensor_to_f64)

pytestmark = pytest.mark.gpu

LSE_TOL = 1e-3


def gpu_attn_on_mask(inp, mask_np, block, frame_tokens=0, n_text=0, scale=None):
    g = to_gpu(inp)
    B, H, Lq, d = inp["q"].shape
    Lk = inp["k"].shape[2]
    counts, idx = la.mask_to_list(torch.from_numpy(np.ascontiguousarray(mask_np)).cuda(), block, Lq, Lk, d)
    o, lse = la.sparse_attn_fwd(g["q"], g["k"], g["v"], counts, idx, block, scale=scale, n_text=n_text,
                                frame_tokens=frame_tokens, want_lse=True)
    torch.cuda.synchronize()
    return bf16_tensor_to_f64(o), lse.cpu().numpy().astype(np.float64)


def row_tiles_1d(mask, block, Lk):
    """64-key tiles of each query block's own list (a key block has ceil(valid keys / 64)):
    [B*H, NQ]."""
    B, H, NQ, NK = mask.shape
    st = np.array([-(-min(block, Lk - j * block) // 64) for j in range(NK)], np.int64)
    return mask.reshape(B * H, NQ, NK).astype(np.int64) @ st


def compare(o, lse, o_ref, lse_ref, what):
    mx, mean = assert_attn_close(o, o_ref, what)
    fin = np.isfinite(lse_ref)
    assert (np.isneginf(lse[~fin])).all(), what
    if fin.any():
        assert np.abs(lse[fin] - lse_ref[fin]).max() <= LSE_TOL, what
    say(f"[attn] {what}: max-abs {mx:.2e} mean-abs {mean:.2e}")


SMALL = [
    # B, H, Lq, Lk, d, block, seed, F, density, label
    (1, 2, 256, 1024, 64, 64, 0, 0, 0.4, "d64 b64 aligned"),
    (2, 3, 300, 1000, 128, 64, 1, 0, 0.4, "d128 b64 ragged q/k"),
    (1, 2, 200, 1100, 128, 128, 2, 0, 0.5, "d128 b128 ragged"),
    (1, 2, 130, 777, 64, 128, 3, 0, 0.5, "d64 b128 ragged"),
    (1, 2, 400, 1400, 128, 128, 4, 100, 0.6, "frame-causal F=100"),
    (1, 1, 330, 990, 128, 64, 5, 110, 0.7, "frame-causal F=110 b64"),
    (1, 4, 64, 64 * 40, 128, 64, 6, 0, 1.0, "dense one query block"),
]


@pytest.mark.parametrize("case", SMALL, ids=[c[-1] for c in SMALL])
def test_attn_random_masks(case):
    B, H, Lq, Lk, d, block, seed, F, density, label = case
    say(f"[attn] {label}: B={B} H={H} Lq={Lq} Lk={Lk} d={d} block={block} F={F}")
    inp = make_clustered(B, H, Lq, Lk, d, block, seed)
    rng = np.random.default_rng(seed)
    NQ, NK = -(-Lq // block), -(-Lk // block)
    mask = (rng.uniform(size=(B, H, NQ, NK)) < density).astype(np.uint8)
    mask[..., -1] = 1                       # the ragged chunk tail is always in play
    o, lse = gpu_attn_on_mask(inp, mask, block, frame_tokens=F)
    o_ref, lse_ref = O.attention(inp["q"], inp["k"], inp["v"], mask, block, frame_tokens=F)
    compare(o, lse, o_ref, lse_ref, label)


def test_attn_empty_rows_and_custom_scale():
    inp = make_clustered(1, 2, 256, 1024, 64, 64, 7)
    mask = np.zeros((1, 2, 4, 16), np.uint8)
    mask[0, 0, 1, [2, 5]] = 1
    mask[0, 1, 3, :] = 1
    o, lse = gpu_attn_on_mask(inp, mask, 64, scale=0.05)
    o_ref, lse_ref = O.attention(inp["q"], inp["k"], inp["v"], mask, 64, scale=0.05)
    compare(o, lse, o_ref, lse_ref, "empty rows, scale 0.05")
    assert (o[0, 0, :64] == 0).all() and np.isneginf(lse[0, 0, :64]).all()


def test_attn_list_is_a_set():
    # the attention pass uses the set of listed blocks: shuffled order, repeats, entries
    # outside [0, NK) and counts beyond NK must give the same result as the clean list
    B, H, Lq, Lk, d, block = 1, 3, 300, 1300, 128, 64
    inp = make_clustered(B, H, Lq, Lk, d, block, 11)
    rng = np.random.default_rng(11)
    NQ, NK = -(-Lq // block), -(-Lk // block)
    mask = (rng.uniform(size=(B, H, NQ, NK)) < 0.45).astype(np.uint8)
    counts = np.zeros((B, H, NQ), np.int32)
    idx = np.full((B, H, NQ, NK), -7, np.int32)
    for h in range(H):
        for i in range(NQ):
            kept = np.nonzero(mask[0, h, i])[0]
            junk = [NK, NK + 5, -1]
            lst = list(kept) + list(rng.choice(kept, size=min(3, len(kept)))) + junk if len(kept) else junk
            lst = list(rng.permutation(lst))[:NK]
            counts[0, h, i] = len(lst)
            idx[0, h, i, :len(lst)] = lst
    counts[0, 1, 0] = NK + 100          # beyond NK: clamped, the rest of the row is -7 (ignored)
    idx[0, 1, 0, :] = -7
    kept = np.nonzero(mask[0, 1, 0])[0]
    idx[0, 1, 0, :len(kept)] = kept[::-1]
    g = to_gpu(inp)
    o, lse = la.sparse_attn_fwd(g["q"], g["k"], g["v"], torch.from_numpy(counts).cuda(),
                                torch.from_numpy(idx).cuda(), block, want_lse=True)
    torch.cuda.synchronize()
    o_ref, lse_ref = O.attention(inp["q"], inp["k"], inp["v"], mask, block)
    compare(bf16_tensor_to_f64(o), lse.cpu().numpy().astype(np.float64), o_ref, lse_ref, "list as a set")


def test_attn_value_invariants():
    # V = 1 gives O = 1 exactly representable; one-hot V gives rows of weights summing to 1
    inp = make_clustered(1, 1, 128, 512, 64, 64, 8, v_kind="ones")
    mask = np.ones((1, 1, 2, 8), np.uint8)
    mask[0, 0, 0, 1] = 0
    o, _ = gpu_attn_on_mask(inp, mask, 64)
    assert np.abs(o - 1.0).max() <= 2 ** -8


@pytest.mark.parametrize("name", CONFIG_ORDER + ["480p_long_dense"])
def test_attn_named_workloads_on_gpu_mask(name):
    # sampled query blocks (the heaviest rows, random rows, the ragged last block) and, except for
    # the dense run (5.4 TFLOP), every query block of one head
    wl = WORKLOADS[name]
    say(f"[attn] {name}: full size, sampled query blocks vs oracle on the GPU mask")
    inp = make_inputs(wl)
    g = to_gpu(inp)
    mask, counts, idx = la.select_blocks(g["q"], g["k"], wl.block, wl.tau)
    shape = la.make_shape(wl.B, wl.H, wl.Lq, wl.Lk, wl.d, wl.block)
    ws = torch.empty(la.workspace_bytes(shape), dtype=torch.uint8, device="cuda")
    o, lse = la.sparse_attn_fwd(g["q"], g["k"], g["v"], counts, idx, wl.block, want_lse=True, ws=ws)
    torch.cuda.synchronize()
    mask_np = mask.cpu().numpy()
    check_list(mask_np, counts.cpu().numpy(), idx.cpu().numpy())
    info = check_schedule(la.plan_schedule(shape, ws), row_tiles=row_tiles_1d(mask_np, wl.block, wl.Lk))
    say(f"[attn] {name}: schedule {info}")
    o = bf16_tensor_to_f64(o)
    lse = lse.cpu().numpy()
    B, H, NQ = wl.B, wl.H, wl.nq
    rng = np.random.default_rng(100)
    heavy = np.argsort(-mask_np.sum(-1).ravel())[:3]
    rows = set()
    for flat in list(heavy) + list(rng.integers(0, B * H * NQ, size=8)) + [NQ - 1, B * H * NQ - 1]:
        b, rem = divmod(int(flat), H * NQ)
        h, i = divmod(rem, NQ)
        rows.add((b, h, i))
    if name != "480p_long_dense":
        b, rem = divmod(int(heavy[0]), H * NQ)
        rows.update((b, rem // NQ, i) for i in range(NQ))
    ref = O.attention_rows(inp["q"], inp["k"], inp["v"], mask_np, wl.block, sorted(rows))
    for (b, h, i), (ob, lb) in ref.items():
        lo = i * wl.block
        compare(o[b, h, lo:lo + ob.shape[0]], lse[b, h, lo:lo + ob.shape[0]], ob, lb,
                f"{name} row (b={b}, h={h}, i={i}) kept={int(mask_np[b, h, i].sum())}")


def test_attn_tiny_full_and_causal_720p_sample():
    wl = WORKLOADS["tiny"]
    inp = make_inputs(wl)
    g = to_gpu(inp)
    mask, counts, idx = la.select_blocks(g["q"], g["k"], wl.block, wl.tau)
    o, lse = la.sparse_attn_fwd(g["q"], g["k"], g["v"], counts, idx, wl.block, want_lse=True)
    torch.cuda.synchronize()
    o_ref, lse_ref = O.attention(inp["q"], inp["k"], inp["v"], mask.cpu().numpy(), wl.block)
    compare(bf16_tensor_to_f64(o), lse.cpu().numpy(), o_ref, lse_ref, "tiny full")
    # 720P with the frame-causal mask inside the chunk, sampled rows
    wl = WORKLOADS["720p_causal"]
    inp = make_inputs(wl)
    g = to_gpu(inp)
    mask, counts, idx = la.select_blocks(g["q"], g["k"], wl.block, wl.tau)
    o, lse = la.sparse_attn_fwd(g["q"], g["k"], g["v"], counts, idx, wl.block, frame_tokens=wl.frame_tokens,
                                want_lse=True)
    torch.cuda.synchronize()
    mask_np = mask.cpu().numpy()
    o = bf16_tensor_to_f64(o)
    lse = lse.cpu().numpy()
    rows = [(0, 0, 0), (0, 3, 27), (0, 5, 28), (0, 11, 56), (0, 23, 112), (0, 17, 84)]
    ref = O.attention_rows(inp["q"], inp["k"], inp["v"], mask_np, wl.block, rows, frame_tokens=wl.frame_tokens)
    for (b, h, i), (ob, lb) in ref.items():
        lo = i * wl.block
        compare(o[b, h, lo:lo + ob.shape[0]], lse[b, h, lo:lo + ob.shape[0]], ob, lb, f"720p causal row {i}")


def test_attn_deterministic_and_split_consistent():
    # the tiny problem runs split over the key range; results are bitwise repeatable
    wl = WORKLOADS["tiny"]
    inp = make_inputs(wl)
    g = to_gpu(inp)
    mask, counts, idx = la.select_blocks(g["q"], g["k"], wl.block, wl.tau)
    o1 = la.sparse_attn_fwd(g["q"], g["k"], g["v"], counts, idx, wl.block)
    o2 = la.sparse_attn_fwd(g["q"], g["k"], g["v"], counts, idx, wl.block)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2)


def test_attn_plan_run_merge_equal_fwd():
    # the three steps give bit-identical o and lse; one plan serves a second run with other q, v
    B, H, Lq, Lk, d, block = 1, 3, 700, 2100, 128, 64
    inp = make_clustered(B, H, Lq, Lk, d, block, 12)
    rng = np.random.default_rng(12)
    NQ, NK = -(-Lq // block), -(-Lk // block)
    mask = (rng.uniform(size=(B, H, NQ, NK)) < 0.4).astype(np.uint8)
    g = to_gpu(inp)
    counts, idx = la.mask_to_list(torch.from_numpy(mask).cuda(), block, Lq, Lk, d)
    o1, lse1 = la.sparse_attn_fwd(g["q"], g["k"], g["v"], counts, idx, block, want_lse=True)
    shape = la.make_shape(B, H, Lq, Lk, d, block)
    ws = torch.empty(la.workspace_bytes(shape), dtype=torch.uint8, device="cuda")
    o2 = torch.empty_like(g["q"])
    lse2 = torch.empty_like(lse1)
    plan, run, merge = la.bind_attn_steps(g["q"], g["k"], g["v"], counts, idx, block, o2, ws, lse=lse2)
    plan()
    run()
    merge()
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(lse1, lse2)
    q2 = (g["q"].float() * 0.5).to(torch.bfloat16)
    v2 = (g["v"].float() * -2.0).to(torch.bfloat16)
    o3 = la.sparse_attn_fwd(q2, g["k"], v2, counts, idx, block)
    run2, merge2 = la.bind_attn_steps(q2, g["k"], v2, counts, idx, block, o2, ws, lse=lse2)[1:]
    for _ in range(3):      # one plan serves any number of runs
        o2.zero_()
        run2()
        merge2()
        torch.cuda.synchronize()
        assert torch.equal(o3, o2)


def test_attn_head_with_more_than_1024_query_blocks():
    # NQ = 1030 query blocks in one head: past the planner's grouping limit, so the units take
    # the query blocks in their natural order; selection and attention on sampled rows
    B, H, d, block = 1, 1, 64, 64
    Lq = 1030 * block - 20                   # ragged last query block
    Lk = Lq + 12 * block
    inp = make_clustered(B, H, Lq, Lk, d, block, 31)
    g = to_gpu(inp)
    mask, counts, idx = la.select_blocks(g["q"], g["k"], block, 0.9)
    o, lse = la.sparse_attn_fwd(g["q"], g["k"], g["v"], counts, idx, block, want_lse=True)
    torch.cuda.synchronize()
    mask_np = mask.cpu().numpy()
    assert mask_np.shape[2] == 1030
    check_selection(mask_np, O.select_blocks(inp["q"], inp["k"], block, tau=tau32(0.9)))
    check_list(mask_np, counts.cpu().numpy(), idx.cpu().numpy())
    o = bf16_tensor_to_f64(o)
    lse = lse.cpu().numpy()
    rng = np.random.default_rng(31)
    rows = sorted({(0, 0, int(i)) for i in list(rng.integers(0, 1030, size=12)) + [0, 1, 3, 4, 1023, 1024, 1029]})
    ref = O.attention_rows(inp["q"], inp["k"], inp["v"], mask_np, block, rows)
    for (b, h, i), (ob, lb) in ref.items():
        lo = i * block
        compare(o[b, h, lo:lo + ob.shape[0]], lse[b, h, lo:lo + ob.shape[0]], ob, lb, f"NQ=1030 row {i}")


def test_attn_rounds_long_units_and_empty_units():
    # Enough units for two or more rounds of whole units on a 256-CU device (B*H = 640 units of
    # one 256-row query tile each), mostly short lists, some heads keeping every block (units
    # longer than the per-round share, which go to stream-K), some keeping nothing (one unowned
    # tile).  Compared with the oracle on a sample of heads that covers every kind.
    B, H, Lq, Lk, d, block = 2, 320, 256, 2048, 64, 64
    say(f"[attn] rounds: B={B} H={H} Lq={Lq} Lk={Lk} d={d} block={block}")
    inp = make_clustered(B, H, Lq, Lk, d, block, 11)
    rng = np.random.default_rng(11)
    NQ, NK = Lq // block, Lk // block
    mask = (rng.uniform(size=(B, H, NQ, NK)) < 0.2).astype(np.uint8)
    dense_heads = rng.choice(B * H, size=24, replace=False)
    empty_heads = rng.choice(np.setdiff1d(np.arange(B * H), dense_heads), size=24, replace=False)
    flat = mask.reshape(B * H, NQ, NK)
    flat[dense_heads] = 1
    flat[empty_heads] = 0
    o, lse = gpu_attn_on_mask(inp, mask, block)
    sample = np.concatenate([dense_heads[:6], empty_heads[:6],
                             rng.choice(np.setdiff1d(np.arange(B * H), np.r_[dense_heads, empty_heads]), 12,
                                        replace=False)])
    for bh in sample:
        b, h = divmod(int(bh), H)
        sl = {x: inp[x][b:b + 1, h:h + 1] for x in "qkv"}
        o_ref, lse_ref = O.attention(sl["q"], sl["k"], sl["v"], mask[b:b + 1, h:h + 1], block)
        compare(o[b:b + 1, h:h + 1], lse[b:b + 1, h:h + 1], o_ref, lse_ref, f"rounds head {bh}")


SCHED = [
    # B, H, Lq, Lk, d, block, density, dense heads, empty heads, label
    (2, 320, 256, 2048, 64, 64, 0.2, 24, 24, "two rounds, long and empty units"),
    (4, 128, 512, 3000, 64, 64, 0.1, 16, 8, "three rounds, ragged keys"),
    (1, 64, 1024, 4096, 64, 128, 0.25, 4, 4, "no rounds, block 128"),
    (1, 2, 300, 1000, 128, 64, 0.4, 0, 0, "few units"),
    (1, 1, 1030 * 64 - 20, 1030 * 64 + 700, 64, 64, 0.05, 0, 0, "one head past the grouping limit"),
]


@pytest.mark.parametrize("case", SCHED, ids=[c[-1] for c in SCHED])
def test_attn_schedule_invariants(case):
    # the plan's schedule follows the stated rule (whole units in XCD-major rounds, long units
    # demoted, shares within ceil(T / P) tiles per workgroup), read back from the workspace
    B, H, Lq, Lk, d, block, density, n_dense, n_empty, label = case
    say(f"[sched] {label}: B={B} H={H} Lq={Lq} Lk={Lk} d={d} block={block}")
    rng = np.random.default_rng(B * H + Lq)
    NQ, NK = -(-Lq // block), -(-Lk // block)
    mask = (rng.uniform(size=(B, H, NQ, NK)) < density).astype(np.uint8)
    flat = mask.reshape(B * H, NQ, NK)
    heads = rng.permutation(B * H)
    flat[heads[:n_dense]] = 1
    flat[heads[n_dense:n_dense + n_empty]] = 0
    gen = torch.Generator(device="cuda").manual_seed(7)
    q = torch.randn((B, H, Lq, d), device="cuda", generator=gen).to(torch.bfloat16)
    k = torch.randn((B, H, Lk, d), device="cuda", generator=gen).to(torch.bfloat16)
    v = torch.randn((B, H, Lk, d), device="cuda", generator=gen).to(torch.bfloat16)
    counts, idx = la.mask_to_list(torch.from_numpy(mask).cuda(), block, Lq, Lk, d)
    shape = la.make_shape(B, H, Lq, Lk, d, block)
    ws = torch.empty(la.workspace_bytes(shape), dtype=torch.uint8, device="cuda")
    la.sparse_attn_fwd(q, k, v, counts, idx, block, ws=ws)
    info = check_schedule(la.plan_schedule(shape, ws), row_tiles=row_tiles_1d(mask, block, Lk))
    say(f"[sched] {label}: {info}")
