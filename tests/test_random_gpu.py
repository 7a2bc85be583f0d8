"""Seeded random problems through the whole path against the fp64 oracle.

Each case draws a shape (head dim, block size, batch, heads, ragged query length, text
tokens, context length that need not be a whole number of blocks, frame-causal chunk or
not) and a selection rule (tau or Top-floor(rM)), runs the GPU selection, checks it against
the oracle's, then runs the GPU attention on the GPU's lists and compares every output row
with the oracle's attention on the same mask.  The cases are fixed by the seed below.
"""
import math

import numpy as np
import pytest
import torch

from oracle import la_oracle as O
from paper_2605_31158_amd import la
from paper_2605_31158_amd.workloads import make_clustered
from helpers import say, tau32, to_gpu, check_list, check_selection, assert_attn_close, bf16_tensor_to_f64

pytestmark = pytest.mark.gpu

LSE_TOL = 1e-3


def _draw_cases(n, seed):
    rng = np.random.default_rng(seed)
    cases = []
    for c in range(n):
        d = int(rng.choice([64, 128]))
        block = int(rng.choice([64, 128]))
        B = int(rng.integers(1, 3))
        H = int(rng.integers(1, 5))
        Lq = int(rng.integers(1, 4 * block + 1))
        n_text = int(rng.choice([0, 0, int(rng.integers(1, 2 * block + 1))]))
        L_ctx = int(rng.integers(0, 24 * block + 1))
        F = int(rng.choice([0, 0, int(rng.integers(8, 200))]))
        if rng.random() < 0.5:
            rule = ("tau", float(rng.uniform(0.3, 0.99)))
        else:
            rule = ("topk", float(rng.uniform(0.0, 1.0)))
        cases.append((c, B, H, Lq, n_text + L_ctx + Lq, d, block, n_text, F, rule, 1000 + c))
    return cases


CASES = _draw_cases(80, 20261202)


def _case_id(c):
    i, B, H, Lq, Lk, d, block, n_text, F, rule, _ = c
    return f"{i}-B{B}H{H}-q{Lq}-k{Lk}-d{d}-b{block}-t{n_text}-F{F}-{rule[0]}"


@pytest.mark.parametrize("case", CASES, ids=[_case_id(c) for c in CASES])
def test_random_path(case):
    i, B, H, Lq, Lk, d, block, n_text, F, (rule, r), seed = case
    say(f"[random] {_case_id(case)} rule value {r:.3f}")
    inp = make_clustered(B, H, Lq, Lk, d, block, seed, n_text=n_text)
    g = to_gpu(inp)
    h0 = -(-n_text // block)
    M = max((Lk - Lq) // block - h0, 0)
    if rule == "tau":
        mask, counts, idx = la.select_blocks(g["q"], g["k"], block, r, n_text=n_text)
        sel = O.select_blocks(inp["q"], inp["k"], block, tau=tau32(r), n_text=n_text)
    else:
        keep = int(math.floor(r * M + 1e-9)) if M > 0 else 0
        mask, counts, idx = la.select_blocks_topk(g["q"], g["k"], block, keep, n_text=n_text)
        sel = O.select_blocks(inp["q"], inp["k"], block, topk_r=r, n_text=n_text)
    o, lse = la.sparse_attn_fwd(g["q"], g["k"], g["v"], counts, idx, block, n_text=n_text, frame_tokens=F,
                                want_lse=True)
    torch.cuda.synchronize()
    mask_np = mask.cpu().numpy()
    check_selection(mask_np, sel)
    check_list(mask_np, counts.cpu().numpy(), idx.cpu().numpy())
    o_ref, lse_ref = O.attention(inp["q"], inp["k"], inp["v"], mask_np, block, frame_tokens=F)
    o_gpu = bf16_tensor_to_f64(o)
    lse_gpu = lse.cpu().numpy().astype(np.float64)
    mx, mean = assert_attn_close(o_gpu, o_ref, _case_id(case))
    fin = np.isfinite(lse_ref)
    assert np.isneginf(lse_gpu[~fin]).all()
    assert np.abs(lse_gpu[fin] - lse_ref[fin]).max() <= LSE_TOL
    say(f"[random] M={M} kept {int(mask_np.sum())} of {mask_np.size}: max-abs {mx:.2e} mean-abs {mean:.2e}")
