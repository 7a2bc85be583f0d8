"""GPU block selection vs the fp64 oracle: bit-exact mask outside the ambiguity band,
counts and lists consistent with the mask, and a valid selection everywhere."""
import functools
import math

import numpy as np
import pytest
import torch

from oracle import la_oracle as O
from paper_2605_31158_amd import la
from paper_2605_31158_amd.workloads import WORKLOADS, CONFIG_ORDER, make_inputs, make_clustered, make_spread
from helpers import say, tau32, to_gpu, check_list, check_selection

pytestmark = pytest.mark.gpu


def run_select(inp, block, tau=None, keep=None, n_text=0):
    g = to_gpu(inp)
    if keep is None:
        mask, counts, idx = la.select_blocks(g["q"], g["k"], block, tau, n_text=n_text)
    else:
        mask, counts, idx = la.select_blocks_topk(g["q"], g["k"], block, keep, n_text=n_text)
    torch.cuda.synchronize()
    return mask.cpu().numpy(), counts.cpu().numpy(), idx.cpu().numpy()


@pytest.mark.parametrize("name", CONFIG_ORDER + ["480p_long_dense"])
def test_select_named_workloads(name):
    wl = WORKLOADS[name]
    say(f"[select] {name} shape B={wl.B} H={wl.H} Lq={wl.Lq} Lk={wl.Lk} d={wl.d} block={wl.block} tau={wl.tau}")
    inp = make_inputs(wl)
    mask, counts, idx = run_select(inp, wl.block, tau=wl.tau)
    sel = O.select_blocks(inp["q"], inp["k"], wl.block, tau=tau32(wl.tau))
    check_selection(mask, sel)
    check_list(mask, counts, idx)
    say(f"[select] {name} ok: kept blocks {int(mask.sum())}, oracle {int(sel['mask'].sum())}, "
        f"differ {int((mask != sel['mask']).sum())} (all inside the band)")


EDGE = [
    # (B, H, Lq, Lk, d, block, n_text, tau, seed, kind)
    (1, 2, 64, 640, 64, 64, 0, 0.9, 1, "Lq = one block"),
    (2, 3, 100, 900, 128, 64, 0, 0.7, 2, "ragged q and k blocks"),
    (1, 2, 200, 1100, 64, 128, 0, 0.9, 3, "block 128 ragged"),
    (1, 2, 256, 256, 64, 64, 0, 0.9, 4, "M = 0"),
    (1, 2, 200, 330, 128, 64, 0, 0.5, 5, "chunk start inside a block"),
    (1, 2, 128, 4096, 64, 64, 70, 0.9, 6, "text tokens"),
    (1, 2, 128, 4096, 64, 64, 0, 1e-6, 7, "tau -> 0+"),
    (1, 2, 128, 4096, 64, 64, 0, 1.0, 8, "tau = 1"),
    (1, 2, 128, 4096, 64, 64, 0, 3.0, 9, "tau > 1"),
    (1, 1, 64, 64 * 4097, 64, 64, 0, 0.95, 10, "M = 4096 (largest)"),
    (1, 4, 300, 64 * 700, 128, 64, 0, 0.99, 11, "M = 695, peaky"),
]


# Row widths on both sides of every per-lane size of the row kernel (4, 8, 12, 16, 20, 25, 32, 48
# and 64 candidates per lane), under both rules.
ROW_WIDTHS = [256, 257, 512, 513, 768, 769, 1024, 1025, 1280, 1281, 1600, 1601, 2048, 2049, 3072, 3073]


@functools.lru_cache(maxsize=2)
def _width_inputs(M):
    Lq, block = 128, 64
    return make_clustered(1, 2, Lq, Lq + block * M, 64, block, 40 + M % 97)


@pytest.mark.parametrize("rule", ["tau", "topk"])
@pytest.mark.parametrize("M", ROW_WIDTHS)
def test_select_every_row_width(M, rule):
    block = 64
    say(f"[select-width] M={M} rule={rule}")
    inp = _width_inputs(M)
    if rule == "tau":
        mask, counts, idx = run_select(inp, block, tau=0.9)
        sel = O.select_blocks(inp["q"], inp["k"], block, tau=tau32(0.9))
    else:
        keep = int(np.floor(0.175 * M + 1e-9))
        mask, counts, idx = run_select(inp, block, keep=keep)
        sel = O.select_blocks(inp["q"], inp["k"], block, topk_r=0.175)
    check_selection(mask, sel)
    check_list(mask, counts, idx)


@pytest.mark.parametrize("case", EDGE, ids=[c[-1] for c in EDGE])
def test_select_edge_shapes(case):
    B, H, Lq, Lk, d, block, n_text, tau, seed, kind = case
    say(f"[select-edge] {kind}: B={B} H={H} Lq={Lq} Lk={Lk} d={d} block={block} n_text={n_text} tau={tau}")
    inp = make_clustered(B, H, Lq, Lk, d, block, seed, n_text=n_text)
    mask, counts, idx = run_select(inp, block, tau=tau, n_text=n_text)
    sel = O.select_blocks(inp["q"], inp["k"], block, tau=tau32(tau), n_text=n_text)
    check_selection(mask, sel)
    check_list(mask, counts, idx)


def test_select_tied_scores():
    # duplicated key blocks give exactly tied scores: lower block index wins inside the band
    B, H, Lq, Lk, d, block = 1, 2, 128, 2048, 64, 64
    inp = make_clustered(B, H, Lq, Lk, d, block, 12)
    k = inp["k"].copy()
    k[:, :, 64 * 5:64 * 6] = k[:, :, 64 * 3:64 * 4]      # block 5 = block 3
    k[:, :, 64 * 9:64 * 10] = k[:, :, 64 * 3:64 * 4]     # block 9 = block 3
    inp["k"] = k
    for tau in (0.3, 0.9):
        mask, counts, idx = run_select(inp, block, tau=tau)
        sel = O.select_blocks(inp["q"], inp["k"], block, tau=tau32(tau))
        check_selection(mask, sel)
        check_list(mask, counts, idx)


@pytest.mark.parametrize("r", [0.0, 0.175, 0.5, 1.0])
def test_select_topk(r):
    # the paper's Top-floor(rM) rule, keep = floor(r * M) computed on the host
    B, H, Lq, Lk, d, block = 1, 4, 384, 64 * 160, 128, 64
    inp = make_clustered(B, H, Lq, Lk, d, block, 13)
    M = (Lk - Lq) // block
    keep = int(np.floor(r * M + 1e-9))
    say(f"[select-topk] r={r} M={M} keep={keep}")
    mask, counts, idx = run_select(inp, block, keep=keep)
    sel = O.select_blocks(inp["q"], inp["k"], block, topk_r=r)
    check_selection(mask, sel)
    check_list(mask, counts, idx)


def test_select_deterministic():
    wl = WORKLOADS["tiny"]
    inp = make_inputs(wl)
    a = run_select(inp, wl.block, tau=wl.tau)
    b = run_select(inp, wl.block, tau=wl.tau)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)


def test_mask_to_list_random():
    rng = np.random.default_rng(14)
    B, H, NQ, NK = 2, 3, 5, 37
    mask = (rng.uniform(size=(B, H, NQ, NK)) < 0.3).astype(np.uint8)
    mask[0, 0, 0] = 0
    mask[1, 2, 4] = 1
    counts, idx = la.mask_to_list(torch.from_numpy(mask).cuda(), 64, Lq=NQ * 64 - 10, Lk=NK * 64 - 5)
    torch.cuda.synchronize()
    check_list(mask, counts.cpu().numpy(), idx.cpu().numpy())


@pytest.mark.parametrize("tau", [0.05, 0.5, 0.93])
def test_select_all_scores_equal(tau):
    # every historical block is the same block: all M scores tie, the lowest indices are kept
    B, H, Lq, Lk, d, block = 1, 2, 128, 64 * 300, 64, 64
    inp = make_clustered(B, H, Lq, Lk, d, block, 15)
    k = inp["k"].copy()
    M = (Lk - Lq) // block
    for m in range(1, M):
        k[:, :, 64 * m:64 * (m + 1)] = k[:, :, 0:64]
    inp["k"] = k
    mask, counts, idx = run_select(inp, block, tau=tau)
    sel = O.select_blocks(inp["q"], inp["k"], block, tau=tau32(tau))
    check_selection(mask, sel)
    check_list(mask, counts, idx)
    # equal weights: the kernel keeps the smallest k with k / M >= tau (tau as the float it receives),
    # exactly, since its weights are integers; the oracle's fp64 prefix sums may differ from it by
    # one block only where tau * M is an integer (a crossing inside the band)
    from fractions import Fraction
    want = math.ceil(Fraction(float(np.float32(tau))) * M)
    assert (mask[..., :M].sum(-1) == want).all(), (mask[..., :M].sum(-1), want)
    for b in range(B):
        for h in range(H):
            for i in range(mask.shape[2]):
                n = int(mask[b, h, i, :M].sum())
                assert mask[b, h, i, :n].all(), "ties must keep the lowest block indices"


@pytest.mark.parametrize("name", ["tiny", "480p_window"])
def test_pooled_blocks_and_cached_key_means(name):
    # la_pool_blocks gives the block means the oracle defines (ragged last block included), and
    # selecting from cached key means reproduces la_select_blocks exactly
    wl = WORKLOADS[name]
    inp = make_inputs(wl)
    g = to_gpu(inp)
    shape = la.make_shape(wl.B, wl.H, wl.Lq, wl.Lk, wl.d, wl.block, wl.n_text, 0)
    qbar = la.pool_blocks(g["q"], wl.block, "q", shape)
    kbar = la.pool_blocks(g["k"], wl.block, "k", shape)
    mask_p, counts_p, idx_p = la.select_pooled(shape, qbar, kbar, tau=wl.tau)
    mask, counts, idx = la.select_blocks(g["q"], g["k"], wl.block, wl.tau, n_text=wl.n_text)
    torch.cuda.synchronize()
    assert torch.equal(mask_p, mask) and torch.equal(counts_p, counts)
    B, H = wl.B, min(wl.H, 2)
    qb_ref = O.pool_blocks(inp["q"][:, :H], wl.block)
    kb_ref = O.pool_blocks(inp["k"][:, :H], wl.block)
    np.testing.assert_allclose(qbar[:, :H].cpu().numpy(), qb_ref, rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(kbar[:, :H].cpu().numpy(), kb_ref, rtol=1e-5, atol=1e-5)


NEAR_ONE = [0.99999, 1 - 1e-6, 1 - 1e-7, float(np.nextafter(np.float32(1), np.float32(0)))]


@pytest.mark.parametrize("M", [700, 1560])
@pytest.mark.parametrize("tau", NEAR_ONE, ids=["0.99999", "1-1e-6", "1-1e-7", "largest-below-1"])
def test_select_tau_near_one_spread_rows(M, tau):
    # scores ~ N(0, 5^2) with no dominant block: a tau this close to 1 cuts hundreds of blocks
    # deep into a tail of masses down to ~1e-9 each, where the cutoff is decided by the dropped tail
    B, H, Lq, block, d = 1, 4, 256, 64, 128
    Lk = M * block + Lq
    inp = make_spread(B, H, Lq, Lk, d, block, seed=M, sigma=5.0)
    mask, counts, idx = run_select(inp, block, tau=tau)
    sel = O.select_blocks(inp["q"], inp["k"], block, tau=tau32(tau))
    kept = mask[..., :M].sum(-1)
    say(f"[select-near-1] M={M} tau={tau!r}: kept {kept.ravel().tolist()}, "
        f"oracle {sel['mask'][..., :M].sum(-1).ravel().tolist()}")
    assert kept.min() > 1 and kept.max() < M          # a real cut, deep in the tail
    check_selection(mask, sel)
    check_list(mask, counts, idx)


def test_select_without_mask_output():
    # mask = NULL: counts and lists alone, equal to those of the call that also writes the mask
    wl = WORKLOADS["480p_window"]
    inp = make_inputs(wl)
    g = to_gpu(inp)
    mask, counts, idx = la.select_blocks(g["q"], g["k"], wl.block, wl.tau)
    none, counts_n, idx_n = la.select_blocks(g["q"], g["k"], wl.block, wl.tau, want_mask=False)
    torch.cuda.synchronize()
    assert none is None
    assert torch.equal(counts_n, counts)
    c = counts.cpu().numpy()
    a, b = idx.cpu().numpy(), idx_n.cpu().numpy()
    for row in np.ndindex(c.shape):
        np.testing.assert_array_equal(b[row][:c[row]], a[row][:c[row]])
    check_list(mask.cpu().numpy(), c, b)
