"""la_select_blocks_noalloc: the selection with the library's own scratch array (no workspace
argument, nothing allocated by the call) against la_select_blocks with a workspace, through the
C ABI: identical masks, counts and lists (integer work, so bit for bit), on two calls in a row
whose second one is smaller, so the scratch still holds the larger first call's contents."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2605_31158_amd import la
from paper_2605_31158_amd.workloads import WORKLOADS, make_inputs, make_clustered
from helpers import say, to_gpu

pytestmark = pytest.mark.gpu


def _outputs(q, k, block, fill):
    B, H, Lq, _ = q.shape
    NQ, NK = la.nblocks(Lq, block), la.nblocks(k.shape[2], block)
    mask = torch.full((B, H, NQ, NK), fill, dtype=torch.uint8, device=q.device)
    counts = torch.full((B, H, NQ), -3, dtype=torch.int32, device=q.device)
    idx = torch.full((B, H, NQ, NK), -3, dtype=torch.int32, device=q.device)
    return mask, counts, idx


def _compare(inp, block, tau, n_text=0, what=""):
    g = to_gpu(inp)
    mask, counts, idx = la.select_blocks(g["q"], g["k"], block, tau, n_text=n_text)
    m2, c2, i2 = _outputs(g["q"], g["k"], block, 0xAB)
    la.select_blocks_noalloc(g["q"], g["k"], block, tau, m2, c2, i2, n_text=n_text)
    torch.cuda.synchronize()
    assert torch.equal(m2, mask), what
    assert torch.equal(c2, counts), what
    c = counts.cpu().numpy()
    a, b = idx.cpu().numpy(), i2.cpu().numpy()
    for row in np.ndindex(c.shape):
        np.testing.assert_array_equal(b[row][:c[row]], a[row][:c[row]])
    say(f"[noalloc] {what}: {int(mask.sum())} kept blocks, identical to the workspace call")


def test_noalloc_equals_workspace_selection_twice_second_smaller():
    # first the largest benchmark selection (480P long: 10.6 MB of scratch), then a small ragged
    # problem with text tokens and a different head dimension
    wl = WORKLOADS["480p_long"]
    _compare(make_inputs(wl), wl.block, wl.tau, what="480p_long")
    inp = make_clustered(2, 3, 300, 2000, 64, 64, 41, n_text=70)
    _compare(inp, 64, 0.8, n_text=70, what="B2 H3 d64 Lq300 Lk2000 text70")


def test_noalloc_without_mask_and_too_large_shape():
    inp = make_clustered(1, 2, 256, 64 * 300, 128, 64, 42)
    g = to_gpu(inp)
    mask, counts, idx = la.select_blocks(g["q"], g["k"], 64, 0.9)
    _, c2, i2 = _outputs(g["q"], g["k"], 64, 0)
    la.select_blocks_noalloc(g["q"], g["k"], 64, 0.9, None, c2, i2)
    torch.cuda.synchronize()
    assert torch.equal(c2, counts)
    # a shape whose selection scratch exceeds the library's array is refused, nothing enqueued
    q = torch.zeros((1, 16, 6400, 128), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((1, 16, 6400 + 3000 * 64, 128), dtype=torch.bfloat16, device="cuda")
    m3, c3, i3 = _outputs(q, k, 64, 0)
    with pytest.raises(la.LaError) as e:
        la.select_blocks_noalloc(q, k, 64, 0.9, m3, c3, i3)
    assert e.value.status == la.LA_ERR_WORKSPACE
    torch.cuda.synchronize()
    assert (c3 == -3).all()
