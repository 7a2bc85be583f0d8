"""The path at the largest shapes the library accepts, against the fp64 oracle.

* M = 4096 historical candidate blocks (the selection's per-row limit): selection (tau rule
  and Top-k) and attention over the resulting lists, every output row compared.
* B * H = 65535 (the largest (batch, head) count): selection and attention over all heads,
  a sample of heads compared; heads are independent, so the oracle on the sampled heads alone
  is the reference for them.
"""
import numpy as np
import pytest
import torch

from oracle import la_oracle as O
from paper_2605_31158_amd import la
from paper_2605_31158_amd.workloads import make_clustered
from helpers import say, tau32, to_gpu, check_list, check_selection, assert_attn_close, bf16_tensor_to_f64

pytestmark = pytest.mark.gpu

LSE_TOL = 1e-3


def _compare(o, lse, o_ref, lse_ref, what):
    mx, mean = assert_attn_close(o, o_ref, what)
    fin = np.isfinite(lse_ref)
    assert np.isneginf(lse[~fin]).all(), what
    assert np.abs(lse[fin] - lse_ref[fin]).max() <= LSE_TOL, what
    say(f"[limits] {what}: max-abs {mx:.2e} mean-abs {mean:.2e}")


@pytest.mark.parametrize("rule", ["tau", "topk"])
def test_most_candidate_blocks(rule):
    # Lk = 4097 blocks of 64 keys, one query block: M = 4096 historical candidates per row
    B, H, Lq, d, block = 1, 2, 64, 64, 64
    Lk = block * 4097
    say(f"[limits] M = 4096, rule {rule}: B={B} H={H} Lq={Lq} Lk={Lk} d={d}")
    inp = make_clustered(B, H, Lq, Lk, d, block, seed=21)
    g = to_gpu(inp)
    if rule == "tau":
        mask, counts, idx = la.select_blocks(g["q"], g["k"], block, 0.95)
        sel = O.select_blocks(inp["q"], inp["k"], block, tau=tau32(0.95))
    else:
        keep = int(0.175 * 4096)
        mask, counts, idx = la.select_blocks_topk(g["q"], g["k"], block, keep)
        sel = O.select_blocks(inp["q"], inp["k"], block, topk_r=keep / 4096)
    o, lse = la.sparse_attn_fwd(g["q"], g["k"], g["v"], counts, idx, block, want_lse=True)
    torch.cuda.synchronize()
    mask_np = mask.cpu().numpy()
    check_selection(mask_np, sel)
    check_list(mask_np, counts.cpu().numpy(), idx.cpu().numpy())
    o_ref, lse_ref = O.attention(inp["q"], inp["k"], inp["v"], mask_np, block)
    _compare(bf16_tensor_to_f64(o), lse.cpu().numpy().astype(np.float64), o_ref, lse_ref,
             f"M = 4096 {rule}: kept blocks per row {mask_np.sum(-1).ravel().tolist()}")


def test_most_batch_heads():
    # B * H = 65535, two historical key blocks and the chunk block per head
    B, H, Lq, Lk, d, block = 5, 13107, 64, 192, 64, 64
    say(f"[limits] B*H = {B * H}: Lq={Lq} Lk={Lk} d={d} block={block}")
    gen = torch.Generator(device="cuda").manual_seed(22)
    # per-head scale spreads the scores so that both rules see a range of distributions
    sc = torch.rand((B, H, 1, 1), generator=gen, device="cuda") * 3.0
    q = (torch.randn((B, H, Lq, d), generator=gen, device="cuda") * sc).to(torch.bfloat16)
    k = torch.randn((B, H, Lk, d), generator=gen, device="cuda").to(torch.bfloat16)
    v = torch.randn((B, H, Lk, d), generator=gen, device="cuda").to(torch.bfloat16)
    mask, counts, idx = la.select_blocks(q, k, block, 0.6)
    o, lse = la.sparse_attn_fwd(q, k, v, counts, idx, block, want_lse=True)
    torch.cuda.synchronize()
    mask_np, counts_np = mask.cpu().numpy(), counts.cpu().numpy()
    np.testing.assert_array_equal(counts_np, mask_np.astype(np.int64).sum(-1))
    assert (mask_np[..., 2] == 1).all()            # the chunk block is always kept
    rng = np.random.default_rng(23)
    flat = sorted(set([0, B * H - 1, H - 1, H] + rng.integers(0, B * H, size=28).tolist()))
    bs = np.array([f // H for f in flat])
    hs = np.array([f % H for f in flat])
    bs_t, hs_t = torch.as_tensor(bs, device="cuda"), torch.as_tensor(hs, device="cuda")
    pick = lambda t: t[bs_t, hs_t][None].float().cpu().numpy()     # [1, n, L, d], exact bf16 values
    qs, ks, vs = pick(q), pick(k), pick(v)
    sel = O.select_blocks(qs, ks, block, tau=tau32(0.6))
    m_s = mask_np[bs, hs][None]
    check_selection(m_s, sel)
    check_list(m_s, counts_np[bs, hs][None], idx.cpu().numpy()[bs, hs][None])
    o_ref, lse_ref = O.attention(qs, ks, vs, m_s, block)
    o_s = bf16_tensor_to_f64(o[bs_t, hs_t][None])
    lse_s = lse[bs_t, hs_t][None].cpu().numpy().astype(np.float64)
    _compare(o_s, lse_s, o_ref, lse_ref, f"B*H = {B * H}, {len(flat)} heads sampled")
