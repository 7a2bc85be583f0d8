"""GPU path of the 3-D block layout (Sec. 3.3) against the fp64 oracle's block-set definitions.

Q-Prep / KV-Prep: every block-major slot holds the token the oracle's block sets name (bit-exact),
padding slots are zero, regions not asked for are left untouched, and Untile Scatter inverts
Q-Prep exactly.  Block means match the oracle's pooled proxies.  Selection from the pooled means
matches the oracle's mask outside the ambiguity band (both rules).  Attention over the tiled
buffers, with the padding masked through the valid counts, matches the oracle on the GPU's own
mask: max-abs <= 2e-2, mean-abs <= 2e-3, lse within 1e-3."""
import numpy as np
import pytest
import torch

from oracle import la_oracle as O
from paper_2605_31158_amd import la
from paper_2605_31158_amd.workloads import WORKLOADS_3D, Workload3D, make_inputs_3d
from helpers import check_schedule, say, tau32, to_gpu, check_list, check_selection, assert_attn_close, bf16_tensor_to_f64

pytestmark = pytest.mark.gpu

LSE_TOL = 1e-3
SENTINEL = 0x7777   # bf16 bits of a value no prep writes into an untouched region


def grid_of(wl: Workload3D):
    return la.grid3d(wl.B, wl.H, wl.d, wl.n_text, wl.T_ctx, wl.T_q, wl.Hs, wl.Ws, wl.bt, wl.bh, wl.bw, wl.block)


def layout_of(wl: Workload3D):
    return O.layout_3d(wl.n_text, wl.T_ctx, wl.T_q, wl.Hs, wl.Ws, wl.bt, wl.bh, wl.bw, wl.block)


def slot_tokens(sets, block):
    """Token of every block-major slot (-1 for padding)."""
    out = np.full(len(sets) * block, -1, np.int64)
    for n, s in enumerate(sets):
        out[n * block:n * block + s.size] = s
    return out


def bits_of(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def check_tiled(tiled_bits, lin_bits, tokens, what):
    valid = tokens >= 0
    np.testing.assert_array_equal(tiled_bits[:, :, valid], lin_bits[:, :, tokens[valid]], err_msg=what)
    assert (tiled_bits[:, :, ~valid] == 0).all(), f"{what}: padding not zero"


SMALL = {
    "tiny_3d": WORKLOADS_3D["tiny_3d"],
    # whole 4x8x4 blocks but ragged rows (30 = 3 x 8 + 6) and ragged frames (T_ctx = 5)
    "hy_small": Workload3D("hy_small", 1, 2, 128, 70, 5, 4, 30, 52, 4, 8, 4, 128, 21, 2, 1, tau=0.9),
    # 4x4x8 blocks on the 45x80 grid: last block row holds one token row (32 valid slots)
    "mg_small": Workload3D("mg_small", 2, 1, 128, 0, 4, 4, 45, 80, 4, 4, 8, 128, 22, 2, 0, topk_r=0.175),
    # d = 64 with 64-slot blocks of 2x4x8 = 64 tokens, no text, single chunk frame
    "d64_b64": Workload3D("d64_b64", 1, 3, 64, 0, 6, 1, 12, 20, 2, 4, 8, 64, 23, 2, 1, tau=0.8),
    # no context frames (M = 0): text (exactly two blocks) and chunk only
    "no_ctx": Workload3D("no_ctx", 1, 2, 64, 128, 0, 3, 7, 10, 2, 3, 4, 64, 24, 0, 0, tau=0.9),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_prep_q_layout_means_and_untile_identity(name):
    wl = SMALL[name]
    say(f"[3d] prep_q {name}")
    inp = make_inputs_3d(wl)
    g = to_gpu(inp)
    grid = grid_of(wl)
    L = layout_of(wl)
    q_t, qbar = la.prep_q_3d(grid, g["q"])
    o_lin, _ = la.untile_o_3d(grid, q_t)
    torch.cuda.synchronize()
    check_tiled(bits_of(q_t), inp["q"], slot_tokens(L["qsets"], wl.block), f"{name} q_tiled")
    np.testing.assert_array_equal(bits_of(o_lin), inp["q"], err_msg=f"{name}: untile(prep_q(q)) != q")
    qb = O.pool_sets(_f64(inp["q"]), L["qsets"])
    np.testing.assert_allclose(qbar.cpu().numpy(), qb, rtol=1e-5, atol=1e-5)


def _f64(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("name", list(SMALL))
def test_prep_kv_regions_layout_and_means(name):
    wl = SMALL[name]
    say(f"[3d] prep_kv {name}")
    inp = make_inputs_3d(wl)
    g = to_gpu(inp)
    grid = grid_of(wl)
    L = layout_of(wl)
    shape = la.grid3d_shape(grid)
    NK = shape.Lk // wl.block
    NT = shape.n_text // wl.block
    NQ = shape.Lq // wl.block
    NC = NK - NT - NQ
    kt = torch.full((wl.B, wl.H, shape.Lk, wl.d), 0, dtype=torch.int16, device="cuda")
    kt.fill_(SENTINEL)
    kt = kt.view(torch.bfloat16)
    vt = kt.clone()
    kbar = torch.full((wl.B, wl.H, NK, wl.d), 12345.0, dtype=torch.float32, device="cuda")
    tokens = slot_tokens(L["ksets"], wl.block)
    region = np.repeat(np.array([0] * NT + [1] * NC + [2] * NQ), wl.block)
    # chunk only: text and context regions keep the sentinel
    la.prep_kv_3d(grid, g["k"], g["v"], la.LA_PART_CHUNK, kt, vt, kbar)
    torch.cuda.synchronize()
    kb = bits_of(kt)
    assert (kb[:, :, region != 2] == SENTINEL).all()
    assert (kbar[:, :, :NT + NC].cpu().numpy() == 12345.0).all()
    sel = region == 2
    check_tiled(kb[:, :, sel], inp["k"], tokens[sel], f"{name} chunk K")
    # then text + context
    la.prep_kv_3d(grid, g["k"], g["v"], la.LA_PART_TEXT | la.LA_PART_CONTEXT, kt, vt, kbar)
    torch.cuda.synchronize()
    check_tiled(bits_of(kt), inp["k"], tokens, f"{name} K")
    check_tiled(bits_of(vt), inp["v"], tokens, f"{name} V")
    kb_ref = O.pool_sets(_f64(inp["k"]), L["ksets"])
    np.testing.assert_allclose(kbar.cpu().numpy(), kb_ref, rtol=1e-5, atol=1e-5)


def run_path(wl, inp, keep_blocks=None, tau=None):
    g = to_gpu(inp)
    grid = grid_of(wl)
    o, lse, mask, counts, idx = la.sparse_attn_3d(grid, g["q"], g["k"], g["v"], tau=tau, keep_blocks=keep_blocks,
                                                  want_lse=True)
    torch.cuda.synchronize()
    return (bf16_tensor_to_f64(o), lse.cpu().numpy().astype(np.float64), mask.cpu().numpy(), counts.cpu().numpy(),
            idx.cpu().numpy())


def rule_args(wl, M):
    if wl.tau is not None:
        return dict(tau=wl.tau), dict(tau=tau32(wl.tau))
    return dict(keep_blocks=int(np.floor(wl.topk_r * M))), dict(topk_r=wl.topk_r)


def compare_rows(o, lse, inp, L, mask, rows, what, scale=None):
    ref = O.attention_sets_rows(inp["q"], inp["k"], inp["v"], L["qsets"], L["ksets"], mask, rows, scale=scale)
    mx = mean_sum = n = 0.0
    for (b, h, i), (ob, lb) in ref.items():
        qi = L["qsets"][i]
        assert_attn_close(o[b, h, qi], ob, f"{what} row {(b, h, i)}")
        d = np.abs(o[b, h, qi] - ob)
        mx, mean_sum, n = max(mx, float(d.max())), mean_sum + float(d.sum()), n + d.size
        assert np.abs(lse[b, h, qi] - lb).max() <= LSE_TOL, (what, b, h, i)
    assert mean_sum / n <= 2e-3
    say(f"[3d] {what}: {len(rows)} query blocks, max-abs {mx:.2e} mean-abs {mean_sum / n:.2e}")


@pytest.mark.parametrize("name", list(SMALL))
def test_path_matches_oracle(name):
    wl = SMALL[name]
    say(f"[3d] path {name}")
    inp = make_inputs_3d(wl)
    L = layout_of(wl)
    M = int((~L["forced"]).sum())
    gargs, oargs = rule_args(wl, M)
    o, lse, mask, counts, idx = run_path(wl, inp, **gargs)
    sel = O.select_blocks_sets(inp["q"], inp["k"], L["qsets"], L["ksets"], L["forced"], **oargs)
    check_selection(mask, sel)
    check_list(mask, counts, idx)
    rows = [(b, h, i) for b in range(wl.B) for h in range(wl.H) for i in range(len(L["qsets"]))]
    if len(rows) > 40:     # every edge block (the ragged ones) of the first head, then a sample
        NQ = len(L["qsets"])
        qv = np.array([s.size for s in L["qsets"]])
        edge = [(0, 0, i) for i in np.nonzero(qv < wl.bt * wl.bh * wl.bw)[0][:16]]
        rng = np.random.default_rng(1)
        rest = [rows[j] for j in rng.choice(len(rows), size=24, replace=False)]
        rows = sorted(set(edge + rest + [rows[0], rows[-1]]))
    compare_rows(o, lse, inp, L, mask, rows, name)


@pytest.mark.parametrize("name", ["tiny_3d", "hy_small"])
def test_both_rules_on_pooled_means(name):
    wl = SMALL[name]
    inp = make_inputs_3d(wl)
    g = to_gpu(inp)
    grid = grid_of(wl)
    L = layout_of(wl)
    shape = la.grid3d_shape(grid)
    _, qbar = la.prep_q_3d(grid, g["q"])
    _, _, kbar = la.prep_kv_3d(grid, g["k"], g["v"])
    M = int((~L["forced"]).sum())
    for tau in (0.5, 0.95, 1.0):
        mask, counts, idx = la.select_pooled(shape, qbar, kbar, tau=tau)
        sel = O.select_blocks_sets(inp["q"], inp["k"], L["qsets"], L["ksets"], L["forced"], tau=tau32(tau))
        check_selection(mask.cpu().numpy(), sel)
        check_list(mask.cpu().numpy(), counts.cpu().numpy(), idx.cpu().numpy())
    for r in (0.1, 0.5):
        mask, counts, idx = la.select_pooled(shape, qbar, kbar, keep_blocks=int(np.floor(r * M)))
        sel = O.select_blocks_sets(inp["q"], inp["k"], L["qsets"], L["ksets"], L["forced"], topk_r=r)
        check_selection(mask.cpu().numpy(), sel)


def test_valid_counts_mask_padding_and_full_counts_change_nothing():
    wl = SMALL["hy_small"]
    inp = make_inputs_3d(wl)
    g = to_gpu(inp)
    grid = grid_of(wl)
    shape = la.grid3d_shape(grid)
    kvalid = torch.from_numpy(la.grid3d_valid(grid)[1]).cuda()
    q_t, _ = la.prep_q_3d(grid, g["q"], want_qbar=False)
    k_t, v_t, _ = la.prep_kv_3d(grid, g["k"], g["v"], want_kbar=False)
    NQ, NK = shape.Lq // wl.block, shape.Lk // wl.block
    mask = torch.ones((wl.B, wl.H, NQ, NK), dtype=torch.uint8, device="cuda")
    counts, idx = la.mask_to_list(mask, wl.block, shape.Lq, shape.Lk, wl.d)
    ws = torch.empty(la.workspace_bytes(shape), dtype=torch.uint8, device="cuda")
    o1, l1 = la.sparse_attn_fwd(q_t, k_t, v_t, counts, idx, wl.block, n_text=shape.n_text, want_lse=True,
                                kvalid=kvalid, ws=ws)
    # the plan leaves out the sub-tiles with no valid key: a key block of v valid keys has
    # ceil(v / 64) tiles, and every query block keeps every key block here
    kv = la.grid3d_valid(grid)[1].astype(np.int64)
    per_row = int(sum(-(-min(wl.block, int(x)) // 64) for x in kv))
    check_schedule(la.plan_schedule(shape, ws), row_tiles=np.full((wl.B * wl.H, NQ), per_row))
    # garbage in every padding slot: the valid counts keep it out
    pad = torch.from_numpy(la.grid3d_valid(grid)[1]).cuda()
    slot = torch.arange(shape.Lk, device="cuda") % wl.block
    is_pad = slot >= pad.repeat_interleave(wl.block)
    k2, v2 = k_t.clone(), v_t.clone()
    k2[:, :, is_pad] = 30.0
    v2[:, :, is_pad] = -500.0
    o2, l2 = la.sparse_attn_fwd(q_t, k2, v2, counts, idx, wl.block, n_text=shape.n_text, want_lse=True,
                                kvalid=kvalid)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    # all slots valid: the plain call and the _valid call agree bit for bit
    full = torch.full_like(kvalid, wl.block)
    o3, l3 = la.sparse_attn_fwd(q_t, k_t, v_t, counts, idx, wl.block, n_text=shape.n_text, want_lse=True,
                                kvalid=full)
    o4, l4 = la.sparse_attn_fwd(q_t, k_t, v_t, counts, idx, wl.block, n_text=shape.n_text, want_lse=True)
    torch.cuda.synchronize()
    assert torch.equal(o3, o4) and torch.equal(l3, l4)


@pytest.mark.slow
@pytest.mark.parametrize("name", ["480p_3d", "720p_3d"])
def test_named_3d_workloads(name):
    wl = WORKLOADS_3D[name]
    say(f"[3d] {name}: drawing inputs")
    inp = make_inputs_3d(wl)
    L = layout_of(wl)
    M = int((~L["forced"]).sum())
    gargs, oargs = rule_args(wl, M)
    o, lse, mask, counts, idx = run_path(wl, inp, **gargs)
    say(f"[3d] {name}: GPU path done, oracle selection")
    sel = O.select_blocks_sets(inp["q"], inp["k"], L["qsets"], L["ksets"], L["forced"], **oargs)
    check_selection(mask, sel)
    NQ = len(L["qsets"])
    rng = np.random.default_rng(5)
    pick = sorted({0, NQ - 1, *rng.integers(0, NQ, size=4).tolist()})
    rows = [(0, int(h), i) for i, h in zip(pick, rng.integers(0, wl.H, size=len(pick)))]
    compare_rows(o, lse, inp, L, mask, rows, name)


@pytest.mark.parametrize("block", [64, 128])
def test_kvalid_truncates_key_blocks(block):
    # any valid counts per key block (0, partial, full): attention sees the first kvalid[m] keys
    # of every kept block m, as the oracle over the truncated block sets
    rng = np.random.default_rng(block)
    B, H, d, NQ, NK = 1, 2, 128, 3, 9
    Lq, Lk = NQ * block, NK * block
    from paper_2605_31158_amd.workloads import make_clustered
    inp = make_clustered(B, H, Lq, Lk, d, block, 40 + block)
    kv = rng.integers(0, block + 1, size=NK).astype(np.int32)
    kv[0], kv[-1] = 0, block // 2 + 3
    mask = (rng.uniform(size=(B, H, NQ, NK)) < 0.6).astype(np.uint8)
    mask[..., -1] = 1
    g = to_gpu(inp)
    counts, idx = la.mask_to_list(torch.from_numpy(mask).cuda(), block, Lq, Lk, d)
    o, lse = la.sparse_attn_fwd(g["q"], g["k"], g["v"], counts, idx, block, want_lse=True,
                                kvalid=torch.from_numpy(kv).cuda())
    torch.cuda.synchronize()
    qsets = [np.arange(i * block, (i + 1) * block) for i in range(NQ)]
    ksets = [np.arange(m * block, m * block + kv[m]) for m in range(NK)]
    rows = [(0, h, i) for h in range(H) for i in range(NQ)]
    ref = O.attention_sets_rows(inp["q"], inp["k"], inp["v"], qsets, ksets, mask, rows)
    o_np, lse_np = bf16_tensor_to_f64(o), lse.cpu().numpy().astype(np.float64)
    for (b, h, i), (ob, lb) in ref.items():
        rs = slice(i * block, (i + 1) * block)
        assert_attn_close(o_np[b, h, rs], ob, f"kvalid block {block} row {(b, h, i)}")
        fin = np.isfinite(lb)
        assert np.isneginf(lse_np[b, h, rs][~fin]).all()
        if fin.any():
            assert np.abs(lse_np[b, h, rs][fin] - lb[fin]).max() <= LSE_TOL
