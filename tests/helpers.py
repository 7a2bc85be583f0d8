"""Shared test helpers: GPU tensors from generator bits, parity checks against the oracle."""
import math
import sys

import numpy as np

from oracle import la_oracle as O

# Attention parity bar (bf16 inputs and output, fp32 softmax/accumulation).
ATTN_MAX_ABS = 2e-2
ATTN_MEAN_ABS = 2e-3
# Selection: scores within this distance of the cutoff (or a tau crossing within this much
# mass) may legitimately flip between the fp32 kernel and the fp64 oracle.
SEL_TOL = 1e-4


def tau32(tau):
    """The cumulative-mass threshold as the C ABI receives it (a float): the oracle evaluates the
    rule at exactly that value, so that both sides cut at the same tau."""
    return None if tau is None else float(np.float32(tau))


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_gpu(inp):
    from paper_2605_31158_amd import la
    return {x: la.bf16_from_bits(inp[x]) for x in "qkv"}


def check_list(mask, counts, idx):
    """counts == popcount(mask) and idx[:count] == ascending nonzero(mask), row by row."""
    B, H, NQ, NK = mask.shape
    np.testing.assert_array_equal(counts, mask.astype(np.int64).sum(-1))
    for b in range(B):
        for h in range(H):
            for i in range(NQ):
                n = counts[b, h, i]
                np.testing.assert_array_equal(idx[b, h, i, :n], np.nonzero(mask[b, h, i])[0])


def check_selection(gpu_mask, sel, tol=SEL_TOL):
    """GPU mask equals the oracle's outside the ambiguity band; the GPU's own choice is a
    valid selection (forced blocks kept, kept scores dominate dropped ones, and for the tau
    rule the kept mass reaches tau while dropping the weakest kept block would not)."""
    want = sel["mask"]
    amb = O.ambiguous_blocks(sel, tol)
    diff = (gpu_mask != want) & ~amb
    assert not diff.any(), f"{diff.sum()} mask entries differ outside the band, first at {np.argwhere(diff)[:5]}"
    part = sel["part"]
    hist, forced = part["hist"], part["forced"]
    assert (gpu_mask[..., forced] == 1).all()
    s = sel["scores"]
    B, H, NQ, M = s.shape
    for b in range(B):
        for h in range(H):
            for i in range(NQ):
                kept = gpu_mask[b, h, i, hist].astype(bool)
                if M == 0:
                    continue
                sr = s[b, h, i]
                if kept.any() and (~kept).any():
                    assert sr[kept].min() >= sr[~kept].max() - tol, (b, h, i)
                if sel["tau"] is not None:
                    p = O.softmax_rows(sr)
                    mass = math.fsum(p[kept])
                    tau = sel["tau"]
                    if tau >= 1.0:
                        assert kept.all()
                    else:
                        assert mass >= tau - tol, (b, h, i, mass)
                        weakest = np.nonzero(kept)[0][np.argmin(sr[kept])]
                        assert mass - p[weakest] < tau + tol, (b, h, i, mass)
                else:
                    assert kept.sum() == sel["rows"][(b, h, i)]["kstar"]


def attn_errors(o_gpu, o_ref):
    d = np.abs(o_gpu.astype(np.float64) - o_ref)
    return float(d.max()), float(d.mean())


def assert_attn_close(o_gpu, o_ref, what=""):
    mx, mean = attn_errors(o_gpu, o_ref)
    assert mx <= ATTN_MAX_ABS and mean <= ATTN_MEAN_ABS, f"{what}: max-abs {mx:.3g} mean-abs {mean:.3g}"
    return mx, mean


def bf16_tensor_to_f64(t):
    import torch
    return t.detach().float().cpu().numpy().astype(np.float64)


def check_schedule(s, row_tiles=None):
    """Checks the schedule of an attention plan (la.plan_schedule) against the rule the library
    states (include/la.h, la_sparse_attn_schedule): the units' tile ranges fill [0, T) without
    overlap; workgroup l runs, on [dp_start[l], dp_start[l+1]), the units x R P/8 + r P/8 + c
    (l = x P/8 + c, r < R = (U - P/4) / P) that are at most T / (P R) tiles long, in that order;
    every other unit follows from dp_start[P] = T_dp on, in unit order; the shares
    [sk_start[l], sk_start[l+1]) fill [T_dp, T); and no workgroup gets more than ceil(T/P)
    tiles.  row_tiles (optional, [B*H, NQ]): the tiles of each query block's own list; the
    tiles of a head's units then lie between the longest list and the sum of its lists.
    Returns a summary (T, rounds, round tiles, largest and mean workgroup load)."""
    P, U = int(s["P"]), int(s["U"])
    ts = np.asarray(s["tstart"], np.int64)
    uc = np.asarray(s["ucount"], np.int64)
    dp = np.asarray(s["dp_start"], np.int64)
    sk = np.asarray(s["sk_start"], np.int64)
    assert ts.shape == (U + 1,) and uc.shape == (U,) and dp.shape == (P + 1,) and sk.shape == (P + 1,)
    assert P >= 8 and P % 8 == 0 and P <= 256, P
    assert (uc >= 0).all()
    n = np.maximum(1, uc)
    T = int(n.sum())
    assert ts[U] == T, (ts[U], T)
    order = np.argsort(ts[:U], kind="stable")
    starts = ts[:U][order]
    assert starts[0] == 0 and (starts[1:] == starts[:-1] + n[order][:-1]).all(), "unit ranges overlap or leave gaps"
    R = (U - P // 4) // P if U > P // 4 else 0
    PX = P // 8
    thr = max(1, T // (P * R)) if R > 0 else 0
    in_r = np.zeros(U, bool)
    in_r[:R * P] = n[:R * P] <= thr
    Tdp = int(n[in_r].sum())
    assert dp[0] == 0 and dp[P] == Tdp and (np.diff(dp) >= 0).all(), "round ranges"
    for lam in range(P):
        pos = dp[lam]
        for r in range(R):
            u = (lam // PX) * R * PX + r * PX + lam % PX
            if in_r[u]:
                assert ts[u] == pos, (lam, r, u, ts[u], pos)
                pos += n[u]
        assert pos == dp[lam + 1], (lam, pos, dp[lam + 1])
    pos = Tdp
    for u in np.nonzero(~in_r)[0]:
        assert ts[u] == pos, (u, ts[u], pos)
        pos += n[u]
    assert pos == T
    assert sk[0] == Tdp and sk[P] == T and (np.diff(sk) >= 0).all(), "shares"
    load = np.diff(dp) + np.diff(sk)
    assert load.max() <= -(-T // P), (int(load.max()), T, P)
    if row_tiles is not None:
        rt = np.asarray(row_tiles, np.int64)
        BH = rt.shape[0]
        assert U % BH == 0
        per_head = uc.reshape(BH, U // BH).sum(1)
        assert (per_head >= rt.max(1)).all() and (per_head <= rt.sum(1)).all(), "unit tiles vs lists"
    return {"T": T, "R": R, "T_rounds": Tdp, "max_load": int(load.max()), "mean_load": T / P}
