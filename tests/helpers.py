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
