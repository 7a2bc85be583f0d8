"""Pins for the fp64 oracle: closed forms, brute force, library attention, invariants.

None of these re-types the oracle's own formula: each checks it against something
the paper's equations (Sec. 3.3) or plain mathematics fix independently.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

import oracle
from oracle import la_oracle as O
from paper_2605_31158_amd.workloads import WORKLOADS, make_inputs, make_clustered, f32_to_bf16_bits

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------
# pins, written as functions so that tests/test_oracle_mutants.py can run them
# against an oracle with a planted mistake and watch them fail.

def pin_bf16_decode():
    bits = np.array([0x3F80, 0xC000, 0x3F81, 0x0000, 0x8000, 0x4049, 0x0001], np.uint16)
    want = [1.0, -2.0, 1.0 + 2.0 ** -7, 0.0, -0.0, 3.140625, 2.0 ** -133]
    got = O.bf16_bits_to_f64(bits)
    assert got.tolist() == want


def pin_partition():
    # block counts of the benchmark shapes: ceil divisions and the chunk's block range
    for (Lq, Lk, b, NQ, NK, M) in [(256, 1024, 64, 4, 16, 12), (6240, 18720, 64, 98, 293, 195),
                                   (6240, 43680, 64, 98, 683, 585), (14400, 72000, 128, 113, 563, 450),
                                   (6240, 106080, 64, 98, 1658, 1560)]:
        p = O.partition(Lq, Lk, b)
        assert (p["NQ"], p["NK"], p["M"]) == (NQ, NK, M)
        assert p["forced"][M:].all() and not p["forced"][:M].any()
    # chunk start not block aligned: block 1 = [64,128) straddles the chunk start 100
    p = O.partition(Lq=60, Lk=160, block=64)
    assert p["forced"].tolist() == [False, True, True] and p["hist"].tolist() == [0]
    # text tokens: blocks overlapping [0, 70) are forced
    p = O.partition(Lq=64, Lk=640, block=64, n_text=70)
    assert p["forced"].tolist() == [True, True] + [False] * 7 + [True]
    # no history at all
    p = O.partition(Lq=128, Lk=128, block=64)
    assert p["M"] == 0 and p["forced"].all()


def pin_pool_closed_form():
    # x[t, c] = a_c + t * s_c: the mean over tokens [lo, hi) is a_c + s_c * (lo + hi - 1) / 2
    L, d, b = 150, 5, 64
    a = np.array([1.0, -2.0, 0.5, 3.0, 0.0])
    s = np.array([0.25, 1.0, -0.5, 0.0, 2.0])
    x = a[None, :] + np.arange(L)[:, None] * s[None, :]
    got = O.pool_blocks(x, b)
    for i, (lo, hi) in enumerate([(0, 64), (64, 128), (128, 150)]):
        want = a + s * (lo + hi - 1) / 2.0
        np.testing.assert_allclose(got[i], want, rtol=0, atol=1e-12)


def pin_scores_closed_form():
    d = 16
    qbar = np.zeros((2, d))
    kbar = np.zeros((3, d))
    qbar[0, 0] = 2.0
    qbar[1, 1] = -1.0
    qbar[1, 2] = 3.0
    kbar[0, 0] = 4.0           # parallel to q0
    kbar[1, 1] = 5.0           # orthogonal to q0
    kbar[2, 2] = 1.0
    kbar[2, 0] = 1.0
    got = O.block_scores(qbar, kbar, d)
    want = np.array([[8.0, 0.0, 2.0], [0.0, -5.0, 3.0]]) / 4.0   # sqrt(16) = 4
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-15)


def pin_softmax_properties():
    rng = np.random.default_rng(3)
    s = rng.normal(size=(5, 9)) * 4
    p = O.softmax_rows(s)
    np.testing.assert_allclose(p.sum(-1), 1.0, atol=1e-14)
    # ratio of two probabilities is exp of the score difference
    np.testing.assert_allclose(p[:, 2] / p[:, 7], np.exp(s[:, 2] - s[:, 7]), rtol=1e-12)
    big = O.softmax_rows(np.array([[1000.0, 999.0, -1000.0]]))
    np.testing.assert_allclose(big[0], [1 / (1 + math.e ** -1), math.e ** -1 / (1 + math.e ** -1), 0.0],
                               rtol=1e-12, atol=1e-300)


def _brute_tau(s, tau):
    """All 2^M subsets: the smallest subset whose softmax mass reaches tau; among
    those the largest mass; remaining ties go to the lexicographically smallest
    sorted index tuple (lower block index first)."""
    M = s.size
    e = np.exp(s - s.max())
    p = e / e.sum()
    if tau >= 1.0:
        return tuple(range(M))
    best = None
    for k in range(1, M + 1):
        for sub in itertools.combinations(range(M), k):
            mass = math.fsum(p[list(sub)])
            if mass >= tau:
                key = (-mass, sub)
                if best is None or key < best:
                    best = key
        if best is not None:
            return best[1]
    return tuple(range(M))


def pin_tau_brute_force():
    rng = np.random.default_rng(11)
    for trial in range(300):
        M = int(rng.integers(1, 11))
        s = rng.normal(size=M) * float(rng.choice([0.3, 1.0, 3.0]))
        tau = float(rng.uniform(0.05, 0.999))
        got = tuple(O.select_tau_row(s, tau)["selected"].tolist())
        assert got == _brute_tau(s, tau), (trial, s, tau)
    # exact score ties: lower index wins
    s = np.array([1.0, 2.0, 2.0, 0.0, 2.0])
    e = np.exp(s - 2.0)
    p = e / e.sum()
    one = p[1]
    assert tuple(O.select_tau_row(s, one * 0.5)["selected"]) == (1,)
    assert tuple(O.select_tau_row(s, one * 1.5)["selected"]) == (1, 2)
    assert tuple(O.select_tau_row(s, one * 2.5)["selected"]) == (1, 2, 4)
    # C_k meeting tau exactly stops there (the rule is C_k >= tau): two equal scores, tau = 1/2
    assert tuple(O.select_tau_row(np.array([0.0, 0.0]), 0.5)["selected"]) == (0,)
    assert tuple(O.select_tau_row(np.array([0.0, 0.0, 0.0, 0.0]), 0.5)["selected"]) == (0, 1)
    # tau >= 1 keeps all; a tiny tau keeps exactly the argmax; M = 0 keeps nothing
    assert O.select_tau_row(s, 1.0)["kstar"] == 5
    assert tuple(O.select_tau_row(np.array([0.1, 0.9, 0.3]), 1e-9)["selected"]) == (1,)
    assert O.select_tau_row(np.zeros(0), 0.9)["kstar"] == 0


def pin_topk_brute_force():
    rng = np.random.default_rng(12)
    for _ in range(200):
        M = int(rng.integers(1, 12))
        s = np.round(rng.normal(size=M), 1)          # rounding makes ties common
        r = float(rng.uniform(0.0, 1.0))
        k = math.floor(r * M + 1e-9)
        got = tuple(O.select_topk_row(s, r)["selected"].tolist())
        best = None
        for sub in itertools.combinations(range(M), k):
            key = (-math.fsum(s[list(sub)]), sub)
            if best is None or key < best:
                best = key
        assert got == (best[1] if best is not None else ())


def pin_golden_hand_worked():
    with open(os.path.join(GOLDEN, "hand_worked_select.json")) as f:
        g = json.load(f)
    q = np.array(g["q"], np.float64)[None, None]
    k = np.array(g["k"], np.float64)[None, None]
    v = np.array(g["v"], np.float64)[None, None]
    sel = O.select_blocks(q, k, g["block"], tau=0.9)
    np.testing.assert_allclose(sel["scores"][0, 0, 0], [1.5, 0.5, -0.5], atol=1e-15)
    e = math.e
    Z = e * e + e + 1
    np.testing.assert_allclose(sel["rows"][(0, 0, 0)]["p"], [e * e / Z, e / Z, 1 / Z], rtol=1e-14)
    for tau, want in g["expect_mask"].items():
        m = O.select_blocks(q, k, g["block"], tau=float(tau))["mask"]
        assert m[0, 0, 0].tolist() == want, tau
    for r, want in g["expect_topk_mask"].items():
        m = O.select_blocks(q, k, g["block"], topk_r=float(r))["mask"]
        assert m[0, 0, 0].tolist() == want, r
    m = O.select_blocks(q, k, g["block"], tau=0.5)["mask"]
    o, lse = O.attention(q, k, v, m, g["block"])
    e4, e2 = math.exp(4), math.exp(2)
    den = e4 + e2 + 2
    np.testing.assert_allclose(o[0, 0, 0], np.array([e4 + 1, e2, 1, 2]) / den, rtol=1e-14)
    np.testing.assert_allclose(lse[0, 0, 0], math.log(den), rtol=1e-14)
    # query token 1 is the zero vector: uniform weights over the 4 visible keys
    np.testing.assert_allclose(o[0, 0, 1], (v[0, 0, 0] + v[0, 0, 1] + v[0, 0, 6] + v[0, 0, 7]) / 4,
                               rtol=1e-14)
    np.testing.assert_allclose(lse[0, 0, 1], math.log(4.0), rtol=1e-14)


def _sdpa(q, k, v, allowed, scale):
    """torch's fp64 CPU attention with a boolean mask [Lq, Lk] (True = attend)."""
    tq = torch.from_numpy(q)[None]
    tk = torch.from_numpy(k)[None]
    tv = torch.from_numpy(v)[None]
    am = torch.from_numpy(allowed)[None]
    return torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=am, scale=scale)[0].numpy()


def pin_attention_dense_matches_library():
    # keep-all (tau = 1) is plain softmax attention
    inp = make_clustered(1, 2, Lq=100, Lk=300, d=32, block=32, seed=5)
    q, k, v = (O.bf16_bits_to_f64(inp[x]) for x in "qkv")
    sel = O.select_blocks(inp["q"], inp["k"], 32, tau=1.0)
    assert sel["mask"].all()
    o, lse = O.attention(q, k, v, sel["mask"], 32)
    for h in range(2):
        want = _sdpa(q[0, h], k[0, h], v[0, h], np.ones((100, 300), bool), 1 / math.sqrt(32))
        np.testing.assert_allclose(o[0, h], want, rtol=0, atol=1e-12)
        logits = q[0, h] @ k[0, h].T / math.sqrt(32)
        np.testing.assert_allclose(lse[0, h], logsumexp(logits, axis=1), rtol=1e-13)


def pin_attention_sparse_matches_library():
    # a random block mask, expanded to tokens by np.kron, through the library routine
    rng = np.random.default_rng(8)
    Lq, Lk, b, d = 96, 320, 32, 16
    q = rng.normal(size=(1, 1, Lq, d))
    k = rng.normal(size=(1, 1, Lk, d))
    v = rng.normal(size=(1, 1, Lk, d))
    NQ, NK = 3, 10
    mask = (rng.uniform(size=(1, 1, NQ, NK)) < 0.4).astype(np.uint8)
    mask[..., -3:] = 1
    o, lse = O.attention(q, k, v, mask, b, scale=0.3)
    allowed = np.kron(mask[0, 0], np.ones((b, b))).astype(bool)
    want = _sdpa(q[0, 0], k[0, 0], v[0, 0], allowed, 0.3)
    np.testing.assert_allclose(o[0, 0], want, rtol=0, atol=1e-12)


def pin_attention_frame_causal_matches_library():
    rng = np.random.default_rng(9)
    Lq, Lk, b, d, F = 90, 250, 32, 8, 30      # frames of 30 tokens, not block aligned
    q, k, v = (rng.normal(size=(1, 1, L, d)) for L in (Lq, Lk, Lk))
    NQ, NK = 3, 8
    mask = np.ones((1, 1, NQ, NK), np.uint8)
    mask[0, 0, :, 1] = 0
    o, lse = O.attention(q, k, v, mask, b, frame_tokens=F)
    c0 = Lk - Lq
    qf = np.arange(Lq) // F
    kf = np.where(np.arange(Lk) < c0, -1, (np.arange(Lk) - c0) // F)
    allowed = (kf[None, :] <= qf[:, None]) & np.repeat(mask[0, 0].astype(bool), b, axis=1)[
        np.minimum(np.arange(Lq) // b, NQ - 1)][:, :Lk]
    want = _sdpa(q[0, 0], k[0, 0], v[0, 0], allowed, 1 / math.sqrt(d))
    np.testing.assert_allclose(o[0, 0], want, rtol=0, atol=1e-12)


def pin_attention_invariants():
    rng = np.random.default_rng(10)
    Lq, Lk, b, d = 64, 192, 32, 8
    q, k = (rng.normal(size=(1, 1, L, d)) for L in (Lq, Lk))
    mask = np.ones((1, 1, 2, 6), np.uint8)
    mask[0, 0, 0, 0] = 0
    # V = 1 everywhere gives O = 1
    o, _ = O.attention(q, k, np.ones((1, 1, Lk, d)), mask, b)
    np.testing.assert_allclose(o, 1.0, atol=1e-14)
    # one-hot V: column n of O is the attention weight of key n; rows sum to 1, zero off-mask
    vv = np.zeros((1, 1, Lk, Lk))
    vv[0, 0] = np.eye(Lk)
    P, _ = O.attention(q, k, vv, mask, b)
    np.testing.assert_allclose(P.sum(-1), 1.0, atol=1e-13)
    assert (P[0, 0, :32, :32] == 0).all() and (P[0, 0, 32:, :32] > 0).all()
    # each weight ratio is exp of the scaled logit difference
    lg = q[0, 0] @ k[0, 0].T / math.sqrt(d)
    np.testing.assert_allclose(P[0, 0, :, 40] / P[0, 0, :, 100], np.exp(lg[:, 40] - lg[:, 100]), rtol=1e-10)
    # a single visible key: the output is that key's value row.  Frames of one token make
    # chunk query 0 see chunk key 0 (key 4) only, and only chunk blocks are kept.
    Lq2, Lk2 = 4, 8
    q2 = rng.normal(size=(1, 1, Lq2, d))
    k2 = rng.normal(size=(1, 1, Lk2, d))
    v2 = rng.normal(size=(1, 1, Lk2, d))
    m2 = np.array([[[[0, 0, 1, 1], [0, 0, 1, 1]]]], np.uint8)
    o2, lse2 = O.attention(q2, k2, v2, m2, 2, frame_tokens=1)
    np.testing.assert_allclose(o2[0, 0, 0], v2[0, 0, 4], atol=1e-15)
    np.testing.assert_allclose(lse2[0, 0, 0], q2[0, 0, 0] @ k2[0, 0, 4] / math.sqrt(d), atol=1e-14)
    # no visible key at all: o = 0, lse = -inf
    none = np.zeros((1, 1, 2, 4), np.uint8)
    o3, lse3 = O.attention(q2, k2, v2, none, 2)
    assert (o3 == 0).all() and np.isneginf(lse3).all()


def pin_permutation_invariance():
    # permuting historical key blocks (K and V together) permutes the mask and leaves O unchanged
    inp = make_clustered(1, 1, Lq=64, Lk=384, d=16, block=32, seed=21)
    q, k, v = (O.bf16_bits_to_f64(inp[x]) for x in "qkv")
    perm = np.array([3, 0, 7, 5, 1, 6, 2, 4])        # the 8 historical blocks; chunk blocks 8, 9 stay
    tok = np.concatenate([np.arange(32 * p, 32 * p + 32) for p in perm] + [np.arange(256, 384)])
    sel = O.select_blocks(q, k, 32, tau=0.8)
    sel_p = O.select_blocks(q, k[:, :, tok], 32, tau=0.8)
    np.testing.assert_array_equal(sel_p["mask"][..., :8], sel["mask"][..., perm])
    o, _ = O.attention(q, k, v, sel["mask"], 32)
    o_p, _ = O.attention(q, k[:, :, tok], v[:, :, tok], sel_p["mask"], 32)
    np.testing.assert_allclose(o_p, o, atol=1e-13)


def pin_kept_flops():
    mask = np.ones((1, 2, 3, 5), np.uint8)
    assert O.kept_flops(mask, Lq=150, Lk=300, block=64, d=8) == 4 * 2 * 150 * 300 * 8
    mask[0, 0, 2, 4] = 0           # drops a (22-row) x (44-key) tile
    assert O.kept_flops(mask, Lq=150, Lk=300, block=64, d=8) == 4 * 8 * (2 * 150 * 300 - 22 * 44)


def _band_row(case):
    """The selection dict ambiguous_blocks reads, for one golden row of scores."""
    s = np.array(case["scores"], np.float64)[None, None, None]
    tau, r = case.get("tau"), case.get("r")
    row = O.select_tau_row(s[0, 0, 0], tau) if tau is not None else O.select_topk_row(s[0, 0, 0], r)
    return {"scores": s, "part": {"hist": np.array(case["hist"]), "NK": case["NK"]}, "tau": tau,
            "topk_r": r, "rows": {(0, 0, 0): row}}


def pin_ambiguity_band_golden():
    # every clause of the band on its own, worked by hand (tests/golden/ambiguity_band.json)
    with open(os.path.join(GOLDEN, "ambiguity_band.json")) as f:
        g = json.load(f)
    assert g["tol"] == 1e-4          # the stated tolerance, which is also the band's default
    for case in g["cases"]:
        amb = O.ambiguous_blocks(_band_row(case))
        assert amb[0, 0, 0].tolist() == case["expect_blocks"], case["name"]


def pin_ambiguity_band_covers_perturbations():
    # a flip caused by moving every score by at most 3e-5 (well inside tol = 1e-4) must land
    # in the band: each golden row, all 3^M moves of its scores by -3e-5, 0 or +3e-5
    with open(os.path.join(GOLDEN, "ambiguity_band.json")) as f:
        g = json.load(f)
    for case in g["cases"]:
        base = _band_row(case)
        amb = O.ambiguous_blocks(base, g["tol"])[0, 0, 0]
        s0 = np.array(case["scores"], np.float64)
        hist = np.array(case["hist"])
        keep0 = np.zeros(case["NK"], bool)
        keep0[hist[base["rows"][(0, 0, 0)]["selected"]]] = True
        for moves in itertools.product((-3e-5, 0.0, 3e-5), repeat=s0.size):
            s1 = s0 + np.array(moves)
            row = O.select_tau_row(s1, case["tau"]) if "tau" in case else O.select_topk_row(s1, case["r"])
            keep1 = np.zeros(case["NK"], bool)
            keep1[hist[row["selected"]]] = True
            assert not ((keep1 != keep0) & ~amb).any(), (case["name"], moves)


ALL_PINS = [pin_bf16_decode, pin_partition, pin_pool_closed_form, pin_scores_closed_form,
            pin_softmax_properties, pin_tau_brute_force, pin_topk_brute_force, pin_golden_hand_worked,
            pin_attention_dense_matches_library, pin_attention_sparse_matches_library,
            pin_attention_frame_causal_matches_library, pin_attention_invariants,
            pin_permutation_invariance, pin_kept_flops, pin_ambiguity_band_golden,
            pin_ambiguity_band_covers_perturbations]


@pytest.mark.parametrize("pin", ALL_PINS, ids=[p.__name__ for p in ALL_PINS])
def test_pin(pin):
    pin()


# ---------------------------------------------------------------------------
# generator + oracle together, on the tiny configuration

def test_tiny_config_structure():
    # each query block copies one context block's centroid: that block dominates the pooled
    # scores, so every row keeps exactly 1 historical block plus the 4 chunk blocks
    wl = WORKLOADS["tiny"]
    inp = make_inputs(wl)
    sel = O.select_blocks(inp["q"], inp["k"], wl.block, tau=wl.tau)
    m = sel["mask"]
    assert m.shape == (1, 2, 4, 16)
    assert (m[..., 12:] == 1).all()
    assert (m[..., :12].sum(-1) == 1).all()
    assert not O.ambiguous_blocks(sel).any()


def test_ambiguity_band_flags_crossing():
    # C_1 = 0.5 exactly with two equal scores: the tie and tau crossings are flagged
    s = np.array([[[[2.0, 2.0, -30.0]]]])
    sel = {"scores": s, "part": {"hist": np.arange(3), "NK": 3}, "tau": 0.5,
           "rows": {(0, 0, 0): O.select_tau_row(s[0, 0, 0], 0.5)}}
    amb = O.ambiguous_blocks(sel)
    assert amb[0, 0, 0].tolist() == [True, True, False]
    s2 = np.array([[[[5.0, 0.0, -1.0]]]])
    sel2 = {"scores": s2, "part": {"hist": np.arange(3), "NK": 3}, "tau": 0.9,
            "rows": {(0, 0, 0): O.select_tau_row(s2[0, 0, 0], 0.9)}}
    assert not O.ambiguous_blocks(sel2).any()
