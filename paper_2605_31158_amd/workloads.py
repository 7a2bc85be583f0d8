"""Seeded synthetic inputs for AR chunk attention (query chunk vs. long K/V context).

This module only draws numbers: it holds none of the method's arithmetic (no
pooling, scoring, selection or attention).  It is the one piece shared by the
GPU path's tests and bench and by the fp64 oracle's tests.

Shapes follow the paper's autoregressive setting (Sec. 3.3, "Autoregressive
Adaptation"; Sec. 4.1 "Models"): a chunk of Lq query tokens (the frames being
denoised) attends to Lk keys laid out as
[text tokens][historical visual context][current chunk], and the chunk's own
tokens are the last Lq keys.  The latent grids are those of the evaluated
models: 30x52 = 1560 tokens per latent frame at 480P and 45x80 = 3600 at 720P.
The paper's model activations are not available; these draws stand in for
them (the recipe is written out in `make_inputs`).

All tensors are returned as numpy uint16 arrays holding bfloat16 bit patterns
(round-to-nearest-even from float32), layout [B, H, L, d] contiguous.
"""
from __future__ import annotations

import dataclasses
import math
from concurrent.futures import ThreadPoolExecutor
from typing import Dict, Optional

import numpy as np

__all__ = ["Workload", "WORKLOADS", "make_inputs", "make_clustered", "f32_to_bf16_bits",
           "frame_slot_tables_size", "Workload3D", "WORKLOADS_3D", "make_inputs_3d"]


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic AR-chunk attention problem.

    kind selects the centroid structure (see `make_inputs`); frame_tokens is
    the number of tokens per latent frame used by the centroid structure, and
    causal_frames switches on the frame-causal mask inside the chunk (query
    frame f sees chunk frames <= f).
    """
    name: str
    kind: str
    B: int
    H: int
    d: int
    Lq: int
    Lk: int
    block: int
    tau: float
    seed: int
    frame_tokens: int = 0
    causal_frames: bool = False
    n_text: int = 0

    @property
    def nq(self) -> int:
        return -(-self.Lq // self.block)

    @property
    def nk(self) -> int:
        return -(-self.Lk // self.block)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


F480 = 30 * 52   # tokens per latent frame, 480P
F720 = 45 * 80   # tokens per latent frame, 720P

WORKLOADS: Dict[str, Workload] = {
    # 4 query blocks over 16 key blocks; each query block copies one context block's centroid.
    "tiny": Workload("tiny", "tiny", 1, 2, 64, 256, 1024, 64, 0.9, 0),
    # 480P, 4-frame chunk, 8-frame temporal window.
    "480p_window": Workload("480p_window", "walk", 1, 16, 128, 4 * F480, 12 * F480, 64, 0.9, 1,
                            frame_tokens=F480),
    # 480P, 16 retrieved memory frames + 8-frame window.
    "480p_memory": Workload("480p_memory", "memory", 1, 16, 128, 4 * F480, 28 * F480, 64, 0.9, 2,
                            frame_tokens=F480),
    # 720P, 12 unrelated + 4 related context frames, block 128.
    "720p": Workload("720p", "related720", 1, 24, 128, 4 * F720, 20 * F720, 128, 0.85, 3,
                     frame_tokens=F720),
    # 480P long trajectory: 64 context frames drawn from 8 revisited-region clusters.
    "480p_long": Workload("480p_long", "clusters", 1, 16, 128, 4 * F480, 68 * F480, 64, 0.9, 4,
                          frame_tokens=F480),
}
WORKLOADS["720p_causal"] = WORKLOADS["720p"].replace(name="720p_causal", causal_frames=True)
WORKLOADS["480p_long_dense"] = WORKLOADS["480p_long"].replace(name="480p_long_dense", tau=1.0)

# The five configurations in the order they are listed for this workload family.
CONFIG_ORDER = ["tiny", "480p_window", "480p_memory", "720p", "480p_long"]


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit pattern, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).copy()
    bias = (u >> 16) & 1
    bias += 0x7FFF
    u += bias
    u >>= 16
    return u.astype(np.uint16)


def frame_slot_tables_size(frame_tokens: int, block: int) -> int:
    """Number of block slots a per-frame centroid table needs."""
    return -(-frame_tokens // block) + 1


def _frame_slot(j: np.ndarray, block: int, F: int):
    """Frame of key block j (frame holding its first token) and its slot inside that frame."""
    f = (j * block) // F
    r = j - (f * F + block - 1) // block
    return f, r


def _tables_for_kind(wl: Workload, rng: np.random.Generator, n_frames: int, S: int) -> np.ndarray:
    """Per-frame slot tables [n_frames, S, d] (float32) for one head."""
    d = wl.d
    n_chunk = wl.Lq // wl.frame_tokens
    n_ctx = n_frames - n_chunk
    std = lambda *shape: rng.standard_normal(shape, dtype=np.float32)
    if wl.kind == "walk":
        # One random walk over all frames: context then chunk.
        t = np.empty((n_frames, S, d), np.float32)
        t[0] = std(S, d)
        for f in range(1, n_frames):
            t[f] = t[f - 1] + np.float32(0.2) * std(S, d)
        return t
    if wl.kind == "memory":
        # 16 retrieved-memory frames, then a 12-frame walk (8 window + 4 chunk).
        n_mem = n_ctx - 8
        walk = np.empty((8 + n_chunk, S, d), np.float32)
        walk[0] = std(S, d)
        for f in range(1, walk.shape[0]):
            walk[f] = walk[f - 1] + np.float32(0.2) * std(S, d)
        mem = std(n_mem, S, d)
        related = rng.choice(n_mem, size=3, replace=False)
        src = rng.integers(0, n_chunk, size=3)
        for m, c in zip(related, src):
            mem[m] = walk[8 + c]
        return np.concatenate([mem, walk], axis=0)
    if wl.kind == "related720":
        # 12 unrelated context frames, then 4 window frames walking into the 4 chunk frames.
        n_unrel = n_ctx - 4
        unrel = std(n_unrel, S, d)
        walk = np.empty((4 + n_chunk, S, d), np.float32)
        walk[0] = std(S, d)
        for f in range(1, walk.shape[0]):
            walk[f] = walk[f - 1] + np.float32(0.2) * std(S, d)
        return np.concatenate([unrel, walk], axis=0)
    if wl.kind == "clusters":
        # 8 revisited-region cluster tables; each context frame is a noisy copy of one of them.
        C = std(8, S, d)
        assign = rng.permutation(np.repeat(np.arange(8), n_ctx // 8))
        ctx = C[assign] + np.float32(0.2) * std(n_ctx, S, d)
        a, b = rng.choice(8, size=2, replace=False)
        chunk = np.empty((n_chunk, S, d), np.float32)
        for f in range(n_chunk):
            base = C[a] if f < n_chunk // 2 else C[b]
            chunk[f] = base + np.float32(0.2) * std(S, d)
        return np.concatenate([ctx, chunk], axis=0)
    raise ValueError(f"unknown workload kind {wl.kind!r}")


def _head_centroids(wl: Workload, rng: np.random.Generator):
    """Centroid per key block [NK, d] and per query block [NQ, d] for one head."""
    b, NK, NQ = wl.block, wl.nk, wl.nq
    if wl.kind == "tiny":
        kc = rng.standard_normal((NK, wl.d), dtype=np.float32)
        n_hist = (wl.Lk - wl.Lq) // b
        pick = rng.integers(0, n_hist, size=NQ)
        qc = kc[pick].copy()
        return kc, qc
    F = wl.frame_tokens
    assert wl.Lk % F == 0 and wl.Lq % F == 0 and (wl.Lk - wl.Lq) % b == 0
    n_frames = wl.Lk // F
    S = frame_slot_tables_size(F, b)
    tables = _tables_for_kind(wl, rng, n_frames, S)
    j = np.arange(NK)
    f, r = _frame_slot(j, b, F)
    kc = tables[f, r]
    j0 = (wl.Lk - wl.Lq) // b        # first chunk block; the chunk starts block-aligned
    qc = kc[j0:j0 + NQ].copy()
    return kc, qc


def make_inputs(wl: Workload, threads: int = 8) -> Dict[str, np.ndarray]:
    """Draw q, k, v (bf16 bit patterns, [B, H, L, d]) for a workload.

    Recipe, per (batch, head) pair, from its own child of SeedSequence(seed):
      1. centroid structure (`kind`): a centroid per key block and per query block;
         query block i uses the centroid of chunk key block i, so the chunk's keys
         and queries share centroids;
      2. keys: k_n = centroid(block of n) + 0.5 * N(0, I_d);
      3. queries: q_t = centroid(query block of t) + 0.5 * N(0, I_d);
      4. values: v_n ~ N(0, I_d), independent of everything else.
    Float32 arithmetic, then round-to-nearest-even to bfloat16.
    """
    B, H, d = wl.B, wl.H, wl.d
    q = np.empty((B, H, wl.Lq, d), np.uint16)
    k = np.empty((B, H, wl.Lk, d), np.uint16)
    v = np.empty((B, H, wl.Lk, d), np.uint16)
    seeds = np.random.SeedSequence(wl.seed).spawn(B * H)
    kblk = np.minimum(np.arange(wl.Lk) // wl.block, wl.nk - 1)
    qblk = np.arange(wl.Lq) // wl.block

    def one(bh: int):
        bi, hi = divmod(bh, H)
        rng = np.random.default_rng(seeds[bh])
        kc, qc = _head_centroids(wl, rng)
        kn = rng.standard_normal((wl.Lk, d), dtype=np.float32)
        kn *= np.float32(0.5)
        kn += kc[kblk]
        k[bi, hi] = f32_to_bf16_bits(kn)
        del kn
        qn = rng.standard_normal((wl.Lq, d), dtype=np.float32)
        qn *= np.float32(0.5)
        qn += qc[qblk]
        q[bi, hi] = f32_to_bf16_bits(qn)
        vn = rng.standard_normal((wl.Lk, d), dtype=np.float32)
        v[bi, hi] = f32_to_bf16_bits(vn)

    if threads > 1 and B * H > 1:
        with ThreadPoolExecutor(min(threads, B * H)) as ex:
            list(ex.map(one, range(B * H)))
    else:
        for bh in range(B * H):
            one(bh)
    return {"q": q, "k": k, "v": v}


def make_spread(B: int, H: int, Lq: int, Lk: int, d: int, block: int, seed: int,
                sigma: float = 5.0, noise: float = 0.5) -> Dict[str, np.ndarray]:
    """Inputs whose block scores spread evenly, with no dominant block: independent N(0, I)
    centroids for every key block and every query block (no query copies a key block), scaled by
    sqrt(sigma) on both sides, plus 0.5 N(0, I) token noise before scaling.  The scores of a row
    are then roughly N(0, sigma^2), so the softmax mass thins out gradually over many blocks and
    a tau close to 1 cuts deep into a long tail of small masses."""
    rng = np.random.default_rng(seed)
    NK, NQ = -(-Lk // block), -(-Lq // block)
    a = np.float32(math.sqrt(sigma))
    q = np.empty((B, H, Lq, d), np.uint16)
    k = np.empty((B, H, Lk, d), np.uint16)
    v = np.empty((B, H, Lk, d), np.uint16)
    kblk = np.minimum(np.arange(Lk) // block, NK - 1)
    qblk = np.arange(Lq) // block
    for bi in range(B):
        for hi in range(H):
            kc = rng.standard_normal((NK, d), dtype=np.float32)
            qc = rng.standard_normal((NQ, d), dtype=np.float32)
            kn = kc[kblk] + np.float32(noise) * rng.standard_normal((Lk, d), dtype=np.float32)
            qn = qc[qblk] + np.float32(noise) * rng.standard_normal((Lq, d), dtype=np.float32)
            k[bi, hi] = f32_to_bf16_bits(kn * a)
            q[bi, hi] = f32_to_bf16_bits(qn * a)
            v[bi, hi] = f32_to_bf16_bits(rng.standard_normal((Lk, d), dtype=np.float32))
    return {"q": q, "k": k, "v": v}


def make_clustered(B: int, H: int, Lq: int, Lk: int, d: int, block: int, seed: int,
                   n_text: int = 0, noise: float = 0.5, scale: float = 1.0,
                   v_kind: str = "normal") -> Dict[str, np.ndarray]:
    """Small generic inputs: one centroid per key block; each query block copies the
    centroid of a random non-chunk key block (or its own chunk block when there is none).

    `scale` multiplies centroids and noise (larger scale -> peakier block scores).
    v_kind: "normal" (N(0,1)), "ones" (all 1.0) or "index" (v[n, c] = small exact
    integers depending on n and c, useful for exact checks).
    """
    rng = np.random.default_rng(seed)
    NK, NQ = -(-Lk // block), -(-Lq // block)
    q = np.empty((B, H, Lq, d), np.uint16)
    k = np.empty((B, H, Lk, d), np.uint16)
    v = np.empty((B, H, Lk, d), np.uint16)
    n_cand = max((Lk - Lq) // block, 0)
    kblk = np.minimum(np.arange(Lk) // block, NK - 1)
    qblk = np.arange(Lq) // block
    for bi in range(B):
        for hi in range(H):
            kc = rng.standard_normal((NK, d), dtype=np.float32)
            if n_cand > 0:
                pick = rng.integers(0, n_cand, size=NQ)
            else:
                pick = np.minimum(np.arange(NQ) + (Lk - Lq) // block, NK - 1)
            qc = kc[pick]
            kn = (kc[kblk] + np.float32(noise) * rng.standard_normal((Lk, d), dtype=np.float32))
            qn = (qc[qblk] + np.float32(noise) * rng.standard_normal((Lq, d), dtype=np.float32))
            k[bi, hi] = f32_to_bf16_bits(kn * np.float32(scale))
            q[bi, hi] = f32_to_bf16_bits(qn * np.float32(scale))
            if v_kind == "normal":
                vn = rng.standard_normal((Lk, d), dtype=np.float32)
            elif v_kind == "ones":
                vn = np.ones((Lk, d), np.float32)
            elif v_kind == "index":
                vn = ((np.arange(Lk)[:, None] * 7 + np.arange(d)[None, :] * 3) % 17 - 8).astype(np.float32)
            else:
                raise ValueError(v_kind)
            v[bi, hi] = f32_to_bf16_bits(vn)
    return {"q": q, "k": k, "v": v}


# ------------------------------------------------------------------------------------------------
# 3-D block layout workloads (Sec. 3.3; block extents of the evaluated models: (4, 8, 4) on the
# 30x52 latent grid, (4, 4, 8) on the 45x80 grid, 128 tokens per block)

@dataclasses.dataclass(frozen=True)
class Workload3D:
    """One AR chunk in linear order: n_text text keys, T_ctx context frames, T_q chunk frames of
    Hs x Ws tokens; blocks of bt x bh x bw tokens in `block` slots.  Context structure: the last
    `window` context frames walk into the chunk frames (step 0.2); `n_related` of the earlier
    frames copy a chunk frame's field; the other earlier frames are unrelated."""
    name: str
    B: int
    H: int
    d: int
    n_text: int
    T_ctx: int
    T_q: int
    Hs: int
    Ws: int
    bt: int
    bh: int
    bw: int
    block: int
    seed: int
    window: int
    n_related: int
    tau: Optional[float] = None       # cumulative-mass rule, or
    topk_r: Optional[float] = None    # the Top-floor(rM) rule with retained fraction r

    @property
    def frame_tokens(self) -> int:
        return self.Hs * self.Ws

    @property
    def Lq(self) -> int:
        return self.T_q * self.frame_tokens

    @property
    def Lk(self) -> int:
        return self.n_text + (self.T_ctx + self.T_q) * self.frame_tokens

    def replace(self, **kw) -> "Workload3D":
        return dataclasses.replace(self, **kw)


WORKLOADS_3D: Dict[str, Workload3D] = {
    # ragged everywhere: 24-token blocks in 64 slots, frames and text not block multiples
    "tiny_3d": Workload3D("tiny_3d", 1, 2, 64, 40, 6, 3, 7, 10, 2, 3, 4, 64, 10, 2, 1, tau=0.9),
    # 480P latents (30x52), (4, 8, 4) blocks: 16 memory frames (3 related) + 8 window frames; the
    # retained fraction 17.5% of the evaluated 480P model
    "480p_3d": Workload3D("480p_3d", 1, 16, 128, 300, 24, 4, 30, 52, 4, 8, 4, 128, 11, 8, 3, topk_r=0.175),
    # 720P latents (45x80), (4, 4, 8) blocks: 12 unrelated + 4 window frames
    "720p_3d": Workload3D("720p_3d", 1, 24, 128, 0, 16, 4, 45, 80, 4, 4, 8, 128, 12, 4, 0, topk_r=0.175),
}


def _region_fields(wl: Workload3D, rng: np.random.Generator) -> np.ndarray:
    """Centroid fields [T_ctx + T_q, ceil(Hs/bh), ceil(Ws/bw), d] (float32) for one head: one
    centroid per region of bh x bw tokens of a frame."""
    ry, rx = -(-wl.Hs // wl.bh), -(-wl.Ws // wl.bw)
    std = lambda *shape: rng.standard_normal(shape, dtype=np.float32)
    n_walk = min(wl.window, wl.T_ctx) + wl.T_q
    walk = np.empty((n_walk, ry, rx, wl.d), np.float32)
    walk[0] = std(ry, rx, wl.d)
    for f in range(1, n_walk):
        walk[f] = walk[f - 1] + np.float32(0.2) * std(ry, rx, wl.d)
    n_early = wl.T_ctx - min(wl.window, wl.T_ctx)
    early = std(n_early, ry, rx, wl.d)
    if n_early > 0 and wl.n_related > 0:
        rel = rng.choice(n_early, size=min(wl.n_related, n_early), replace=False)
        src = rng.integers(0, wl.T_q, size=rel.size)
        for m, c in zip(rel, src):
            early[m] = walk[n_walk - wl.T_q + c]
    return np.concatenate([early, walk], axis=0)


def make_inputs_3d(wl: Workload3D, threads: int = 8) -> Dict[str, np.ndarray]:
    """Draw q, k, v (bf16 bit patterns, linear order [B, H, L, d]) for a 3-D workload.

    Recipe, per (batch, head) pair, from its own child of SeedSequence(seed):
      1. centroid fields (`_region_fields`), one centroid per bh x bw region of each frame;
      2. keys: text k_n ~ N(0, I_d); visual k = centroid(frame, region) + 0.5 * N(0, I_d);
      3. queries (chunk frames): centroid(frame, region) + 0.5 * N(0, I_d);
      4. values: v_n ~ N(0, I_d), independent of everything else.
    Float32 arithmetic, then round-to-nearest-even to bfloat16.
    """
    B, H, d, F = wl.B, wl.H, wl.d, wl.frame_tokens
    q = np.empty((B, H, wl.Lq, d), np.uint16)
    k = np.empty((B, H, wl.Lk, d), np.uint16)
    v = np.empty((B, H, wl.Lk, d), np.uint16)
    seeds = np.random.SeedSequence(wl.seed).spawn(B * H)
    ys, xs = np.divmod(np.arange(F), wl.Ws)
    reg_y, reg_x = ys // wl.bh, xs // wl.bw
    nf = wl.T_ctx + wl.T_q

    def one(bh: int):
        bi, hi = divmod(bh, H)
        rng = np.random.default_rng(seeds[bh])
        fields = _region_fields(wl, rng)
        cent = fields[:, reg_y, reg_x, :].reshape(nf * F, d)
        kn = rng.standard_normal((wl.Lk, d), dtype=np.float32)
        kn *= np.float32(0.5)
        kn[wl.n_text:] += cent
        kn[:wl.n_text] *= np.float32(2.0)
        k[bi, hi] = f32_to_bf16_bits(kn)
        del kn
        qn = rng.standard_normal((wl.Lq, d), dtype=np.float32)
        qn *= np.float32(0.5)
        qn += cent[wl.T_ctx * F:]
        q[bi, hi] = f32_to_bf16_bits(qn)
        v[bi, hi] = f32_to_bf16_bits(rng.standard_normal((wl.Lk, d), dtype=np.float32))

    if threads > 1 and B * H > 1:
        with ThreadPoolExecutor(min(threads, B * H)) as ex:
            list(ex.map(one, range(B * H)))
    else:
        for bh in range(B * H):
            one(bh)
    return {"q": q, "k": k, "v": v}
