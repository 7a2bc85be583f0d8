"""Plain fp64 NumPy oracle for the AR block-sparse attention path of Light Interaction
(Sec. 3.3).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the bench's
CPU-baseline leg, never by the GPU library.  Slow on purpose: every step is the
definition written out, one (batch, head, query block) at a time.

Steps, in the paper's order and notation:
  * blocks: query blocks Q_i and key blocks K_m of `block` consecutive tokens
    (1-D blocks, as the benchmark configurations use; the 3-D blocks of the paper
    are the second section below);
  * pooled proxies q_bar_i and k_bar_m: means over each block's tokens
    (Sec. 3.3, pooling equation);
  * relevance s_{i,m} = q_bar_i . k_bar_m / sqrt(d) over the M historical blocks
    only (Sec. 3.3, Top-k selection equation);
  * selection of the retained historical set S_i: the paper's Top-floor(rM) rule,
    and the cumulative-mass rule used by the benchmark configurations (keep the
    shortest highest-scoring prefix whose softmax mass reaches tau);
  * context C_i = T u K^curr u S_i: text blocks and current-chunk blocks always
    kept (Sec. 3.3, context-union equation); one index set serves K and V;
  * attention over C_i: softmax(q K_C^T * scale) V_C per query token.

Readings where the paper is silent (each is listed in the design notes too):
  * the tau softmax runs over the M historical candidates only, at the paper's
    score scale 1/sqrt(d); ties in score are ordered by lower block index;
    k* = min{k >= 1 : C_k >= tau}; tau >= 1 keeps all M; M = 0 selects nothing;
  * floor(rM) = 0 selects no historical block;
  * a block overlapping the text region [0, n_text) or the chunk [Lk-Lq, Lk) is
    forced (always kept, never scored); ragged blocks pool over valid tokens;
  * optional frame-causal mask inside the chunk: query frame f sees chunk frames
    <= f; the whole context stays visible (subject to block selection);
  * a query token with no visible key gets o = 0 and lse = -inf.

A second section builds the same steps over 3-D (B_t, B_h, B_w) blocks given as token sets
(Sec. 3.3 and the appendix's block sizes), and a third holds the scalar policy around the
path: latent dynamics, its moving average and the temporal window (Sec. 3.1), the
pose-similarity gate (Sec. 3.1) and the denoising-cache schedule (Sec. 3.2).

Parity pins live in tests/test_oracle.py, tests/test_oracle_3d.py and
tests/test_oracle_policy.py (closed forms, brute force, library attention, invariants);
nothing here is checked against itself.
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import numpy as np


# ---------------------------------------------------------------------------
# inputs

def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> exact float64 values."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def _as_f64(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_bits_to_f64(x)
    return x.astype(np.float64)


# ---------------------------------------------------------------------------
# blocks (Sec. 3.3: Q_i, K_m; context union C_i = T u K^curr u S_i)

def partition(Lq: int, Lk: int, block: int, n_text: int = 0) -> Dict[str, object]:
    """Block counts, the forced key blocks (text u current chunk) and the historical ones.

    Key block m covers tokens [m*block, min((m+1)*block, Lk)).  It is forced when it
    overlaps the text tokens [0, n_text) or the current chunk [Lk-Lq, Lk).
    """
    NQ = -(-Lq // block)
    NK = -(-Lk // block)
    forced = np.zeros(NK, dtype=bool)
    chunk_start = Lk - Lq
    for m in range(NK):
        lo, hi = m * block, min((m + 1) * block, Lk)
        if lo < n_text:
            forced[m] = True
        if hi > chunk_start:
            forced[m] = True
    hist = np.array([m for m in range(NK) if not forced[m]], dtype=np.int64)
    return {"NQ": NQ, "NK": NK, "forced": forced, "hist": hist, "M": int(hist.size)}


def pool_blocks(x: np.ndarray, block: int) -> np.ndarray:
    """Pooled proxy of every block: mean over its tokens (Sec. 3.3, pooling equation).

    x: [..., L, d] -> [..., ceil(L/block), d].  A ragged last block averages over its
    valid tokens only (|Q_i| is the count of tokens in the block).
    """
    x = _as_f64(x)
    L = x.shape[-2]
    nb = -(-L // block)
    out = np.empty(x.shape[:-2] + (nb, x.shape[-1]), dtype=np.float64)
    for i in range(nb):
        lo, hi = i * block, min((i + 1) * block, L)
        total = np.zeros(x.shape[:-2] + (x.shape[-1],), dtype=np.float64)
        for t in range(lo, hi):
            total = total + x[..., t, :]
        out[..., i, :] = total / (hi - lo)
    return out


def block_scores(qbar: np.ndarray, kbar: np.ndarray, d: Optional[int] = None) -> np.ndarray:
    """s_{i,m} = q_bar_i^T k_bar_m / sqrt(d) (Sec. 3.3, selection equation).

    qbar: [..., NQ, d], kbar: [..., M, d] -> [..., NQ, M].
    """
    if d is None:
        d = qbar.shape[-1]
    return np.matmul(qbar, np.swapaxes(kbar, -1, -2)) / math.sqrt(d)


# ---------------------------------------------------------------------------
# selection of the retained historical set S_i

def softmax_rows(s: np.ndarray) -> np.ndarray:
    """Row softmax in fp64, max-subtracted."""
    s = np.asarray(s, dtype=np.float64)
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def _order(s_row: np.ndarray) -> np.ndarray:
    """Candidate positions by score descending, lower position first on ties."""
    pos = np.arange(s_row.size)
    return np.lexsort((pos, -s_row))


def select_tau_row(s_row: np.ndarray, tau: float) -> Dict[str, object]:
    """Cumulative-mass rule for one query block.

    p = softmax(s) over the M candidates; pi = candidates by score descending;
    C_k = p_pi(1) + ... + p_pi(k), summed in that order;
    k* = min{k >= 1 : C_k >= tau} (all M when tau >= 1 or when the sum never reaches tau);
    S_i = {pi(1), ..., pi(k*)}.  Returns positions into the candidate list.
    """
    M = s_row.size
    if M == 0:
        return {"order": np.zeros(0, np.int64), "kstar": 0, "cum": np.zeros(0), "p": np.zeros(0),
                "selected": np.zeros(0, np.int64)}
    p = softmax_rows(s_row)
    order = _order(s_row)
    cum = np.zeros(M, dtype=np.float64)
    running = 0.0
    for r in range(M):
        running = running + p[order[r]]
        cum[r] = running
    if tau >= 1.0:
        kstar = M
    else:
        kstar = M
        for r in range(M):
            if cum[r] >= tau:
                kstar = r + 1
                break
    return {"order": order, "kstar": kstar, "cum": cum, "p": p,
            "selected": np.sort(order[:kstar])}


def select_topk_row(s_row: np.ndarray, r: float) -> Dict[str, object]:
    """Paper's rule: the floor(r*M) highest scores (Sec. 3.3, Top-floor(rM) equation)."""
    M = s_row.size
    kstar = int(math.floor(r * M + 1e-9)) if M > 0 else 0
    kstar = max(0, min(kstar, M))
    order = _order(s_row) if M > 0 else np.zeros(0, np.int64)
    return {"order": order, "kstar": kstar, "selected": np.sort(order[:kstar])}


def select_blocks(q: np.ndarray, k: np.ndarray, block: int, tau: Optional[float] = None,
                  n_text: int = 0, topk_r: Optional[float] = None) -> Dict[str, object]:
    """Block mask [B, H, NQ, NK] (uint8) for the whole problem, plus the intermediate values.

    Exactly one of tau (cumulative-mass rule) and topk_r (paper's Top-floor(rM) rule).
    q: [B, H, Lq, d], k: [B, H, Lk, d] (bf16 bits or floats).
    """
    if (tau is None) == (topk_r is None):
        raise ValueError("give exactly one of tau and topk_r")
    q = _as_f64(q)
    k = _as_f64(k)
    B, H, Lq, d = q.shape
    Lk = k.shape[2]
    part = partition(Lq, Lk, block, n_text)
    NQ, NK, hist, forced = part["NQ"], part["NK"], part["hist"], part["forced"]
    qbar = pool_blocks(q, block)                         # [B, H, NQ, d]
    kbar_all = pool_blocks(k, block)                     # [B, H, NK, d]
    kbar = kbar_all[:, :, hist, :]                       # historical blocks only
    s = block_scores(qbar, kbar, d)                      # [B, H, NQ, M]
    mask = np.zeros((B, H, NQ, NK), dtype=np.uint8)
    rows = {}
    for b in range(B):
        for h in range(H):
            for i in range(NQ):
                if tau is not None:
                    sel = select_tau_row(s[b, h, i], tau)
                else:
                    sel = select_topk_row(s[b, h, i], topk_r)
                rows[(b, h, i)] = sel
                mask[b, h, i, forced] = 1
                mask[b, h, i, hist[sel["selected"]]] = 1
    return {"mask": mask, "scores": s, "qbar": qbar, "kbar": kbar, "rows": rows,
            "part": part, "tau": tau, "topk_r": topk_r}


def ambiguous_blocks(sel: Dict[str, object], tol: float = 1e-4) -> np.ndarray:
    """Key blocks whose kept/dropped status a correct fp32 evaluation may flip.

    For the tau rule, with s* the score of the last kept candidate pi(k*):
      * when another candidate scores within tol of s*: every candidate within tol of s*;
      * pi(k*) when dropping it leaves the mass within tol of tau (tau - C_{k*-1} <= tol);
      * pi(k*+1) when the kept mass exceeds tau by at most tol (C_{k*} - tau <= tol).
    For the top-k rule: when the last kept and first dropped scores are within tol,
    every candidate scoring in [s_first_dropped - tol, s_last_kept + tol].
    Forced blocks are never ambiguous.  Returns bool [B, H, NQ, NK].
    """
    s = sel["scores"]
    part = sel["part"]
    hist = part["hist"]
    B, H, NQ, M = s.shape
    amb = np.zeros((B, H, NQ, part["NK"]), dtype=bool)
    for (b, h, i), row in sel["rows"].items():
        order, kstar = row["order"], row["kstar"]
        sr = s[b, h, i]
        flag = np.zeros(M, dtype=bool)
        if M == 0:
            continue
        if sel["tau"] is not None:
            if sel["tau"] >= 1.0:
                continue
            last = order[kstar - 1]
            near = np.abs(sr - sr[last]) <= tol
            if near.sum() > 1:
                flag |= near
            cum = row["cum"]
            before = cum[kstar - 2] if kstar >= 2 else 0.0
            if sel["tau"] - before <= tol:
                flag[last] = True
            if kstar < M and cum[kstar - 1] - sel["tau"] <= tol:
                flag[order[kstar]] = True
        else:
            if 0 < kstar < M:
                lo_kept, hi_dropped = sr[order[kstar - 1]], sr[order[kstar]]
                if lo_kept - hi_dropped <= tol:
                    flag |= (sr >= hi_dropped - tol) & (sr <= lo_kept + tol)
        amb[b, h, i, hist[flag]] = True
    return amb


# ---------------------------------------------------------------------------
# attention over C_i

def visible_keys(t: int, Lq: int, Lk: int, frame_tokens: int = 0) -> np.ndarray:
    """bool [Lk]: keys query token t (chunk position 0..Lq-1) may see before block selection.

    Without a frame-causal mask every key is visible.  With frame_tokens = F > 0,
    context keys (n < Lk - Lq) stay visible and chunk key n is visible iff its chunk
    frame (n - (Lk - Lq)) // F is <= the query's frame t // F.
    """
    vis = np.ones(Lk, dtype=bool)
    if frame_tokens > 0:
        c0 = Lk - Lq
        chunk_pos = np.arange(Lk - c0)
        vis[c0:] = (chunk_pos // frame_tokens) <= (t // frame_tokens)
    return vis


def attention_block(qb: np.ndarray, kc: np.ndarray, vc: np.ndarray, ok: np.ndarray,
                    scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """Masked softmax attention for a set of query rows over a set of candidate keys.

    qb: [nq, d]; kc, vc: [nc, d] (the keys of the kept blocks); ok: bool [nq, nc]
    (key visible to that query).  o_t = sum_n softmax_n(q_t . k_n * scale) v_n over
    the visible keys; lse_t = log sum_n exp(q_t . k_n * scale).  A row with no
    visible key gets o_t = 0 and lse_t = -inf.
    """
    nq = qb.shape[0]
    o = np.zeros((nq, vc.shape[1]), dtype=np.float64)
    lse = np.full(nq, -np.inf, dtype=np.float64)
    if kc.shape[0] == 0:
        return o, lse
    logits = (qb @ kc.T) * scale
    logits = np.where(ok, logits, -np.inf)
    has = ok.any(axis=1)
    mx = np.where(has, logits.max(axis=1), 0.0)
    w = np.where(ok, np.exp(logits - mx[:, None]), 0.0)
    den = w.sum(axis=1)
    safe = np.where(has, den, 1.0)
    o[has] = (w @ vc)[has] / safe[has, None]
    lse[has] = mx[has] + np.log(den[has])
    return o, lse


def _row_problem(mask, block, Lq, Lk, b, h, i, frame_tokens):
    """Query rows of block i, the tokens of its kept key blocks, and per-row visibility."""
    lo, hi = i * block, min((i + 1) * block, Lq)
    kept_tok = np.zeros(Lk, dtype=bool)
    for m in np.nonzero(mask[b, h, i])[0]:
        kept_tok[m * block:min((m + 1) * block, Lk)] = True
    cand = np.nonzero(kept_tok)[0]
    ok = np.empty((hi - lo, cand.size), dtype=bool)
    for r, t in enumerate(range(lo, hi)):
        ok[r] = visible_keys(t, Lq, Lk, frame_tokens)[cand]
    return lo, hi, cand, ok


def attention_rows(q, k, v, mask, block: int, rows: Iterable[Tuple[int, int, int]],
                   scale: Optional[float] = None, frame_tokens: int = 0):
    """Attention for selected (b, h, query block) triples only.

    Returns {(b, h, i): (o [rows_in_block, d], lse [rows_in_block])}.  Inputs may be bf16
    bits (converted per head on demand) or float arrays.
    """
    d = q.shape[-1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = {}
    cache = {}
    for (b, h, i) in rows:
        if (b, h) not in cache:
            cache = {(b, h): (_as_f64(q[b, h]), _as_f64(k[b, h]), _as_f64(v[b, h]))}
        qh, kh, vh = cache[(b, h)]
        lo, hi, cand, ok = _row_problem(mask, block, q.shape[2], k.shape[2], b, h, i, frame_tokens)
        out[(b, h, i)] = attention_block(qh[lo:hi], kh[cand], vh[cand], ok, scale)
    return out


def attention(q, k, v, mask, block: int, scale: Optional[float] = None,
              frame_tokens: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """Block-sparse attention over C_i for every query block: o [B, H, Lq, d], lse [B, H, Lq]."""
    B, H, Lq, d = q.shape
    NQ = -(-Lq // block)
    o = np.zeros((B, H, Lq, v.shape[-1]), dtype=np.float64)
    lse = np.zeros((B, H, Lq), dtype=np.float64)
    rows = [(b, h, i) for b in range(B) for h in range(H) for i in range(NQ)]
    res = attention_rows(q, k, v, mask, block, rows, scale, frame_tokens)
    for (b, h, i), (ob, lb) in res.items():
        lo = i * block
        o[b, h, lo:lo + ob.shape[0]] = ob
        lse[b, h, lo:lo + ob.shape[0]] = lb
    return o, lse


# ---------------------------------------------------------------------------
# work accounting

def kept_flops(mask: np.ndarray, Lq: int, Lk: int, block: int, d: int) -> int:
    """4*d * sum over kept (query block, key block) pairs of valid_q * valid_k.

    Counts the two matrix products (q k^T and p v) over kept blocks; exp/max not counted.
    """
    NQ, NK = mask.shape[-2], mask.shape[-1]
    nq_valid = np.array([min((i + 1) * block, Lq) - i * block for i in range(NQ)], dtype=np.int64)
    nk_valid = np.array([min((m + 1) * block, Lk) - m * block for m in range(NK)], dtype=np.int64)
    m = mask.reshape(-1, NQ, NK).astype(np.int64)
    return int(4 * d * np.einsum("xij,i,j->", m, nq_valid, nk_valid))


# ---------------------------------------------------------------------------
# 3-D blocks (Sec. 3.3: historical visual tokens partitioned into non-overlapping
# (B_t, B_h, B_w) blocks; text and current-chunk tokens always kept; the appendix's block
# sizes are (4, 8, 4) and (4, 4, 8), 128 tokens each)

def blocks_3d(T: int, Hs: int, Ws: int, bt: int, bh: int, bw: int, offset: int = 0) -> List[np.ndarray]:
    """Token positions of the 3-D blocks of a run of T frames of Hs x Ws visual tokens.

    Token (t, y, x) sits at offset + (t * Hs + y) * Ws + x (frames one after another, each in
    raster order).  Blocks come in raster order of their (t, y, x) block coordinates; a block
    at a grid edge holds the tokens that exist there.  Inside a block, tokens are listed in
    raster order.
    """
    out = []
    for t0 in range(0, T, bt):
        for y0 in range(0, Hs, bh):
            for x0 in range(0, Ws, bw):
                idx = [offset + (t * Hs + y) * Ws + x
                       for t in range(t0, min(t0 + bt, T))
                       for y in range(y0, min(y0 + bh, Hs))
                       for x in range(x0, min(x0 + bw, Ws))]
                out.append(np.array(idx, dtype=np.int64))
    return out


def layout_3d(n_text: int, T_ctx: int, T_q: int, Hs: int, Ws: int, bt: int, bh: int, bw: int,
              text_block: int) -> Dict[str, object]:
    """Blocks of one AR chunk with 3-D visual blocks.

    Keys, in linear order: n_text text tokens, T_ctx context frames, T_q chunk frames.  Key
    blocks: the text in 1-D blocks of text_block tokens, then the 3-D blocks of the context
    frames, then those of the chunk frames.  Text and chunk blocks are forced; the context
    blocks are the historical candidates.  Query blocks: the 3-D blocks of the chunk frames,
    as positions inside the chunk.
    """
    F = Hs * Ws
    ktext = [np.arange(s, min(s + text_block, n_text), dtype=np.int64) for s in range(0, n_text, text_block)]
    kctx = blocks_3d(T_ctx, Hs, Ws, bt, bh, bw, offset=n_text)
    kchunk = blocks_3d(T_q, Hs, Ws, bt, bh, bw, offset=n_text + T_ctx * F)
    ksets = ktext + kctx + kchunk
    forced = np.array([True] * len(ktext) + [False] * len(kctx) + [True] * len(kchunk), dtype=bool)
    qsets = blocks_3d(T_q, Hs, Ws, bt, bh, bw, offset=0)
    return {"qsets": qsets, "ksets": ksets, "forced": forced, "Lq": T_q * F,
            "Lk": n_text + (T_ctx + T_q) * F}


def pool_sets(x: np.ndarray, sets: Sequence[np.ndarray]) -> np.ndarray:
    """Pooled proxy of every block given by its token positions: the mean over them
    (Sec. 3.3, pooling equation).  x: [..., L, d] -> [..., len(sets), d]."""
    x = _as_f64(x)
    out = np.empty(x.shape[:-2] + (len(sets), x.shape[-1]), dtype=np.float64)
    for i, idx in enumerate(sets):
        total = np.zeros(x.shape[:-2] + (x.shape[-1],), dtype=np.float64)
        for t in idx:
            total = total + x[..., int(t), :]
        out[..., i, :] = total / len(idx)
    return out


def select_blocks_sets(q, k, qsets, ksets, forced, tau: Optional[float] = None,
                       topk_r: Optional[float] = None) -> Dict[str, object]:
    """Block selection with blocks given as token sets (the 3-D layout); same rules as
    select_blocks.  Returns the mask [B, H, NQ, NK] and the intermediate values, with a
    "part" entry shaped like partition()'s."""
    if (tau is None) == (topk_r is None):
        raise ValueError("give exactly one of tau and topk_r")
    q = _as_f64(q)
    k = _as_f64(k)
    B, H, _, d = q.shape
    NQ, NK = len(qsets), len(ksets)
    forced = np.asarray(forced, dtype=bool)
    hist = np.nonzero(~forced)[0].astype(np.int64)
    qbar = pool_sets(q, qsets)
    kbar = pool_sets(k, [ksets[int(m)] for m in hist])
    s = block_scores(qbar, kbar, d)
    mask = np.zeros((B, H, NQ, NK), dtype=np.uint8)
    rows = {}
    for b in range(B):
        for h in range(H):
            for i in range(NQ):
                sel = select_tau_row(s[b, h, i], tau) if tau is not None else select_topk_row(s[b, h, i], topk_r)
                rows[(b, h, i)] = sel
                mask[b, h, i, forced] = 1
                mask[b, h, i, hist[sel["selected"]]] = 1
    part = {"NQ": NQ, "NK": NK, "forced": forced, "hist": hist, "M": int(hist.size)}
    return {"mask": mask, "scores": s, "qbar": qbar, "kbar": kbar, "rows": rows, "part": part,
            "tau": tau, "topk_r": topk_r}


def attention_sets_rows(q, k, v, qsets, ksets, mask, rows: Iterable[Tuple[int, int, int]],
                        scale: Optional[float] = None):
    """Attention of the query tokens of block i over the tokens of its kept key blocks, for
    selected (b, h, i); every kept key is visible.  Returns {(b, h, i): (o [|Q_i|, d] in the
    order of qsets[i], lse [|Q_i|])}."""
    d = q.shape[-1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    out = {}
    cache = {}
    for (b, h, i) in rows:
        if (b, h) not in cache:
            cache = {(b, h): (_as_f64(q[b, h]), _as_f64(k[b, h]), _as_f64(v[b, h]))}
        qh, kh, vh = cache[(b, h)]
        kept = np.nonzero(mask[b, h, i])[0]
        cand = np.sort(np.concatenate([ksets[int(m)] for m in kept])) if kept.size else np.zeros(0, np.int64)
        qi = qsets[i]
        ok = np.ones((qi.size, cand.size), dtype=bool)
        out[(b, h, i)] = attention_block(qh[qi], kh[cand], vh[cand], ok, scale)
    return out


# ---------------------------------------------------------------------------
# Adaptive context management (Sec. 3.1) and the denoising cache (Sec. 3.2): the scalar policy
# around the attention path.  Camera-pose similarities are inputs (the paper instantiates them
# with an FOV overlap it does not define).

def latent_mse(z_prev: np.ndarray, z_prev2: np.ndarray) -> float:
    """D_t = MSE(z_{t-1}, z_{t-2}), the mean over every latent dimension of the squared
    difference of the two most recent stable units (Sec. 3.1, latent-dynamics equation).
    Arrays of one size (uint16 = bf16 bit patterns); the sum is exact (math.fsum)."""
    a = _as_f64(z_prev).ravel()
    b = _as_f64(z_prev2).ravel()
    if a.size != b.size or a.size == 0:
        raise ValueError("two non-empty latents of one size are needed")
    return math.fsum(((a - b) ** 2).tolist()) / a.size


def ema_dynamics(D_t: float, D_bar_prev: Optional[float], alpha: float) -> float:
    """D_bar_t = alpha D_t + (1 - alpha) D_bar_{t-1}, started by the first valid D_t
    (D_bar_prev None) (Sec. 3.1, smoothing equation); alpha in (0, 1]."""
    if not (0.0 < alpha <= 1.0):
        raise ValueError("alpha must lie in (0, 1]")
    if D_bar_prev is None:
        return float(D_t)
    return alpha * D_t + (1.0 - alpha) * D_bar_prev


def temporal_window(D_bar: float, kappa: float, L_m: int) -> int:
    """L_t = clip(floor(L_m kappa / (D_bar + kappa)), 1, L_m) (Sec. 3.1, window equation);
    kappa > 0, L_m >= 1, D_bar >= 0."""
    if not (kappa > 0.0) or L_m < 1 or not (D_bar >= 0.0):
        raise ValueError("kappa > 0, L_m >= 1 and D_bar >= 0 are needed")
    return int(min(max(math.floor(L_m * kappa / (D_bar + kappa)), 1), L_m))


def revisiting(similarities: Sequence[float], tau_pose: float) -> bool:
    """max_j S_pose(t, j) >= tau_pose: a reliable pose-aware reference exists (Sec. 3.1 gate
    and Sec. 3.2 reuse condition).  False (pure exploration) also when there is no candidate."""
    return len(similarities) > 0 and max(float(s) for s in similarities) >= tau_pose


def keep_retrieved_memory(similarities: Sequence[float], tau_pose: float) -> bool:
    """Retrieved spatial memory is kept unless the step is pure exploration, i.e. the largest
    similarity is below tau_pose (Sec. 3.1, retrieved-memory gate)."""
    return revisiting(similarities, tau_pose)


def model_calls(K: int, reuse: bool) -> List[bool]:
    """Which of the K denoising steps evaluate the model (Sec. 3.2): with reuse (revisiting)
    and K > 2, only the first and the last; steps 1..K-2 reuse the first output.  Otherwise
    every step."""
    if K < 1:
        raise ValueError("K >= 1")
    if not reuse or K <= 2:
        return [True] * K
    return [i == 0 or i == K - 1 for i in range(K)]


def reuse_source(K: int, reuse: bool) -> List[int]:
    """For each of the K steps, the step whose model output it uses: itself, or step 0 for
    the reused intermediate steps (Sec. 3.2, reuse equation)."""
    calls = model_calls(K, reuse)
    return [i if calls[i] else 0 for i in range(K)]
