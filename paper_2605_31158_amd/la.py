"""ctypes binding of libla (include/la.h): argument marshalling only.

Every step of selection and attention runs in the HIP kernels of libla.so; this
module checks tensor shapes, dtypes and devices, allocates outputs and the
workspace with torch, and passes raw device pointers and torch's current HIP
stream across the C ABI.  There is no fallback: a missing library or a non-GPU
tensor raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libla.so")

LA_OK, LA_ERR_ARG, LA_ERR_SHAPE, LA_ERR_WORKSPACE, LA_ERR_HIP = range(5)


class Shape(ctypes.Structure):
    """la_shape."""
    _fields_ = [(n, ctypes.c_int32) for n in ("B", "H", "Lq", "Lk", "d", "block", "n_text", "frame_tokens")]

    def __repr__(self):
        return "Shape(" + ", ".join(f"{n}={getattr(self, n)}" for n, _ in self._fields_) + ")"


class LaError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {status_string(status)} (status {status})")
        self.status = status


class Grid3D(ctypes.Structure):
    """la_grid3d: 3-D block layout of one AR chunk (text, context frames, chunk frames)."""
    _fields_ = [(n, ctypes.c_int32) for n in ("B", "H", "d", "n_text", "T_ctx", "T_q", "Hs", "Ws", "bt", "bh", "bw",
                                              "block")]

    def __repr__(self):
        return "Grid3D(" + ", ".join(f"{n}={getattr(self, n)}" for n, _ in self._fields_) + ")"


LA_PART_TEXT, LA_PART_CONTEXT, LA_PART_CHUNK, LA_PART_ALL = 1, 2, 4, 7

_lib = None
_P = ctypes.c_void_p
_SP = ctypes.POINTER(Shape)
_GP = ctypes.POINTER(Grid3D)

_SIGNATURES = {
    "la_workspace_bytes": (ctypes.c_size_t, [_SP]),
    "la_select_blocks": (ctypes.c_int, [_SP, _P, _P, ctypes.c_float, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_select_blocks_topk": (ctypes.c_int, [_SP, _P, _P, ctypes.c_int32, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_select_blocks_noalloc": (ctypes.c_int, [_SP, _P, _P, ctypes.c_float, _P, _P, _P, _P]),
    "la_sparse_attn_fwd": (ctypes.c_int, [_SP, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_sparse_attn_plan": (ctypes.c_int, [_SP, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_sparse_attn_run": (ctypes.c_int, [_SP, _P, _P, _P, ctypes.c_float, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_sparse_attn_merge": (ctypes.c_int, [_SP, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_sparse_attn_schedule": (ctypes.c_int, [_SP, _P, ctypes.c_size_t, _P, _P, _P, _P, _P, _P, _P]),
    "la_mask_to_list": (ctypes.c_int, [_SP, _P, _P, _P, _P]),
    "la_grid3d_shape": (ctypes.c_int, [_GP, _SP]),
    "la_grid3d_valid": (ctypes.c_int, [_GP, _P, _P]),
    "la_prep_q_3d": (ctypes.c_int, [_GP, _P, _P, _P, _P]),
    "la_prep_kv_3d": (ctypes.c_int, [_GP, _P, _P, ctypes.c_uint32, _P, _P, _P, _P]),
    "la_pool_blocks": (ctypes.c_int, [_SP, _P, ctypes.c_int32, _P, _P]),
    "la_select_pooled": (ctypes.c_int, [_SP, _P, _P, ctypes.c_float, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_select_pooled_topk": (ctypes.c_int, [_SP, _P, _P, ctypes.c_int32, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_sparse_attn_fwd_valid": (ctypes.c_int, [_SP, _P, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P,
                                                ctypes.c_size_t, _P]),
    "la_sparse_attn_plan_valid": (ctypes.c_int, [_SP, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_untile_o_3d": (ctypes.c_int, [_GP, _P, _P, _P, _P, _P]),
    "la_latent_mse": (ctypes.c_int, [_P, _P, ctypes.c_int64, ctypes.c_int32, _P, _P, ctypes.c_size_t, _P]),
    "la_dynamics_ema": (ctypes.c_int, [ctypes.c_double, _P, ctypes.c_double, _P]),
    "la_temporal_window": (ctypes.c_int, [ctypes.c_double, ctypes.c_double, ctypes.c_int32, _P]),
    "la_pose_revisiting": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_float, _P]),
    "la_denoise_schedule": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, _P]),
    "la_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "la_abi_version": (ctypes.c_int32, []),
}


def lib() -> ctypes.CDLL:
    """Loads libla.so (torch first, so the library binds to the HIP runtime torch loaded)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                               "(or python -m paper_2605_31158_amd.build)")
        h = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(h, name)
            fn.restype = res
            fn.argtypes = args
        _lib = h
    return _lib


def status_string(status: int) -> str:
    return lib().la_status_string(status).decode()


def make_shape(B, H, Lq, Lk, d, block, n_text=0, frame_tokens=0) -> Shape:
    return Shape(B, H, Lq, Lk, d, block, n_text, frame_tokens)


def workspace_bytes(shape: Shape) -> int:
    return int(lib().la_workspace_bytes(ctypes.byref(shape)))


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(t: torch.Tensor):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _check_qkv(name, t: torch.Tensor, B=None, H=None, d=None):
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise TypeError(f"{name} must be a GPU tensor")
    if t.dtype != torch.bfloat16 or t.dim() != 4 or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous bfloat16 [B, H, L, d] tensor")
    if (B is not None and t.shape[0] != B) or (H is not None and t.shape[1] != H) or \
            (d is not None and t.shape[3] != d):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, inconsistent with the other operands")


def _workspace(shape: Shape, device, ws: Optional[torch.Tensor]):
    need = workspace_bytes(shape)
    if need == 0 and ws is None:
        return None, 0
    if ws is None:
        ws = torch.empty(max(need, 256), dtype=torch.uint8, device=device)
    return ws, ws.numel()


def _call(fn: str, *args):
    st = getattr(lib(), fn)(*args)
    if st != LA_OK:
        raise LaError(fn, st)


def nblocks(L: int, block: int) -> int:
    return -(-L // block)


def select_blocks(q: torch.Tensor, k: torch.Tensor, block: int, tau: float, n_text: int = 0,
                  want_mask: bool = True, ws: Optional[torch.Tensor] = None,
                  out: Optional[Tuple[torch.Tensor, torch.Tensor, torch.Tensor]] = None):
    """Cumulative-mass block selection -> (mask uint8 [B,H,NQ,NK] or None, counts int32 [B,H,NQ],
    idx int32 [B,H,NQ,NK] ascending in the first counts[] slots)."""
    return _select("la_select_blocks", ctypes.c_float(tau), q, k, block, n_text, want_mask, ws, out)


def select_blocks_topk(q: torch.Tensor, k: torch.Tensor, block: int, keep_blocks: int, n_text: int = 0,
                       want_mask: bool = True, ws: Optional[torch.Tensor] = None,
                       out: Optional[Tuple[torch.Tensor, torch.Tensor, torch.Tensor]] = None):
    """Top-keep_blocks selection (the paper's Top-floor(rM) rule with keep_blocks = floor(r*M))."""
    return _select("la_select_blocks_topk", ctypes.c_int32(keep_blocks), q, k, block, n_text, want_mask, ws, out)


def select_blocks_noalloc(q: torch.Tensor, k: torch.Tensor, block: int, tau: float, mask: Optional[torch.Tensor],
                          counts: torch.Tensor, idx: torch.Tensor, n_text: int = 0):
    """la_select_blocks_noalloc into the caller's outputs (mask may be None): the library's own
    scratch instead of a workspace, nothing allocated by the call or here."""
    _check_qkv("q", q)
    B, H, Lq, d = q.shape
    _check_qkv("k", k, B, H, d)
    shape = make_shape(B, H, Lq, k.shape[2], d, block, n_text, 0)
    _call("la_select_blocks_noalloc", ctypes.byref(shape), _ptr(q), _ptr(k), ctypes.c_float(tau), _ptr(mask),
          _ptr(counts), _ptr(idx), _stream(q))


def _select(fn, rule_arg, q, k, block, n_text, want_mask, ws, out):
    _check_qkv("q", q)
    B, H, Lq, d = q.shape
    _check_qkv("k", k, B, H, d)
    Lk = k.shape[2]
    shape = make_shape(B, H, Lq, Lk, d, block, n_text, 0)
    NQ, NK = nblocks(Lq, block), nblocks(Lk, block)
    if out is None:
        mask = torch.empty((B, H, NQ, NK), dtype=torch.uint8, device=q.device) if want_mask else None
        counts = torch.empty((B, H, NQ), dtype=torch.int32, device=q.device)
        idx = torch.empty((B, H, NQ, NK), dtype=torch.int32, device=q.device)
    else:
        mask, counts, idx = out
    ws, nbytes = _workspace(shape, q.device, ws)
    _call(fn, ctypes.byref(shape), _ptr(q), _ptr(k), rule_arg, _ptr(mask), _ptr(counts), _ptr(idx),
          _ptr(ws), ctypes.c_size_t(nbytes), _stream(q))
    return mask, counts, idx


def sparse_attn_fwd(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, counts: torch.Tensor,
                    idx: torch.Tensor, block: int, scale: Optional[float] = None, n_text: int = 0,
                    frame_tokens: int = 0, want_lse: bool = False, ws: Optional[torch.Tensor] = None,
                    out: Optional[torch.Tensor] = None, lse_out: Optional[torch.Tensor] = None,
                    kvalid: Optional[torch.Tensor] = None):
    """Block-sparse attention over the kept lists -> o bf16 [B,H,Lq,d] (and lse fp32 [B,H,Lq]).
    kvalid (int32 [NK] on the GPU): valid keys at the front of each key block
    (la_sparse_attn_fwd_valid); the other slots are padding."""
    _check_qkv("q", q)
    B, H, Lq, d = q.shape
    _check_qkv("k", k, B, H, d)
    _check_qkv("v", v, B, H, d)
    Lk = k.shape[2]
    if v.shape[2] != Lk:
        raise ValueError("k and v must have the same length")
    NQ, NK = nblocks(Lq, block), nblocks(Lk, block)
    if counts.dtype != torch.int32 or tuple(counts.shape) != (B, H, NQ) or not counts.is_contiguous():
        raise ValueError(f"counts must be contiguous int32 {(B, H, NQ)}")
    if idx.dtype != torch.int32 or tuple(idx.shape) != (B, H, NQ, NK) or not idx.is_contiguous():
        raise ValueError(f"idx must be contiguous int32 {(B, H, NQ, NK)}")
    shape = make_shape(B, H, Lq, Lk, d, block, n_text, frame_tokens)
    o = out if out is not None else torch.empty_like(q)
    lse = lse_out if lse_out is not None else (
        torch.empty((B, H, Lq), dtype=torch.float32, device=q.device) if want_lse else None)
    ws, nbytes = _workspace(shape, q.device, ws)
    sc = ctypes.c_float(scale if scale is not None else 0.0)
    if kvalid is None:
        _call("la_sparse_attn_fwd", ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v), _ptr(counts), _ptr(idx), sc,
              _ptr(o), _ptr(lse), _ptr(ws), ctypes.c_size_t(nbytes), _stream(q))
    else:
        if kvalid.device != q.device or kvalid.dtype != torch.int32 or tuple(kvalid.shape) != (NK,):
            raise ValueError(f"kvalid must be an int32 [{NK}] tensor on {q.device}")
        _call("la_sparse_attn_fwd_valid", ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v), _ptr(counts), _ptr(idx),
              _ptr(kvalid), sc, _ptr(o), _ptr(lse), _ptr(ws), ctypes.c_size_t(nbytes), _stream(q))
    return (o, lse) if (want_lse or lse_out is not None) else o


class BoundCall:
    """One C-ABI call with its arguments marshalled once (tensors, shape, stream fixed), for
    loops that issue the same call many times; calling it returns nothing and raises LaError
    on a failed status."""

    def __init__(self, fn: str, *args, keep=()):
        self._name = fn
        self._fn = getattr(lib(), fn)
        self._args = args
        self._keep = keep          # tensors and structs the raw pointers refer to

    def __call__(self):
        st = self._fn(*self._args)
        if st != LA_OK:
            raise LaError(self._name, st)


LA_POOL_Q, LA_POOL_K = 0, 1


def pool_blocks(x: torch.Tensor, block: int, which: str, shape: Shape, out: Optional[torch.Tensor] = None):
    """Block means of q (which="q", -> [B,H,NQ,d]) or k (which="k", -> [B,H,NK,d]) of `shape`, fp32;
    a ragged last block is the mean of its valid rows."""
    wcode = {"q": LA_POOL_Q, "k": LA_POOL_K}[which]
    L = shape.Lq if which == "q" else shape.Lk
    _check_qkv(which, x, shape.B, shape.H, shape.d)
    if x.shape[2] != L:
        raise ValueError(f"{which} must hold {L} tokens")
    nb = nblocks(L, block)
    if out is None:
        out = torch.empty((shape.B, shape.H, nb, shape.d), dtype=torch.float32, device=x.device)
    _call("la_pool_blocks", ctypes.byref(shape), _ptr(x), ctypes.c_int32(wcode), _ptr(out), _stream(x))
    return out


def bind_attn_steps(q, k, v, counts, idx, block, o, ws, scale: Optional[float] = None, n_text: int = 0,
                    frame_tokens: int = 0, lse: Optional[torch.Tensor] = None):
    """(plan, run, merge) of la_sparse_attn_fwd as BoundCalls on fixed tensors and the current
    stream; plan + run + merge computes the same o (and lse) as sparse_attn_fwd.  One plan serves
    any number of runs, as long as no other call uses `ws` in between (a selection call writes
    its scores there): after such a call, plan again before the next run."""
    _check_qkv("q", q)
    B, H, Lq, d = q.shape
    _check_qkv("k", k, B, H, d)
    _check_qkv("v", v, B, H, d)
    Lk = k.shape[2]
    shape = make_shape(B, H, Lq, Lk, d, block, n_text, frame_tokens)
    nbytes = ctypes.c_size_t(ws.numel())
    st = _stream(q)
    keep = (q, k, v, counts, idx, o, ws, lse, shape)
    sc = ctypes.c_float(scale if scale is not None else 0.0)
    plan = BoundCall("la_sparse_attn_plan", ctypes.byref(shape), _ptr(counts), _ptr(idx), _ptr(ws), nbytes, st,
                     keep=keep)
    run = BoundCall("la_sparse_attn_run", ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v), sc, _ptr(o), _ptr(lse),
                    _ptr(ws), nbytes, st, keep=keep)
    merge = BoundCall("la_sparse_attn_merge", ctypes.byref(shape), _ptr(o), _ptr(lse), _ptr(ws), nbytes, st,
                      keep=keep)
    return plan, run, merge


def plan_schedule(shape: Shape, ws: torch.Tensor) -> dict:
    """The schedule of the plan in ws (la_sparse_attn_schedule): P, U and the arrays tstart
    [U+1], ucount [U], dp_start [P+1], sk_start [P+1] as int64 CPU tensors (synchronises)."""
    P, U = ctypes.c_int32(0), ctypes.c_int32(0)
    _call("la_sparse_attn_schedule", ctypes.byref(shape), _ptr(ws), ctypes.c_size_t(ws.numel()), ctypes.byref(P),
          ctypes.byref(U), None, None, None, None, _stream(ws))
    arrs = {"tstart": int(U.value) + 1, "ucount": int(U.value), "dp_start": int(P.value) + 1,
            "sk_start": int(P.value) + 1}
    bufs = {k: torch.empty(n, dtype=torch.int32, device=ws.device) for k, n in arrs.items()}
    _call("la_sparse_attn_schedule", ctypes.byref(shape), _ptr(ws), ctypes.c_size_t(ws.numel()), ctypes.byref(P),
          ctypes.byref(U), _ptr(bufs["tstart"]), _ptr(bufs["ucount"]), _ptr(bufs["dp_start"]),
          _ptr(bufs["sk_start"]), _stream(ws))
    out = {k: b.cpu().to(torch.int64) for k, b in bufs.items()}
    out["P"], out["U"] = int(P.value), int(U.value)
    return out


def bind_select_cached(q, block, tau, kbar, qbar, mask, counts, idx, ws, Lk: int, n_text: int = 0):
    """(pool Q, select from pooled means) as BoundCalls: the selection of a step whose key means
    kbar [B,H,NK,d] were pooled earlier (la_pool_blocks); qbar [B,H,NQ,d] is written."""
    _check_qkv("q", q)
    B, H, Lq, d = q.shape
    shape = make_shape(B, H, Lq, Lk, d, block, n_text, 0)
    st = _stream(q)
    keep = (q, kbar, qbar, mask, counts, idx, ws, shape)
    pool = BoundCall("la_pool_blocks", ctypes.byref(shape), _ptr(q), ctypes.c_int32(LA_POOL_Q), _ptr(qbar), st,
                     keep=keep)
    sel = BoundCall("la_select_pooled", ctypes.byref(shape), _ptr(qbar), _ptr(kbar), ctypes.c_float(tau), _ptr(mask),
                    _ptr(counts), _ptr(idx), _ptr(ws), ctypes.c_size_t(ws.numel()), st, keep=keep)
    return pool, sel


def bind_select(q, k, block, tau, mask, counts, idx, ws, n_text: int = 0) -> BoundCall:
    """la_select_blocks as a BoundCall on fixed tensors and the current stream."""
    _check_qkv("q", q)
    B, H, Lq, d = q.shape
    _check_qkv("k", k, B, H, d)
    shape = make_shape(B, H, Lq, k.shape[2], d, block, n_text, 0)
    return BoundCall("la_select_blocks", ctypes.byref(shape), _ptr(q), _ptr(k), ctypes.c_float(tau), _ptr(mask),
                     _ptr(counts), _ptr(idx), _ptr(ws), ctypes.c_size_t(ws.numel()), _stream(q),
                     keep=(q, k, mask, counts, idx, ws, shape))


def mask_to_list(mask: torch.Tensor, block: int, Lq: int, Lk: int, d: int = 128):
    """Block mask uint8 [B,H,NQ,NK] -> (counts, idx) as la_sparse_attn_fwd reads them."""
    if mask.device.type != "cuda" or mask.dtype != torch.uint8 or mask.dim() != 4 or not mask.is_contiguous():
        raise TypeError("mask must be a contiguous uint8 [B, H, NQ, NK] GPU tensor")
    B, H, NQ, NK = mask.shape
    if NQ != nblocks(Lq, block) or NK != nblocks(Lk, block):
        raise ValueError("mask shape does not match Lq, Lk and block")
    shape = make_shape(B, H, Lq, Lk, d, block, 0, 0)
    counts = torch.empty((B, H, NQ), dtype=torch.int32, device=mask.device)
    idx = torch.empty((B, H, NQ, NK), dtype=torch.int32, device=mask.device)
    _call("la_mask_to_list", ctypes.byref(shape), _ptr(mask), _ptr(counts), _ptr(idx), _stream(mask))
    return counts, idx


# ----------------------------------------------------------------------------------------------
# 3-D block layout

def grid3d(B, H, d, n_text, T_ctx, T_q, Hs, Ws, bt, bh, bw, block=128) -> Grid3D:
    return Grid3D(B, H, d, n_text, T_ctx, T_q, Hs, Ws, bt, bh, bw, block)


def grid3d_shape(g: Grid3D) -> Shape:
    """la_shape of the tiled problem (Lq = NQ block, Lk = NK block, n_text = NT block)."""
    shape = Shape()
    _call("la_grid3d_shape", ctypes.byref(g), ctypes.byref(shape))
    return shape


def grid3d_valid(g: Grid3D):
    """(qvalid int32 [NQ], kvalid int32 [NK]) as numpy arrays: valid tokens per block."""
    import numpy as np
    shape = grid3d_shape(g)
    qv = np.zeros(nblocks(shape.Lq, g.block), dtype=np.int32)
    kv = np.zeros(nblocks(shape.Lk, g.block), dtype=np.int32)
    _call("la_grid3d_valid", ctypes.byref(g), qv.ctypes.data_as(_P), kv.ctypes.data_as(_P))
    return qv, kv


def _check_lin(name, t, g: Grid3D, L):
    _check_qkv(name, t, g.B, g.H, g.d)
    if t.shape[2] != L:
        raise ValueError(f"{name} must hold {L} tokens, got {t.shape[2]}")


def prep_q_3d(g: Grid3D, q: torch.Tensor, q_tiled: Optional[torch.Tensor] = None,
              qbar: Optional[torch.Tensor] = None, want_qbar: bool = True):
    """Fused Q-Prep: q linear [B,H,T_q Hs Ws,d] -> (q_tiled bf16 [B,H,NQ block,d], qbar fp32 [B,H,NQ,d])."""
    _check_lin("q", q, g, g.T_q * g.Hs * g.Ws)
    shape = grid3d_shape(g)
    NQ = nblocks(shape.Lq, g.block)
    if q_tiled is None:
        q_tiled = torch.empty((g.B, g.H, shape.Lq, g.d), dtype=torch.bfloat16, device=q.device)
    if qbar is None and want_qbar:
        qbar = torch.empty((g.B, g.H, NQ, g.d), dtype=torch.float32, device=q.device)
    _call("la_prep_q_3d", ctypes.byref(g), _ptr(q), _ptr(q_tiled), _ptr(qbar), _stream(q))
    return q_tiled, qbar


def prep_kv_3d(g: Grid3D, k: torch.Tensor, v: torch.Tensor, parts: int = LA_PART_ALL,
               k_tiled: Optional[torch.Tensor] = None, v_tiled: Optional[torch.Tensor] = None,
               kbar: Optional[torch.Tensor] = None, want_kbar: bool = True):
    """Fused KV-Prep of the regions in `parts`: k, v linear [B,H,n_text+(T_ctx+T_q) Hs Ws,d] ->
    (k_tiled, v_tiled bf16 [B,H,NK block,d], kbar fp32 [B,H,NK,d])."""
    L = g.n_text + (g.T_ctx + g.T_q) * g.Hs * g.Ws
    _check_lin("k", k, g, L)
    _check_lin("v", v, g, L)
    shape = grid3d_shape(g)
    NK = nblocks(shape.Lk, g.block)
    if k_tiled is None:
        k_tiled = torch.empty((g.B, g.H, shape.Lk, g.d), dtype=torch.bfloat16, device=k.device)
    if v_tiled is None:
        v_tiled = torch.empty((g.B, g.H, shape.Lk, g.d), dtype=torch.bfloat16, device=k.device)
    if kbar is None and want_kbar:
        kbar = torch.empty((g.B, g.H, NK, g.d), dtype=torch.float32, device=k.device)
    _call("la_prep_kv_3d", ctypes.byref(g), _ptr(k), _ptr(v), ctypes.c_uint32(parts), _ptr(k_tiled), _ptr(v_tiled),
          _ptr(kbar), _stream(k))
    return k_tiled, v_tiled, kbar


def select_pooled(shape: Shape, qbar: torch.Tensor, kbar: torch.Tensor, tau: Optional[float] = None,
                  keep_blocks: Optional[int] = None, want_mask: bool = True, ws: Optional[torch.Tensor] = None):
    """Selection from pooled means (qbar fp32 [B,H,NQ,d], kbar fp32 [B,H,NK,d]) with the tau rule or
    the top-keep_blocks rule -> (mask, counts, idx) as select_blocks."""
    if (tau is None) == (keep_blocks is None):
        raise ValueError("give exactly one of tau and keep_blocks")
    B, H, d, block = shape.B, shape.H, shape.d, shape.block
    NQ, NK = nblocks(shape.Lq, block), nblocks(shape.Lk, block)
    for name, t, n in (("qbar", qbar, NQ), ("kbar", kbar, NK)):
        if t.device.type != "cuda" or t.dtype != torch.float32 or tuple(t.shape) != (B, H, n, d) \
                or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous float32 {(B, H, n, d)} GPU tensor")
    mask = torch.empty((B, H, NQ, NK), dtype=torch.uint8, device=qbar.device) if want_mask else None
    counts = torch.empty((B, H, NQ), dtype=torch.int32, device=qbar.device)
    idx = torch.empty((B, H, NQ, NK), dtype=torch.int32, device=qbar.device)
    ws, nbytes = _workspace(shape, qbar.device, ws)
    if tau is not None:
        fn, arg = "la_select_pooled", ctypes.c_float(tau)
    else:
        fn, arg = "la_select_pooled_topk", ctypes.c_int32(keep_blocks)
    _call(fn, ctypes.byref(shape), _ptr(qbar), _ptr(kbar), arg, _ptr(mask), _ptr(counts), _ptr(idx), _ptr(ws),
          ctypes.c_size_t(nbytes), _stream(qbar))
    return mask, counts, idx


def untile_o_3d(g: Grid3D, o_tiled: torch.Tensor, lse_tiled: Optional[torch.Tensor] = None,
                o: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None):
    """Fused Untile Scatter: o_tiled [B,H,NQ block,d] (and lse_tiled) -> o linear [B,H,T_q Hs Ws,d] (and lse)."""
    shape = grid3d_shape(g)
    _check_lin("o_tiled", o_tiled, g, shape.Lq)
    L = g.T_q * g.Hs * g.Ws
    if o is None:
        o = torch.empty((g.B, g.H, L, g.d), dtype=torch.bfloat16, device=o_tiled.device)
    if lse is None and lse_tiled is not None:
        lse = torch.empty((g.B, g.H, L), dtype=torch.float32, device=o_tiled.device)
    _call("la_untile_o_3d", ctypes.byref(g), _ptr(o_tiled), _ptr(lse_tiled), _ptr(o), _ptr(lse), _stream(o_tiled))
    return o, lse


def bind_3d(g: Grid3D, q, k, v, q_t, k_t, v_t, qbar, kbar, mask, counts, idx, kvalid, o_t, lse_t, o, lse, ws,
            tau: Optional[float] = None, keep_blocks: Optional[int] = None, parts: int = LA_PART_ALL,
            scale: Optional[float] = None):
    """The 3-D path as BoundCalls on fixed tensors and the current stream:
    (prep_q, prep_kv, select, plan, run, merge, untile); in this order they compute what
    sparse_attn_3d computes."""
    if (tau is None) == (keep_blocks is None):
        raise ValueError("give exactly one of tau and keep_blocks")
    shape = grid3d_shape(g)
    st = _stream(q)
    nb = ctypes.c_size_t(ws.numel())
    keep = (g, shape, q, k, v, q_t, k_t, v_t, qbar, kbar, mask, counts, idx, kvalid, o_t, lse_t, o, lse, ws)
    gp, sp = ctypes.byref(g), ctypes.byref(shape)
    sc = ctypes.c_float(scale if scale is not None else 0.0)
    prep_q = BoundCall("la_prep_q_3d", gp, _ptr(q), _ptr(q_t), _ptr(qbar), st, keep=keep)
    prep_kv = BoundCall("la_prep_kv_3d", gp, _ptr(k), _ptr(v), ctypes.c_uint32(parts), _ptr(k_t), _ptr(v_t),
                        _ptr(kbar), st, keep=keep)
    if tau is not None:
        select = BoundCall("la_select_pooled", sp, _ptr(qbar), _ptr(kbar), ctypes.c_float(tau), _ptr(mask),
                           _ptr(counts), _ptr(idx), _ptr(ws), nb, st, keep=keep)
    else:
        select = BoundCall("la_select_pooled_topk", sp, _ptr(qbar), _ptr(kbar), ctypes.c_int32(keep_blocks),
                           _ptr(mask), _ptr(counts), _ptr(idx), _ptr(ws), nb, st, keep=keep)
    plan = BoundCall("la_sparse_attn_plan_valid", sp, _ptr(counts), _ptr(idx), _ptr(kvalid), _ptr(ws), nb, st,
                     keep=keep)
    run = BoundCall("la_sparse_attn_run", sp, _ptr(q_t), _ptr(k_t), _ptr(v_t), sc, _ptr(o_t), _ptr(lse_t), _ptr(ws),
                    nb, st, keep=keep)
    merge = BoundCall("la_sparse_attn_merge", sp, _ptr(o_t), _ptr(lse_t), _ptr(ws), nb, st, keep=keep)
    untile = BoundCall("la_untile_o_3d", gp, _ptr(o_t), _ptr(lse_t), _ptr(o), _ptr(lse), st, keep=keep)
    return prep_q, prep_kv, select, plan, run, merge, untile


def sparse_attn_3d(g: Grid3D, q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, tau: Optional[float] = None,
                   keep_blocks: Optional[int] = None, scale: Optional[float] = None, want_lse: bool = False,
                   kvalid: Optional[torch.Tensor] = None):
    """The whole 3-D path on linear-order inputs: Q-Prep, KV-Prep, selection from the pooled means,
    attention over the tiled buffers with the padding masked, Untile Scatter.  Returns
    (o linear, lse linear or None, mask over the tiled blocks, counts, idx)."""
    shape = grid3d_shape(g)
    if kvalid is None:
        kvalid = torch.from_numpy(grid3d_valid(g)[1]).to(q.device)
    q_t, qbar = prep_q_3d(g, q)
    k_t, v_t, kbar = prep_kv_3d(g, k, v)
    ws, _ = _workspace(shape, q.device, None)
    mask, counts, idx = select_pooled(shape, qbar, kbar, tau=tau, keep_blocks=keep_blocks, ws=ws)
    res = sparse_attn_fwd(q_t, k_t, v_t, counts, idx, g.block, scale=scale, n_text=shape.n_text, want_lse=want_lse,
                          ws=ws, kvalid=kvalid)
    o_t, lse_t = res if want_lse else (res, None)
    o, lse = untile_o_3d(g, o_t, lse_t)
    return o, lse, mask, counts, idx


# ----------------------------------------------------------------------------------------------
# scalar policy (Sec. 3.1, Sec. 3.2)

LA_DTYPE_F32, LA_DTYPE_BF16 = 0, 1
LATENT_MSE_WS_BYTES = 8192


def latent_mse(z_a: torch.Tensor, z_b: torch.Tensor, ws: Optional[torch.Tensor] = None,
               out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """D_t = MSE(z_a, z_b) over every value (fp32 or bf16 GPU tensors of one shape) -> float64
    GPU tensor of one element."""
    for name, t in (("z_a", z_a), ("z_b", z_b)):
        if not isinstance(t, torch.Tensor) or t.device.type != "cuda" or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous GPU tensor")
    if z_a.dtype != z_b.dtype or z_a.shape != z_b.shape:
        raise ValueError("z_a and z_b must have one dtype and one shape")
    dt = {torch.float32: LA_DTYPE_F32, torch.bfloat16: LA_DTYPE_BF16}.get(z_a.dtype)
    if dt is None:
        raise TypeError("latents must be float32 or bfloat16")
    if ws is None:
        ws = torch.empty(LATENT_MSE_WS_BYTES, dtype=torch.uint8, device=z_a.device)
    if out is None:
        out = torch.empty(1, dtype=torch.float64, device=z_a.device)
    _call("la_latent_mse", _ptr(z_a), _ptr(z_b), ctypes.c_int64(z_a.numel()), ctypes.c_int32(dt), _ptr(out),
          _ptr(ws), ctypes.c_size_t(ws.numel()), _stream(z_a))
    return out


def dynamics_ema(D_t: float, D_bar_prev: Optional[float], alpha: float) -> float:
    """D_bar_t = alpha D_t + (1 - alpha) D_bar_{t-1}; None starts the average (host only)."""
    res = ctypes.c_double()
    prev = None if D_bar_prev is None else ctypes.byref(ctypes.c_double(D_bar_prev))
    _call("la_dynamics_ema", ctypes.c_double(D_t), prev, ctypes.c_double(alpha), ctypes.byref(res))
    return res.value


def temporal_window(D_bar: float, kappa: float, L_m: int) -> int:
    """L_t = clip(floor(L_m kappa / (D_bar + kappa)), 1, L_m) (host only)."""
    res = ctypes.c_int32()
    _call("la_temporal_window", ctypes.c_double(D_bar), ctypes.c_double(kappa), ctypes.c_int32(L_m),
          ctypes.byref(res))
    return res.value


def pose_revisiting(similarities, tau_pose: float) -> bool:
    """max_j similarities[j] >= tau_pose (host only; float32 comparisons)."""
    import numpy as np
    sims = np.ascontiguousarray(similarities, dtype=np.float32)
    res = ctypes.c_int32()
    _call("la_pose_revisiting", sims.ctypes.data_as(_P) if sims.size else None, ctypes.c_int32(sims.size),
          ctypes.c_float(tau_pose), ctypes.byref(res))
    return bool(res.value)


def denoise_schedule(K: int, reuse: bool):
    """For each of the K denoising steps, the step whose model output it uses (host only)."""
    import numpy as np
    src = np.zeros(max(K, 1), dtype=np.int32)
    _call("la_denoise_schedule", ctypes.c_int32(K), ctypes.c_int32(1 if reuse else 0), src.ctypes.data_as(_P))
    return [int(x) for x in src[:K]]


def bf16_from_bits(bits, device="cuda") -> torch.Tensor:
    """uint16 numpy array of bfloat16 bit patterns -> bfloat16 tensor on `device` (no rounding)."""
    import numpy as np
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    return t.to(device)
