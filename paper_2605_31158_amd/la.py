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


_lib = None
_P = ctypes.c_void_p
_SP = ctypes.POINTER(Shape)

_SIGNATURES = {
    "la_workspace_bytes": (ctypes.c_size_t, [_SP]),
    "la_select_blocks": (ctypes.c_int, [_SP, _P, _P, ctypes.c_float, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_select_blocks_topk": (ctypes.c_int, [_SP, _P, _P, ctypes.c_int32, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_sparse_attn_fwd": (ctypes.c_int, [_SP, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_sparse_attn_plan": (ctypes.c_int, [_SP, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_sparse_attn_run": (ctypes.c_int, [_SP, _P, _P, _P, ctypes.c_float, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_sparse_attn_merge": (ctypes.c_int, [_SP, _P, _P, _P, ctypes.c_size_t, _P]),
    "la_mask_to_list": (ctypes.c_int, [_SP, _P, _P, _P, _P]),
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
                    out: Optional[torch.Tensor] = None, lse_out: Optional[torch.Tensor] = None):
    """Block-sparse attention over the kept lists -> o bf16 [B,H,Lq,d] (and lse fp32 [B,H,Lq])."""
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
    _call("la_sparse_attn_fwd", ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v), _ptr(counts), _ptr(idx),
          ctypes.c_float(scale if scale is not None else 0.0), _ptr(o), _ptr(lse), _ptr(ws),
          ctypes.c_size_t(nbytes), _stream(q))
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


def bind_attn_steps(q, k, v, counts, idx, block, o, ws, scale: Optional[float] = None, n_text: int = 0,
                    frame_tokens: int = 0, lse: Optional[torch.Tensor] = None):
    """(plan, run, merge) of la_sparse_attn_fwd as BoundCalls on fixed tensors and the current
    stream; plan + run + merge computes the same o (and lse) as sparse_attn_fwd."""
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


def bf16_from_bits(bits, device="cuda") -> torch.Tensor:
    """uint16 numpy array of bfloat16 bit patterns -> bfloat16 tensor on `device` (no rounding)."""
    import numpy as np
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16)
    return t.to(device)
