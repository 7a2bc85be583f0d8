"""The C-ABI library: it loads, exports every declared entry point, and rejects bad
arguments before touching the GPU.  Every call here fails validation by construction, so
none of them enqueues a kernel (the fake pointers are never dereferenced)."""
import ctypes
import os
import re

import pytest

from paper_2605_31158_amd import la

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _no_gpu():
    import torch
    return not torch.cuda.is_available()


# The rejection tests pass fake device pointers; they only ever run where no GPU exists.
cpu_only = pytest.mark.skipif(not _no_gpu(), reason="fake-pointer validation tests run on CPU hosts only")


def declared_functions():
    names = []
    for fn in os.listdir(os.path.join(ROOT, "include")):
        if fn.endswith(".h"):
            text = open(os.path.join(ROOT, "include", fn)).read()
            text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
            names += re.findall(r"\b(la_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert "la_select_blocks" in names and "la_sparse_attn_fwd" in names
    lib = la.lib()
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings_and_version():
    assert la.lib().la_abi_version() == 1
    for st in range(5):
        assert la.status_string(st)
    assert la.status_string(99) == "unknown status"


def test_workspace_sizing():
    s = la.make_shape(1, 16, 6240, 106080, 128, 64)
    nq, m = 98, 1560
    assert la.workspace_bytes(s) >= 16 * nq * 128 * 4 + 16 * nq * m * 4
    assert la.workspace_bytes(la.make_shape(1, 1, 64, 64, 96, 64)) == 0      # d = 96 unsupported


BAD_SHAPES = [
    dict(d=96), dict(block=32), dict(Lq=0), dict(Lq=2000, Lk=1000), dict(B=0),
    dict(n_text=-1), dict(n_text=1000, Lq=100, Lk=1000), dict(Lk=16384 * 128 + 1, block=128, Lq=128),
    dict(Lk=6000 * 64, Lq=64),   # M = 5999 historical candidates > 4096
]


@cpu_only
@pytest.mark.parametrize("bad", BAD_SHAPES, ids=[str(b) for b in BAD_SHAPES])
def test_bad_shapes_rejected(bad):
    base = dict(B=1, H=2, Lq=256, Lk=1024, d=64, block=64, n_text=0, frame_tokens=0)
    base.update(bad)
    s = la.make_shape(**base)
    p = ctypes.c_void_p(4096)
    lib = la.lib()
    assert lib.la_select_blocks(ctypes.byref(s), p, p, ctypes.c_float(0.9), p, p, p, p, 1 << 30, None) == la.LA_ERR_SHAPE
    assert lib.la_sparse_attn_fwd(ctypes.byref(s), p, p, p, p, p, ctypes.c_float(0), p, None, p, 1 << 30,
                                  None) == la.LA_ERR_SHAPE
    assert lib.la_mask_to_list(ctypes.byref(s), p, p, p, None) == la.LA_ERR_SHAPE
    assert lib.la_sparse_attn_plan(ctypes.byref(s), p, p, p, 1 << 30, None) == la.LA_ERR_SHAPE
    assert lib.la_sparse_attn_run(ctypes.byref(s), p, p, p, ctypes.c_float(0), p, None, p, 1 << 30,
                                  None) == la.LA_ERR_SHAPE
    assert lib.la_sparse_attn_merge(ctypes.byref(s), p, None, p, 1 << 30, None) == la.LA_ERR_SHAPE
    n = ctypes.c_int32(0)
    assert lib.la_sparse_attn_schedule(ctypes.byref(s), p, 1 << 30, ctypes.byref(n), ctypes.byref(n), p, p, p, p,
                                       None) == la.LA_ERR_SHAPE


@cpu_only
def test_tile_index_bound_rejected():
    # 65535 heads x 1 unit x 16384 key blocks x 2 sub-tiles of 64 keys exceeds 32-bit tile indices
    s = la.make_shape(1, 65535, 128, 16384 * 128, 64, 128)
    assert la.workspace_bytes(s) == 0
    # a few heads over 4000 key blocks fit
    assert la.workspace_bytes(la.make_shape(1, 4, 128, 4000 * 64, 64, 64)) > 0


@cpu_only
def test_bad_arguments_rejected():
    lib = la.lib()
    s = la.make_shape(1, 2, 256, 1024, 64, 64)
    p = ctypes.c_void_p(4096)
    odd = ctypes.c_void_p(4098)
    ws = la.workspace_bytes(s)
    sel = lib.la_select_blocks
    assert sel(None, p, p, ctypes.c_float(0.9), p, p, p, p, ws, None) == la.LA_ERR_ARG
    assert sel(ctypes.byref(s), None, p, ctypes.c_float(0.9), p, p, p, p, ws, None) == la.LA_ERR_ARG
    assert sel(ctypes.byref(s), p, p, ctypes.c_float(0.0), p, p, p, p, ws, None) == la.LA_ERR_ARG
    assert sel(ctypes.byref(s), p, p, ctypes.c_float(-1.0), p, p, p, p, ws, None) == la.LA_ERR_ARG
    assert sel(ctypes.byref(s), p, p, ctypes.c_float(float("nan")), p, p, p, p, ws, None) == la.LA_ERR_ARG
    assert sel(ctypes.byref(s), odd, p, ctypes.c_float(0.9), p, p, p, p, ws, None) == la.LA_ERR_ARG
    assert sel(ctypes.byref(s), p, p, ctypes.c_float(0.9), p, None, p, p, ws, None) == la.LA_ERR_ARG
    assert sel(ctypes.byref(s), p, p, ctypes.c_float(0.9), p, p, p, None, ws, None) == la.LA_ERR_WORKSPACE
    assert sel(ctypes.byref(s), p, p, ctypes.c_float(0.9), p, p, p, p, 255, None) == la.LA_ERR_WORKSPACE
    assert sel(ctypes.byref(s), p, p, ctypes.c_float(0.9), p, p, p, ctypes.c_void_p(4096 + 16), ws,
               None) == la.LA_ERR_WORKSPACE
    topk = lib.la_select_blocks_topk
    assert topk(ctypes.byref(s), p, p, ctypes.c_int32(-1), p, p, p, p, ws, None) == la.LA_ERR_ARG
    att = lib.la_sparse_attn_fwd
    assert att(ctypes.byref(s), p, p, None, p, p, ctypes.c_float(0), p, None, p, ws, None) == la.LA_ERR_ARG
    assert att(ctypes.byref(s), p, p, p, p, p, ctypes.c_float(float("inf")), p, None, p, ws, None) == la.LA_ERR_ARG
    assert att(ctypes.byref(s), p, p, p, p, p, ctypes.c_float(0), odd, None, p, ws, None) == la.LA_ERR_ARG
    assert lib.la_mask_to_list(ctypes.byref(s), None, p, p, None) == la.LA_ERR_ARG
    assert lib.la_sparse_attn_plan(ctypes.byref(s), None, p, p, ws, None) == la.LA_ERR_ARG
    assert lib.la_sparse_attn_plan(ctypes.byref(s), p, p, None, ws, None) == la.LA_ERR_WORKSPACE
    assert lib.la_sparse_attn_plan(ctypes.byref(s), p, p, p, 255, None) == la.LA_ERR_WORKSPACE
    run = lib.la_sparse_attn_run
    assert run(ctypes.byref(s), p, None, p, ctypes.c_float(0), p, None, p, ws, None) == la.LA_ERR_ARG
    assert run(ctypes.byref(s), p, p, p, ctypes.c_float(float("nan")), p, None, p, ws, None) == la.LA_ERR_ARG
    assert run(ctypes.byref(s), p, p, p, ctypes.c_float(0), p, None, p, 16, None) == la.LA_ERR_WORKSPACE
    assert lib.la_sparse_attn_merge(ctypes.byref(s), None, None, p, ws, None) == la.LA_ERR_ARG
    assert lib.la_pool_blocks(ctypes.byref(s), p, 2, p, None) == la.LA_ERR_ARG
    assert lib.la_pool_blocks(ctypes.byref(s), None, 0, p, None) == la.LA_ERR_ARG
    assert lib.la_pool_blocks(ctypes.byref(s), p, 1, odd, None) == la.LA_ERR_ARG
    assert lib.la_sparse_attn_merge(ctypes.byref(s), odd, None, p, ws, None) == la.LA_ERR_ARG
    sch = lib.la_sparse_attn_schedule
    n = ctypes.c_int32(-5)
    assert sch(ctypes.byref(s), p, ws, None, ctypes.byref(n), p, p, p, p, None) == la.LA_ERR_ARG
    assert sch(ctypes.byref(s), p, ws, ctypes.byref(n), None, p, p, p, p, None) == la.LA_ERR_ARG
    assert sch(ctypes.byref(s), None, ws, ctypes.byref(n), ctypes.byref(n), p, p, p, p, None) == la.LA_ERR_WORKSPACE
    assert sch(ctypes.byref(s), p, 16, ctypes.byref(n), ctypes.byref(n), p, p, p, p, None) == la.LA_ERR_WORKSPACE
    assert sch(None, p, ws, ctypes.byref(n), ctypes.byref(n), p, p, p, p, None) == la.LA_ERR_ARG
    assert n.value == -5                 # nothing written on an error


@cpu_only
def test_noalloc_selection_rejects_before_any_gpu_call():
    # bad arguments, bad shapes and shapes whose selection scratch exceeds the library's array
    # (4 B x B*H*NQ*(d + M) > 16 MiB) are refused before the scratch is looked up
    lib = la.lib()
    p = ctypes.c_void_p(4096)
    odd = ctypes.c_void_p(4098)
    na = lib.la_select_blocks_noalloc
    s = la.make_shape(1, 2, 256, 1024, 64, 64)
    assert na(ctypes.byref(s), p, p, ctypes.c_float(0.0), p, p, p, None) == la.LA_ERR_ARG
    assert na(ctypes.byref(s), p, p, ctypes.c_float(float("nan")), p, p, p, None) == la.LA_ERR_ARG
    assert na(ctypes.byref(s), None, p, ctypes.c_float(0.9), p, p, p, None) == la.LA_ERR_ARG
    assert na(ctypes.byref(s), p, odd, ctypes.c_float(0.9), p, p, p, None) == la.LA_ERR_ARG
    assert na(ctypes.byref(s), p, p, ctypes.c_float(0.9), p, p, None, None) == la.LA_ERR_ARG
    assert na(None, p, p, ctypes.c_float(0.9), p, p, p, None) == la.LA_ERR_ARG
    assert na(ctypes.byref(la.make_shape(1, 2, 256, 1024, 96, 64)), p, p, ctypes.c_float(0.9), p, p, p,
              None) == la.LA_ERR_SHAPE
    big = la.make_shape(1, 16, 6400, 6400 + 3000 * 64, 128, 64)      # 16 x 100 x (128 + 3000) x 4 B = 20 MB
    assert na(ctypes.byref(big), p, p, ctypes.c_float(0.9), p, p, p, None) == la.LA_ERR_WORKSPACE


def test_binding_refuses_cpu_tensors():
    import torch
    q = torch.zeros(1, 1, 64, 64, dtype=torch.bfloat16)
    with pytest.raises(TypeError):
        la.select_blocks(q, q, 64, 0.9)
    with pytest.raises(TypeError):
        la.sparse_attn_fwd(q, q, q, torch.zeros(1, 1, 1, dtype=torch.int32),
                           torch.zeros(1, 1, 1, 1, dtype=torch.int32), 64)
