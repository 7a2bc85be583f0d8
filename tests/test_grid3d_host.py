"""Host side of the 3-D block layout: the tiled shape and the per-block valid counts the library
derives from a la_grid3d, checked against the oracle's block sets, and argument rejection of the
3-D entry points before anything reaches the GPU (fake pointers, CPU hosts only)."""
import ctypes

import numpy as np
import pytest

from oracle import la_oracle as O
from paper_2605_31158_amd import la
from paper_2605_31158_amd.workloads import WORKLOADS_3D

GRIDS = [
    # B, H, d, n_text, T_ctx, T_q, Hs, Ws, bt, bh, bw, block
    (1, 16, 128, 300, 24, 4, 30, 52, 4, 8, 4, 128),
    (1, 24, 128, 0, 16, 4, 45, 80, 4, 4, 8, 128),
    (1, 2, 64, 40, 6, 3, 7, 10, 2, 3, 4, 64),
    (2, 3, 128, 128, 0, 1, 5, 5, 1, 1, 1, 64),
    (1, 1, 64, 1, 5, 7, 3, 9, 4, 2, 8, 64),
]


@pytest.mark.parametrize("g", GRIDS, ids=[str(g) for g in GRIDS])
def test_tiled_shape_and_valid_counts_match_oracle_sets(g):
    B, H, d, n_text, T_ctx, T_q, Hs, Ws, bt, bh, bw, block = g
    grid = la.grid3d(*g)
    shape = la.grid3d_shape(grid)
    L = O.layout_3d(n_text, T_ctx, T_q, Hs, Ws, bt, bh, bw, block)
    NQ, NK = len(L["qsets"]), len(L["ksets"])
    NT = -(-n_text // block)
    assert (shape.B, shape.H, shape.d, shape.block) == (B, H, d, block)
    assert shape.Lq == NQ * block and shape.Lk == NK * block
    assert shape.n_text == NT * block and shape.frame_tokens == 0
    qv, kv = la.grid3d_valid(grid)
    np.testing.assert_array_equal(qv, [len(s) for s in L["qsets"]])
    np.testing.assert_array_equal(kv, [len(s) for s in L["ksets"]])
    # forced blocks of the tiled shape (text and chunk) are the oracle's forced blocks
    h0, h1 = NT, (shape.Lk - shape.Lq) // block
    forced = np.ones(NK, bool)
    forced[h0:h1] = False
    np.testing.assert_array_equal(forced, L["forced"])


def test_named_3d_workloads_have_valid_grids():
    for wl in WORKLOADS_3D.values():
        grid = la.grid3d(wl.B, wl.H, wl.d, wl.n_text, wl.T_ctx, wl.T_q, wl.Hs, wl.Ws, wl.bt, wl.bh, wl.bw, wl.block)
        shape = la.grid3d_shape(grid)
        assert la.workspace_bytes(shape) > 0
        assert wl.bt * wl.bh * wl.bw <= wl.block


BAD = [dict(bt=8), dict(block=32), dict(d=96), dict(T_q=0), dict(Hs=0), dict(n_text=-1), dict(T_ctx=-1),
       dict(bw=0), dict(T_ctx=40000)]


@pytest.mark.parametrize("bad", BAD, ids=[str(b) for b in BAD])
def test_bad_grids_rejected(bad):
    base = dict(B=1, H=2, d=64, n_text=40, T_ctx=6, T_q=3, Hs=7, Ws=10, bt=4, bh=4, bw=4, block=64)
    base.update(bad)
    grid = la.Grid3D(*[base[n] for n, _ in la.Grid3D._fields_])
    lib = la.lib()
    s = la.Shape()
    p = ctypes.c_void_p(4096)
    assert lib.la_grid3d_shape(ctypes.byref(grid), ctypes.byref(s)) == la.LA_ERR_SHAPE
    assert lib.la_grid3d_valid(ctypes.byref(grid), None, None) == la.LA_ERR_SHAPE
    assert lib.la_prep_q_3d(ctypes.byref(grid), p, p, p, None) == la.LA_ERR_SHAPE
    assert lib.la_prep_kv_3d(ctypes.byref(grid), p, p, la.LA_PART_ALL, p, p, p, None) == la.LA_ERR_SHAPE
    assert lib.la_untile_o_3d(ctypes.byref(grid), p, p, p, p, None) == la.LA_ERR_SHAPE


def _no_gpu():
    import torch
    return not torch.cuda.is_available()


@pytest.mark.skipif(not _no_gpu(), reason="fake-pointer validation tests run on CPU hosts only")
def test_bad_arguments_rejected_3d():
    lib = la.lib()
    grid = la.grid3d(1, 2, 64, 40, 6, 3, 7, 10, 2, 3, 4, 64)
    g = ctypes.byref(grid)
    p, odd = ctypes.c_void_p(4096), ctypes.c_void_p(4100)
    assert lib.la_grid3d_shape(None, None) == la.LA_ERR_ARG
    assert lib.la_grid3d_shape(g, None) == la.LA_ERR_ARG
    assert lib.la_prep_q_3d(g, None, p, p, None) == la.LA_ERR_ARG
    assert lib.la_prep_q_3d(g, p, odd, p, None) == la.LA_ERR_ARG
    assert lib.la_prep_kv_3d(g, p, p, 0, p, p, p, None) == la.LA_ERR_ARG
    assert lib.la_prep_kv_3d(g, p, p, 8, p, p, p, None) == la.LA_ERR_ARG
    assert lib.la_prep_kv_3d(g, p, None, la.LA_PART_ALL, p, p, p, None) == la.LA_ERR_ARG
    assert lib.la_prep_kv_3d(g, p, p, la.LA_PART_ALL, p, p, odd, None) == la.LA_ERR_ARG
    assert lib.la_untile_o_3d(g, None, None, p, None, None) == la.LA_ERR_ARG
    s = la.grid3d_shape(grid)
    ws = la.workspace_bytes(s)
    sp = lib.la_select_pooled
    assert sp(ctypes.byref(s), p, p, ctypes.c_float(0.0), p, p, p, p, ws, None) == la.LA_ERR_ARG
    assert sp(ctypes.byref(s), None, p, ctypes.c_float(0.9), p, p, p, p, ws, None) == la.LA_ERR_ARG
    assert sp(ctypes.byref(s), p, odd, ctypes.c_float(0.9), p, p, p, p, ws, None) == la.LA_ERR_ARG
    assert sp(ctypes.byref(s), p, p, ctypes.c_float(0.9), p, p, p, p, 16, None) == la.LA_ERR_WORKSPACE
    assert lib.la_select_pooled_topk(ctypes.byref(s), p, p, ctypes.c_int32(-1), p, p, p, p, ws,
                                     None) == la.LA_ERR_ARG
    fv = lib.la_sparse_attn_fwd_valid
    assert fv(ctypes.byref(s), p, p, p, None, p, p, ctypes.c_float(0), p, None, p, ws, None) == la.LA_ERR_ARG
    assert fv(ctypes.byref(s), p, p, p, p, p, p, ctypes.c_float(0), p, None, p, 16, None) == la.LA_ERR_WORKSPACE
    assert lib.la_sparse_attn_plan_valid(ctypes.byref(s), p, None, p, p, ws, None) == la.LA_ERR_ARG
