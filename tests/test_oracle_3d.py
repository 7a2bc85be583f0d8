"""Pins of the oracle's 3-D block layout (Sec. 3.3: visual tokens in (B_t, B_h, B_w) blocks).

Each check reaches the same quantity by a second route: the block partition by decoding token
coordinates, the pooled proxies by slicing the (T, H, W) grid, whole-frame blocks by the pinned
1-D oracle, keep-all attention by torch's fp64 attention, and set semantics by reordering."""
import math

import numpy as np
import pytest
import torch

from oracle import la_oracle as O


def _decode(pos, offset, Hs, Ws):
    r = pos - offset
    return r // (Hs * Ws), (r // Ws) % Hs, r % Ws


@pytest.mark.parametrize("T,Hs,Ws,bt,bh,bw", [(8, 30, 52, 4, 8, 4), (4, 45, 80, 4, 4, 8), (5, 7, 9, 2, 3, 4),
                                            (1, 1, 1, 4, 8, 4)])
def test_blocks_partition_the_grid(T, Hs, Ws, bt, bh, bw):
    off = 37
    sets = O.blocks_3d(T, Hs, Ws, bt, bh, bw, offset=off)
    nb = -(-T // bt) * -(-Hs // bh) * -(-Ws // bw)
    assert len(sets) == nb
    allpos = np.sort(np.concatenate(sets))
    np.testing.assert_array_equal(allpos, np.arange(off, off + T * Hs * Ws))
    # block index n holds exactly the tokens whose coordinates fall in its box
    nby, nbx = -(-Hs // bh), -(-Ws // bw)
    for n, s in enumerate(sets):
        cb_t, rem = divmod(n, nby * nbx)
        cb_y, cb_x = divmod(rem, nbx)
        t, y, x = _decode(s, off, Hs, Ws)
        assert (t // bt == cb_t).all() and (y // bh == cb_y).all() and (x // bw == cb_x).all()
        ext = (min(bt, T - cb_t * bt), min(bh, Hs - cb_y * bh), min(bw, Ws - cb_x * bw))
        assert s.size == ext[0] * ext[1] * ext[2]


def test_pool_sets_equals_grid_slices():
    rng = np.random.default_rng(3)
    T, Hs, Ws, bt, bh, bw, d = 5, 7, 9, 2, 3, 4, 6
    x = rng.standard_normal((2, T * Hs * Ws, d))
    sets = O.blocks_3d(T, Hs, Ws, bt, bh, bw)
    pooled = O.pool_sets(x, sets)
    grid = x.reshape(2, T, Hs, Ws, d)
    n = 0
    for t0 in range(0, T, bt):
        for y0 in range(0, Hs, bh):
            for x0 in range(0, Ws, bw):
                want = grid[:, t0:t0 + bt, y0:y0 + bh, x0:x0 + bw, :].reshape(2, -1, d).mean(axis=1)
                np.testing.assert_allclose(pooled[:, n], want, rtol=0, atol=1e-12)
                n += 1


def test_layout_blocks_and_forced_set():
    L = O.layout_3d(70, 8, 4, 30, 52, 4, 8, 4, 128)
    assert L["Lq"] == 4 * 1560 and L["Lk"] == 70 + 12 * 1560
    assert len(L["qsets"]) == 52 and len(L["ksets"]) == 1 + 104 + 52
    forced = L["forced"]
    assert forced[0] and not forced[1:105].any() and forced[105:].all()
    # every key position in exactly one block; query blocks are chunk positions
    np.testing.assert_array_equal(np.sort(np.concatenate(L["ksets"])), np.arange(L["Lk"]))
    np.testing.assert_array_equal(np.sort(np.concatenate(L["qsets"])), np.arange(L["Lq"]))
    # the chunk's key blocks are its query blocks shifted by the context length
    for qs, ks in zip(L["qsets"], L["ksets"][105:]):
        np.testing.assert_array_equal(ks, qs + 70 + 8 * 1560)


def _problem(seed, B, H, Lq, Lk, d):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((B, H, Lq, d)), rng.standard_normal((B, H, Lk, d)),
            rng.standard_normal((B, H, Lk, d)))


def test_whole_frame_blocks_reduce_to_1d_blocks():
    # (1, Hs, Ws) blocks are whole frames: 1-D blocks of F = Hs * Ws tokens
    Hs, Ws, T_ctx, T_q, d = 3, 4, 5, 2, 8
    F = Hs * Ws
    n_text = F
    L = O.layout_3d(n_text, T_ctx, T_q, Hs, Ws, 1, Hs, Ws, F)
    q, k, v = _problem(5, 1, 2, L["Lq"], L["Lk"], d)
    for tau in (0.3, 0.8, 1.0):
        a = O.select_blocks_sets(q, k, L["qsets"], L["ksets"], L["forced"], tau=tau)
        b = O.select_blocks(q, k, F, tau=tau, n_text=n_text)
        np.testing.assert_array_equal(a["mask"], b["mask"])
        np.testing.assert_allclose(a["scores"], b["scores"], rtol=0, atol=1e-12)
        rows = [(0, h, i) for h in range(2) for i in range(len(L["qsets"]))]
        ra = O.attention_sets_rows(q, k, v, L["qsets"], L["ksets"], a["mask"], rows)
        rb = O.attention_rows(q, k, v, b["mask"], F, rows)
        for key in rows:
            np.testing.assert_allclose(ra[key][0], rb[key][0], rtol=0, atol=1e-12)
            np.testing.assert_allclose(ra[key][1], rb[key][1], rtol=0, atol=1e-12)


def test_keep_all_equals_dense_attention():
    Hs, Ws, T_ctx, T_q, d = 5, 6, 3, 2, 16
    L = O.layout_3d(7, T_ctx, T_q, Hs, Ws, 2, 2, 4, 16)
    q, k, v = _problem(8, 1, 2, L["Lq"], L["Lk"], d)
    sel = O.select_blocks_sets(q, k, L["qsets"], L["ksets"], L["forced"], tau=1.0)
    assert sel["mask"].all()
    rows = [(0, h, i) for h in range(2) for i in range(len(L["qsets"]))]
    res = O.attention_sets_rows(q, k, v, L["qsets"], L["ksets"], sel["mask"], rows)
    dense = torch.nn.functional.scaled_dot_product_attention(torch.from_numpy(q), torch.from_numpy(k),
                                                             torch.from_numpy(v)).numpy()
    for (b, h, i), (o, lse) in res.items():
        np.testing.assert_allclose(o, dense[b, h, L["qsets"][i]], rtol=0, atol=1e-12)
        logits = q[b, h, L["qsets"][i]] @ k[b, h].T / math.sqrt(d)
        mx = logits.max(axis=1)
        np.testing.assert_allclose(lse, mx + np.log(np.exp(logits - mx[:, None]).sum(axis=1)), rtol=0, atol=1e-12)


def test_selection_and_attention_read_blocks_as_sets():
    Hs, Ws, T_ctx, T_q, d = 6, 8, 4, 2, 8
    L = O.layout_3d(0, T_ctx, T_q, Hs, Ws, 2, 4, 4, 32)
    q, k, v = _problem(11, 1, 1, L["Lq"], L["Lk"], d)
    rng = np.random.default_rng(12)
    shuf = lambda sets: [s[rng.permutation(s.size)] for s in sets]
    qs2, ks2 = shuf(L["qsets"]), shuf(L["ksets"])
    a = O.select_blocks_sets(q, k, L["qsets"], L["ksets"], L["forced"], tau=0.7)
    b = O.select_blocks_sets(q, k, qs2, ks2, L["forced"], tau=0.7)
    np.testing.assert_array_equal(a["mask"], b["mask"])
    rows = [(0, 0, i) for i in range(len(L["qsets"]))]
    ra = O.attention_sets_rows(q, k, v, L["qsets"], L["ksets"], a["mask"], rows)
    rb = O.attention_sets_rows(q, k, v, qs2, ks2, b["mask"], rows)
    for key in rows:
        order = np.argsort(qs2[key[2]])      # rb rows follow the shuffled query order
        inv = np.argsort(L["qsets"][key[2]])
        np.testing.assert_allclose(ra[key][0][inv], rb[key][0][order], rtol=0, atol=1e-12)


# planted mistakes in a copy of the oracle's 3-D section: each must fail some pin above
MUTANTS_3D = {
    "pool divides by the block volume": ("out[..., i, :] = total / len(idx)",
                                         "out[..., i, :] = total / max(len(idx), 128)"),
    "edge block cut on the wrong axis": ("for y in range(y0, min(y0 + bh, Hs))",
                                         "for y in range(y0, min(y0 + bh, Ws))"),
    "context frames offset by the chunk": ("kchunk = blocks_3d(T_q, Hs, Ws, bt, bh, bw, offset=n_text + T_ctx * F)",
                                           "kchunk = blocks_3d(T_q, Hs, Ws, bt, bh, bw, offset=n_text + T_ctx * F - 1)"),
    "chunk blocks not forced": ("[True] * len(kchunk)", "[False] * len(kchunk)"),
    "unsorted candidate keys dropped": ("cand = np.sort(np.concatenate([ksets[int(m)] for m in kept]))",
                                        "cand = np.sort(np.concatenate([ksets[int(m)] for m in kept[:-1]]))"),
}


def _pins():
    import inspect
    pins = []
    for name, fn in sorted(globals().items()):
        if name.startswith("test_") and name != "test_pins_catch_3d_mutant" and callable(fn):
            marks = getattr(fn, "pytestmark", [])
            params = [m for m in marks if m.name == "parametrize"]
            if params:
                argnames = [a.strip() for a in params[0].args[0].split(",")]
                for vals in params[0].args[1]:
                    pins.append((fn, dict(zip(argnames, vals))))
            else:
                pins.append((fn, {}))
    return pins


@pytest.mark.parametrize("name", sorted(MUTANTS_3D))
def test_pins_catch_3d_mutant(name, monkeypatch):
    import inspect
    import sys
    import types
    old, new = MUTANTS_3D[name]
    src = inspect.getsource(O)
    assert src.count(old) == 1, old
    mod = types.ModuleType("oracle_mutant_3d")
    exec(compile(src.replace(old, new), "oracle_mutant_3d", "exec"), mod.__dict__)
    monkeypatch.setattr(sys.modules[__name__], "O", mod)
    caught = 0
    for fn, kw in _pins():
        try:
            fn(**kw)
        except Exception:
            caught += 1
    assert caught, f"no pin catches the planted mistake: {name}"
