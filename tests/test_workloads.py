"""The seeded generator: determinism, shapes, block structure."""
import numpy as np
import pytest

from paper_2605_31158_amd.workloads import (WORKLOADS, CONFIG_ORDER, make_inputs, make_clustered,
                                            f32_to_bf16_bits)


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, 1.0 + 2 ** -9], np.float32)
    # 1+2^-8 is a tie between 1 and 1+2^-7: rounds to even (1.0); 1+3*2^-8 rounds up to 1+2^-6
    assert f32_to_bf16_bits(x).tolist() == [0x3F80, 0x3F80, 0x3F82, 0xC020, 0x3F80]


def test_shapes_of_named_workloads():
    want = {"tiny": (2, 64, 256, 1024, 64, 4, 16), "480p_window": (16, 128, 6240, 18720, 64, 98, 293),
            "480p_memory": (16, 128, 6240, 43680, 64, 98, 683), "720p": (24, 128, 14400, 72000, 128, 113, 563),
            "480p_long": (16, 128, 6240, 106080, 64, 98, 1658)}
    for name in CONFIG_ORDER:
        wl = WORKLOADS[name]
        assert (wl.H, wl.d, wl.Lq, wl.Lk, wl.block, wl.nq, wl.nk) == want[name]
    assert WORKLOADS["720p_causal"].causal_frames and WORKLOADS["480p_long_dense"].tau == 1.0


def test_deterministic_per_seed():
    wl = WORKLOADS["tiny"]
    a, b = make_inputs(wl), make_inputs(wl, threads=1)
    for x in "qkv":
        assert a[x].dtype == np.uint16 and a[x].shape[:2] == (1, 2)
        np.testing.assert_array_equal(a[x], b[x])
    c = make_inputs(wl.replace(seed=7))
    assert not np.array_equal(a["q"], c["q"])


def test_frame_structure_shares_centroids_with_chunk():
    # queries and chunk keys share block centroids: their block means nearly coincide
    for kind in ("walk", "memory", "related720", "clusters"):
        n_ctx = {"walk": 8, "memory": 24, "related720": 16, "clusters": 64}[kind]
        wl = WORKLOADS["480p_window"].replace(kind=kind, H=1, d=32, frame_tokens=96, block=32,
                                              Lq=4 * 96, Lk=(n_ctx + 4) * 96)
        inp = make_inputs(wl)
        f = lambda u: (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
        q, k = f(inp["q"][0, 0]), f(inp["k"][0, 0])
        qm = q.reshape(-1, 32, 32).mean(1)
        km = k[wl.Lk - wl.Lq:].reshape(-1, 32, 32).mean(1)
        same = np.abs(qm - km).max()
        other = np.abs(qm[1:] - km[:-1]).mean()
        assert same < 0.5 and other > 0.1, (kind, same, other)


def test_clustered_helper():
    inp = make_clustered(2, 3, Lq=70, Lk=200, d=16, block=32, seed=1, v_kind="index")
    assert inp["q"].shape == (2, 3, 70, 16) and inp["v"].shape == (2, 3, 200, 16)


def test_3d_generator_is_seeded_and_follows_its_recipe():
    from paper_2605_31158_amd.workloads import WORKLOADS_3D, make_inputs_3d
    wl = WORKLOADS_3D["tiny_3d"]
    a, b = make_inputs_3d(wl), make_inputs_3d(wl)
    for x in "qkv":
        np.testing.assert_array_equal(a[x], b[x])
    assert a["q"].shape == (wl.B, wl.H, wl.Lq, wl.d) and a["k"].shape == (wl.B, wl.H, wl.Lk, wl.d)
    c = make_inputs_3d(wl.replace(seed=wl.seed + 1))
    assert not np.array_equal(a["k"], c["k"])
    # recipe: a chunk query and the chunk key at the same position share a centroid (noise 0.5 each),
    # tokens of different regions do not
    f = lambda bits: (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    q, k = f(a["q"][0, 0]), f(a["k"][0, 0])
    ck = k[wl.n_text + wl.T_ctx * wl.frame_tokens:]
    same = np.mean(np.sum(q * ck, axis=1)) / wl.d
    assert 0.6 < same < 1.6, same        # centroid variance ~1 (random walk), noise uncorrelated
    other = np.mean(np.sum(q[: wl.Ws] * np.roll(ck[: wl.Ws], wl.bw, axis=0), axis=1)) / wl.d
    assert abs(other) < 0.4, other
