"""Host-only policy calls of the library (Sec. 3.1 moving average, temporal window, pose gate;
Sec. 3.2 denoising schedule) against the oracle: the same double-precision operations, so the
values and every integer decision are equal, not just close."""
import ctypes

import numpy as np
import pytest

from oracle import la_oracle as O
from paper_2605_31158_amd import la


def test_ema_equals_oracle_bit_for_bit():
    rng = np.random.default_rng(0)
    for _ in range(300):
        alpha = float(rng.uniform(1e-3, 1.0))
        D, prev = float(rng.exponential()), float(rng.exponential())
        assert la.dynamics_ema(D, prev, alpha) == O.ema_dynamics(D, prev, alpha)
        assert la.dynamics_ema(D, None, alpha) == O.ema_dynamics(D, None, alpha)
    assert la.dynamics_ema(2.0, 4.0, 1.0) == 2.0


def test_temporal_window_equals_oracle():
    rng = np.random.default_rng(1)
    for _ in range(2000):
        L_m = int(rng.integers(1, 40))
        kappa = float(rng.uniform(1e-3, 3.0))
        D = float(rng.choice([0.0, kappa, rng.uniform(0, 10), rng.exponential() * 1e-3]))
        assert la.temporal_window(D, kappa, L_m) == O.temporal_window(D, kappa, L_m), (D, kappa, L_m)
    # exact crossings of an integer: L_m kappa / (D + kappa) = 3 exactly
    assert la.temporal_window(1.0, 0.5, 9) == O.temporal_window(1.0, 0.5, 9) == 3


def test_pose_gate_equals_oracle():
    rng = np.random.default_rng(2)
    for _ in range(500):
        n = int(rng.integers(0, 12))
        sims = rng.uniform(0, 1, n).astype(np.float32)
        tau = float(np.float32(rng.uniform(0, 1)))
        if n and rng.random() < 0.3:
            tau = float(sims.max())                          # the boundary: equality revisits
        assert la.pose_revisiting(sims, tau) == O.revisiting(sims.tolist(), tau)


def test_schedule_equals_oracle():
    for K in range(1, 16):
        for reuse in (False, True):
            assert la.denoise_schedule(K, reuse) == O.reuse_source(K, reuse)


def test_policy_arguments_rejected():
    lib = la.lib()
    out = ctypes.c_double()
    L = ctypes.c_int32()
    assert lib.la_dynamics_ema(ctypes.c_double(1.0), None, ctypes.c_double(0.0), ctypes.byref(out)) == la.LA_ERR_ARG
    assert lib.la_dynamics_ema(ctypes.c_double(-1.0), None, ctypes.c_double(0.5), ctypes.byref(out)) == la.LA_ERR_ARG
    assert lib.la_dynamics_ema(ctypes.c_double(1.0), None, ctypes.c_double(0.5), None) == la.LA_ERR_ARG
    assert lib.la_temporal_window(ctypes.c_double(1.0), ctypes.c_double(0.0), 4, ctypes.byref(L)) == la.LA_ERR_ARG
    assert lib.la_temporal_window(ctypes.c_double(1.0), ctypes.c_double(1.0), 0, ctypes.byref(L)) == la.LA_ERR_ARG
    assert lib.la_temporal_window(ctypes.c_double(float("nan")), ctypes.c_double(1.0), 4,
                                  ctypes.byref(L)) == la.LA_ERR_ARG
    sims = np.array([0.5, np.nan], dtype=np.float32)
    assert lib.la_pose_revisiting(sims.ctypes.data_as(ctypes.c_void_p), 2, ctypes.c_float(0.4),
                                  ctypes.byref(L)) == la.LA_ERR_ARG
    assert lib.la_pose_revisiting(None, 3, ctypes.c_float(0.4), ctypes.byref(L)) == la.LA_ERR_ARG
    assert lib.la_denoise_schedule(0, 1, ctypes.byref(L)) == la.LA_ERR_ARG
    p = ctypes.c_void_p(4096)
    ws = ctypes.c_void_p(4096 * 256)
    assert lib.la_latent_mse(p, p, 0, 0, p, ws, la.LATENT_MSE_WS_BYTES, None) == la.LA_ERR_ARG
    assert lib.la_latent_mse(p, p, 10, 2, p, ws, la.LATENT_MSE_WS_BYTES, None) == la.LA_ERR_ARG
    assert lib.la_latent_mse(p, ctypes.c_void_p(4100), 10, 0, p, ws, la.LATENT_MSE_WS_BYTES, None) == la.LA_ERR_ARG
    assert lib.la_latent_mse(p, p, 10, 0, p, ws, 64, None) == la.LA_ERR_WORKSPACE
