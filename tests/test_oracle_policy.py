"""Pins of the oracle's scalar policy (Sec. 3.1 latent dynamics, moving average, temporal window and
pose gate; Sec. 3.2 denoising-cache schedule): closed forms, exact small cases, monotonicity and
brute force, plus planted mistakes that some pin must catch."""
import math

import numpy as np
import pytest

from oracle import la_oracle as O


def test_mse_closed_forms():
    n = 1000
    a = np.arange(n, dtype=np.float64)
    # sum of i^2 over 0..n-1 = (n-1) n (2n-1) / 6
    assert O.latent_mse(a, np.zeros(n)) == (n - 1) * (2 * n - 1) / 6
    rng = np.random.default_rng(0)
    z = rng.standard_normal((4, 16, 30))
    assert O.latent_mse(z, z) == 0.0
    assert O.latent_mse(z, z + 0.25) == 0.0625            # exact: constant offset of 2^-2
    w = rng.standard_normal(z.shape)
    assert O.latent_mse(z, w) == O.latent_mse(w, z)
    assert O.latent_mse(2 * z, 2 * w) == 4 * O.latent_mse(z, w)


def test_mse_reads_bf16_bits_and_rejects_mismatch():
    one, two, three = np.uint16(0x3F80), np.uint16(0x4000), np.uint16(0x4040)
    assert O.latent_mse(np.array([one, two]), np.array([two, three])) == 1.0
    assert O.latent_mse(np.array([three] * 3), np.array([one] * 3)) == 4.0
    with pytest.raises(ValueError):
        O.latent_mse(np.zeros(3), np.zeros(4))
    with pytest.raises(ValueError):
        O.latent_mse(np.zeros(0), np.zeros(0))


def test_ema_closed_forms():
    assert O.ema_dynamics(3.5, None, 0.3) == 3.5           # started by the first valid D_t
    for alpha in (0.25, 0.5, 1.0):
        d = O.ema_dynamics(1.0, None, alpha)
        for k in range(1, 8):
            d = O.ema_dynamics(0.0, d, alpha)
            assert d == pytest.approx((1 - alpha) ** k, abs=1e-15)
    d = None
    for _ in range(5):
        d = O.ema_dynamics(2.0, d, 0.7)
        assert d == pytest.approx(2.0, abs=1e-15)
    assert O.ema_dynamics(5.0, 1.0, 1.0) == 5.0
    for bad in (0.0, -0.1, 1.5):
        with pytest.raises(ValueError):
            O.ema_dynamics(1.0, 1.0, bad)


def test_temporal_window_closed_forms_and_brute_force():
    assert O.temporal_window(0.0, 0.5, 8) == 8
    assert O.temporal_window(0.5, 0.5, 8) == 4              # D_bar = kappa halves the budget
    assert O.temporal_window(0.5, 0.5, 7) == 3
    assert O.temporal_window(1e9, 0.5, 8) == 1              # clipped at 1
    assert O.temporal_window(3.0, 1.0, 1) == 1
    rng = np.random.default_rng(1)
    for _ in range(500):
        L_m = int(rng.integers(1, 20))
        kappa = float(rng.uniform(0.01, 2.0))
        D = float(rng.uniform(0.0, 5.0))
        x = L_m * kappa / (D + kappa)
        want = max(1, max(L for L in range(0, L_m + 1) if L <= x))
        assert O.temporal_window(D, kappa, L_m) == want
    prev = None
    for D in np.linspace(0.0, 10.0, 200):
        L = O.temporal_window(float(D), 0.7, 12)
        assert prev is None or L <= prev
        prev = L


def test_gate_boundaries():
    assert O.revisiting([0.2, 0.7, 0.5], 0.7)               # equality is revisiting
    assert not O.revisiting([0.2, 0.69999], 0.7)
    assert not O.revisiting([], 0.45)
    assert O.keep_retrieved_memory([0.46], 0.45)
    assert not O.keep_retrieved_memory([0.44, 0.1], 0.45)


def test_reuse_schedule():
    assert O.model_calls(1, True) == [True]
    assert O.model_calls(2, True) == [True, True]
    assert O.model_calls(4, True) == [True, False, False, True]
    assert O.model_calls(4, False) == [True] * 4
    for K in range(3, 12):
        calls = O.model_calls(K, True)
        assert sum(calls) == 2 and calls[0] and calls[-1]
    assert O.reuse_source(4, True) == [0, 0, 0, 3]
    assert O.reuse_source(3, False) == [0, 1, 2]
    with pytest.raises(ValueError):
        O.model_calls(0, True)


MUTANTS = {
    "mse over n - 1": ("return math.fsum(((a - b) ** 2).tolist()) / a.size",
                       "return math.fsum(((a - b) ** 2).tolist()) / (a.size - 1)"),
    "ema weights swapped": ("return alpha * D_t + (1.0 - alpha) * D_bar_prev",
                            "return (1.0 - alpha) * D_t + alpha * D_bar_prev"),
    "window rounds up": ("math.floor(L_m * kappa / (D_bar + kappa))", "math.ceil(L_m * kappa / (D_bar + kappa))"),
    "strict gate": ("max(float(s) for s in similarities) >= tau_pose", "max(float(s) for s in similarities) > tau_pose"),
    "last step reused": ("[i == 0 or i == K - 1 for i in range(K)]", "[i == 0 for i in range(K)]"),
    "no reuse at K = 3": ("if not reuse or K <= 2:", "if not reuse or K <= 3:"),
}


def _pins():
    return [fn for name, fn in sorted(globals().items()) if name.startswith("test_") and name != "test_pins_catch_mutant"]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_mutant(name, monkeypatch):
    import inspect
    import sys
    import types
    old, new = MUTANTS[name]
    src = inspect.getsource(O)
    assert src.count(old) == 1, old
    mod = types.ModuleType("oracle_mutant_policy")
    exec(compile(src.replace(old, new), "oracle_mutant_policy", "exec"), mod.__dict__)
    monkeypatch.setattr(sys.modules[__name__], "O", mod)
    caught = 0
    for fn in _pins():
        try:
            fn()
        except Exception:
            caught += 1
    assert caught, f"no pin catches the planted mistake: {name}"
