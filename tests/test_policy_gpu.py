"""GPU latent dynamics D_t = MSE(z_{t-1}, z_{t-2}) (Sec. 3.1) against the oracle's exact fp64 mean:
relative error <= 1e-6 (fp32 sums of at most 8 squares, fp64 beyond), fp32 and bf16 latents, sizes
from one value to several grid strides with ragged tails, and bit-identical repeats."""
import numpy as np
import pytest
import torch

from oracle import la_oracle as O
from paper_2605_31158_amd import la
from helpers import say

pytestmark = pytest.mark.gpu

SIZES = [1, 3, 7, 8, 9, 1000, 4 * 4096 + 5, 399360, 10_000_003]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("n", SIZES)
def test_latent_mse_matches_oracle(n, dtype):
    say(f"[mse] n={n} {dtype}")
    rng = np.random.default_rng(n)
    a = rng.standard_normal(n, dtype=np.float32)
    b = a + np.float32(0.05) * rng.standard_normal(n, dtype=np.float32)
    if dtype == "bf16":
        from paper_2605_31158_amd.workloads import f32_to_bf16_bits
        a_bits, b_bits = f32_to_bf16_bits(a), f32_to_bf16_bits(b)
        ga, gb = la.bf16_from_bits(a_bits), la.bf16_from_bits(b_bits)
        want = O.latent_mse(a_bits, b_bits)
    else:
        ga, gb = torch.from_numpy(a).cuda(), torch.from_numpy(b).cuda()
        want = O.latent_mse(a, b)
    got = la.latent_mse(ga, gb)
    again = la.latent_mse(ga, gb)
    torch.cuda.synchronize()
    g = float(got.item())
    assert abs(g - want) <= 1e-6 * want, (g, want)
    assert g == float(again.item())


def test_latent_mse_identical_and_shifted():
    z = torch.randn(4, 16, 60, 104, device="cuda")
    assert float(la.latent_mse(z, z).item()) == 0.0
    got = float(la.latent_mse(z, z + 0.5).item())
    want = O.latent_mse(z.cpu().numpy(), (z + 0.5).cpu().numpy())
    assert abs(got - want) <= 1e-6 * want
