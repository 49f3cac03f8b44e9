"""The GPU tests' output tolerance (CPU checks of the helper itself)."""
import numpy as np
import torch

from helpers import half_ulp_bf16, rounding_excess


def test_half_ulp_of_bf16():
    # 8 significant bits: the unit in the last place at 1 is 2^-7, in [4, 8) it is 2^-5
    assert half_ulp_bf16(1.0) == 2.0 ** -8
    assert half_ulp_bf16(1.99) == 2.0 ** -8
    assert half_ulp_bf16(-4.11) == 2.0 ** -6
    assert half_ulp_bf16(0.0) == 0.0


def test_exactly_rounded_values_have_no_excess():
    rng = np.random.default_rng(0)
    y = rng.standard_normal(100000) * np.exp(rng.uniform(-3, 3, 100000))
    rounded = torch.tensor(y, dtype=torch.float64).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.all(np.abs(rounded - y) <= half_ulp_bf16(y))
    assert rounding_excess(rounded, y) <= 0.0
    # one more unit in the last place away from the exact value, at the largest value, is an
    # excess of at least half a unit
    i = int(np.argmax(np.abs(y)))
    bad = rounded.copy()
    away = np.sign(rounded[i] - y[i]) or np.sign(y[i])
    bad[i] += 2 * half_ulp_bf16(y[i]) * away
    rms = np.sqrt(np.mean(y ** 2))
    assert rounding_excess(bad, y) >= half_ulp_bf16(y[i]) / rms
