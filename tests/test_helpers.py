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


def test_timeline_summary_of_block_stamps():
    """The profiling driver's block-timeline summary on hand-made stamps (100 MHz ticks):
    two gate/up blocks, a persistent down block of two units, one on XCD 0 and one on 1."""
    import numpy as np
    from paper_2602_07265_amd.profiling import timeline_of

    gu = np.zeros((16384, 2), np.uint64)
    gu[0] = (1000, 3000)          # 0-20 µs
    gu[1] = (1000, 2000)          # 0-10 µs
    dn = np.zeros((16384, 2), np.uint64)
    un = np.zeros((1024, 33), np.uint64)
    un[0, :3] = (3200, 4200, 5000)     # starts 22 µs after t0; units of 10 and 8 µs
    un[1, :2] = (3300, 4400)
    out = timeline_of({"gate_up": gu, "down": dn, "down_units": un})
    g = out["gate_up"]
    assert g["blocks"] == 2 and g["span"] == 20.0 and g["block_us"][0] == 15.0
    assert g["running_per_10us"] == [2, 1]
    d = out["down_persistent"]
    assert d["blocks"] == 2 and d["unit_us"][0][0] == 10.5 and d["unit_us"][1][0] == 8.0
    assert d["end_by_xcd"] == [40.0, 34.0]
    assert out["gap_us"] == 2.0 and "down" not in out
