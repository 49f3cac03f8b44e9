"""Pins for the MXFP4 weight format in the oracle (OCP MX: E2M1 elements, one E8M0 scale per
32 elements along a row) and for the seeded quantizer that prepares such weights.

* decode_e2m1 against the format's table of values (tests/golden/e2m1_values.json);
* decode_e8m0 against torch's float8_e8m0fnu conversion on all 256 codes;
* dequant_mx: nibble order and block boundaries on hand-built rows;
* the quantizer: the format's ties-to-even and saturation on hand-derived values, exact
  round trips of representable blocks, the per-element error bound of the chosen scale;
* the FFN on MXFP4 weights equals the FFN on the same values given as bf16 (every MXFP4
  weight of a normal scale is exact in bf16).
"""
import json
import os

import numpy as np
import pytest
import torch

import workloads as W
from oracle import ffn as OF

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "e2m1_values.json")


def test_e2m1_against_the_format_table():
    g = json.load(open(GOLDEN))
    got = OF.decode_e2m1(np.arange(16, dtype=np.uint8))
    want = np.array([g["codes"][str(c)] for c in range(16)])
    assert np.array_equal(got, want)
    assert np.array_equal(np.signbit(got), np.signbit(want))    # -0.0 for code 8
    pos = got[:8]
    assert pos.max() == g["max_normal"] and pos[2] == g["min_normal"] and pos[1] == g["subnormal"]
    assert np.all(np.diff(pos) > 0)


def test_e8m0_against_torch_on_every_code():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e8m0fnu).to(torch.float32).numpy()
    got = OF.decode_e8m0(codes)
    assert np.isnan(got[255]) and np.isnan(ref[255])
    assert np.array_equal(got[:255], ref[:255].astype(np.float64))


def test_dequant_nibble_order_and_blocks():
    # row 0: block 0 scale 2^0, block 1 scale 2^-3; elements 0, 1 = codes 0x3, 0x5 (byte 0x53)
    packed = np.zeros((2, 32), dtype=np.uint8)
    packed[0, 0] = 0x53          # element 0 = 1.5, element 1 = 3.0
    packed[0, 15] = 0x7F         # element 30 = -6.0, element 31 = 6.0 (block 0)
    packed[0, 16] = 0x12         # element 32 = 1.0, element 33 = 0.5 (block 1)
    packed[1, 31] = 0xA0         # row 1: element 62 = 0, element 63 = -1.0
    scales = np.array([[127, 124], [130, 130]], dtype=np.uint8)
    w = OF.dequant_mx(packed, scales)
    assert w.shape == (2, 64)
    assert (w[0, 0], w[0, 1], w[0, 30], w[0, 31]) == (1.5, 3.0, -6.0, 6.0)
    assert (w[0, 32], w[0, 33]) == (1.0 / 8, 0.5 / 8)
    assert (w[1, 62], w[1, 63]) == (0.0, -8.0)
    assert np.count_nonzero(w) == 7


@pytest.mark.parametrize("v,q", [(0.25, 0.0), (0.75, 1.0), (1.25, 1.0), (1.75, 2.0),
                                 (2.5, 2.0), (3.5, 4.0), (5.0, 4.0), (5.5, 6.0), (7.0, 6.0),
                                 (-2.6, -3.0), (0.2, 0.0), (0.3, 0.5)])
def test_quantizer_rounding_and_saturation(v, q):
    # the first element fixes the block's scale at 2^0 (max |v| in [4, 8): X = 2 - 2)
    row = torch.zeros(1, 32)
    row[0, 0] = 6.0
    row[0, 1] = v
    p, e = W.quantize_mx_e2m1(row)
    assert int(e[0, 0]) == 127
    assert OF.dequant_mx(p.numpy(), e.numpy())[0, 1] == q


def test_quantizer_round_trip_and_error_bound():
    g = torch.Generator().manual_seed(5)
    vals = torch.tensor([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])
    idx = torch.randint(0, 8, (64, 128), generator=g)
    sign = torch.where(torch.rand(64, 128, generator=g) < 0.5, -1.0, 1.0)
    blk_exp = torch.randint(-20, 5, (64, 4), generator=g).float()
    exact = vals[idx] * sign * torch.exp2(blk_exp).repeat_interleave(32, dim=1)
    exact[:, ::32] = 6.0 * torch.exp2(blk_exp)             # each block reaches its max
    p, e = W.quantize_mx_e2m1(exact)
    assert np.array_equal(OF.dequant_mx(p.numpy(), e.numpy()), exact.double().numpy())
    w = torch.randn(32, 256, generator=g) * 0.02
    p, e = W.quantize_mx_e2m1(w)
    deq = OF.dequant_mx(p.numpy(), e.numpy())
    scale = OF.decode_e8m0(e.numpy()).repeat(32, axis=1)
    a = np.abs(w.double().numpy()) / scale                  # in [0, 8): the block max is < 8
    half_step = np.where(a < 2, 0.25, np.where(a < 4, 0.5, 1.0)) * scale
    assert np.all(np.abs(deq - w.double().numpy()) <= np.maximum(half_step,
                                                                  (a > 6) * (a - 6) * scale))


def test_ffn_on_mxfp4_weights_equals_bf16_path_on_the_same_values():
    d, f = 64, 96
    torch.manual_seed(3)
    mats = [torch.randn(f, d) * 0.05, torch.randn(f, d) * 0.05, torch.randn(d, f) * 0.05]
    deq = []
    for m in mats:
        p, e = W.quantize_mx_e2m1(m)
        deq.append(OF.dequant_mx(p.numpy(), e.numpy()))
    bits = [torch.from_numpy(v.astype(np.float32)).to(torch.bfloat16) for v in deq]
    for v, b in zip(deq, bits):                              # exact in bf16
        assert np.array_equal(b.float().double().numpy(), v)
    x = W.bf16_bits(torch.randn(5, d).to(torch.bfloat16))
    a = OF.expert_ffn(OF.bf16_to_f64(x), *deq)
    b = OF.expert_ffn(OF.bf16_to_f64(x), *[W.bf16_bits(t) for t in bits])
    assert np.array_equal(a, b)
