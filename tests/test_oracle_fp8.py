"""Pins for the FP8 expert weights of the oracle (OCP FP8 E4M3FN codes, one fp32 scale per
output row).

* the decoder against values fixed by the format (1.0, 448, the smallest subnormal 2^-9,
  the smallest normal 2^-6, signed zero, NaN) and against torch's float8_e4m3fn on all 256
  codes (an independent library routine);
* the per-row quantizer of the input module: every code is the nearest E4M3 value of
  w / scale (ties to even), so the error is at most half an E4M3 step;
* a SwiGLU expert on dequantized FP8 weights equals the bf16 path on the same values when
  the scales are powers of two (the dequantized weights are then exactly bf16).
"""
import numpy as np
import torch

import workloads as W
from oracle import ffn as O


def test_decoder_fixed_values():
    d = O.decode_e4m3(np.array([0x38, 0x7E, 0x01, 0x08, 0xB8, 0x00, 0x80, 0x7F, 0xFF, 0x07,
                                0x3C], np.uint8))
    assert list(d[:5]) == [1.0, 448.0, 2.0 ** -9, 2.0 ** -6, -1.0]
    assert d[5] == 0.0 and np.signbit(d[6]) and d[6] == 0.0
    assert np.isnan(d[7]) and np.isnan(d[8])
    assert d[9] == 7 * 2.0 ** -9 and d[10] == 1.5


def test_decoder_matches_torch_on_every_code():
    codes = np.arange(256, dtype=np.uint8)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = O.decode_e4m3(codes)
    both_nan = np.isnan(ref) & np.isnan(got)
    assert np.all(both_nan | (ref == got))
    assert np.sum(np.isnan(got)) == 2


def test_quantizer_is_round_to_nearest():
    w = W.expert_matrix(3, "w1", 96, 40, 1)
    q, s = W.quantize_rows_e4m3(w)
    assert q.dtype == torch.uint8 and s.dtype == torch.float32
    vals = O.decode_e4m3(np.arange(256, dtype=np.uint8))
    finite = np.sort(np.unique(vals[np.isfinite(vals)]))
    target = (w.float() / s[:, None]).double().numpy()
    deq = O.decode_e4m3(q.numpy())
    assert np.all(np.isfinite(deq)) and np.max(np.abs(deq)) <= 448.0
    # the chosen code is a nearest representable value of the target
    idx = np.searchsorted(finite, target)
    lo = finite[np.clip(idx - 1, 0, len(finite) - 1)]
    hi = finite[np.clip(idx, 0, len(finite) - 1)]
    best = np.minimum(np.abs(target - lo), np.abs(target - hi))
    assert np.all(np.abs(deq - target) <= best + 1e-12)
    # each row's largest magnitude maps onto 448
    assert np.allclose(np.max(np.abs(deq), axis=1), 448.0)


def test_fp8_expert_equals_bf16_expert_with_power_of_two_scales():
    rng = np.random.default_rng(0)
    d, f, t = 64, 96, 5
    codes = [rng.integers(0, 256, size=shape).astype(np.uint8) for shape in ((f, d), (f, d), (d, f))]
    for c in codes:
        c[(c & 0x7F) == 0x7F] = 0x3C                          # no NaN codes
    scales = [np.exp2(rng.integers(-12, -6, size=c.shape[0])).astype(np.float32) for c in codes]
    deq = [O.dequant_rows(c, s) for c, s in zip(codes, scales)]
    bits = [torch.tensor(m, dtype=torch.float32).to(torch.bfloat16).view(torch.int16).numpy()
            .view(np.uint16) for m in deq]
    assert all(np.array_equal(O.bf16_to_f64(b), m) for b, m in zip(bits, deq))   # exact in bf16
    x = O.bf16_to_f64(W.bf16_bits(W.activations(t, d, 0)))
    assert np.array_equal(O.expert_ffn(x, *deq), O.expert_ffn(x, *bits))
