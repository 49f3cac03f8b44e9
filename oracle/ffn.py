"""MoE layer output with SwiGLU experts (oracle side), in float64.

Section 2.1: y = sum_i g_i(x) E_i(x) over the routed experts, plus the always-on
shared experts when given.  Each expert is a SwiGLU FFN in nn.Linear [out, in]
layout:  E(x) = W2 (silu(W1 x) * (W3 x)),  silu(z) = z / (1 + e^-z),
W1, W3 in R^{f x d}, W2 in R^{d x f}.  Inputs are bf16 bit patterns (exact in
float64), or expert weights already in float64 (the FP8 weights below, decoded
and scaled exactly); nothing is rounded until the caller compares.

FP8 expert weights (the paper is silent on precision): OCP FP8 E4M3FN codes
(1 sign bit, 4 exponent bits with bias 7, 3 mantissa bits; exponent field 0 is
subnormal, code 0x7F / 0xFF is NaN, no infinities, largest finite 448) with one
fp32 scale per output row: w[r, c] = decode(q[r, c]) * scale[r].

MXFP4 expert weights (OCP Microscaling formats, MXFP4): FP4 E2M1 element codes
(1 sign bit, 2 exponent bits with bias 1, 1 mantissa bit; exponent field 0 is
subnormal with value m / 2; no infinities or NaN; largest 6), two per byte with
element 2c in the low nibble; every block of 32 consecutive elements of a row
(along the input index, the reduction dimension) shares one E8M0 scale byte e,
whose value is 2^(e - 127) (e = 255 is NaN):
w[r, c] = decode(q[r, c]) * 2^(e[r, c // 32] - 127).
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def silu(z):
    return z / (1.0 + np.exp(-z))


def decode_e4m3(codes) -> np.ndarray:
    """OCP FP8 E4M3FN codes -> float64 values (NaN for 0x7F and 0xFF)."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    sign = np.where(c >> 7, -1.0, 1.0)
    e = (c >> 3) & 15
    m = (c & 7).astype(np.float64)
    v = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    v = sign * v
    return np.where((e == 15) & ((c & 7) == 7), np.nan, v)


_E4M3_VALUES = None


def dequant_rows(codes, scale) -> np.ndarray:
    """Weights of one FP8 matrix: decode(q[r, c]) * scale[r] in float64 (exact); the codes are
    looked up in the table of all 256 decoded values."""
    global _E4M3_VALUES
    if _E4M3_VALUES is None:
        _E4M3_VALUES = decode_e4m3(np.arange(256, dtype=np.uint8))
    return _E4M3_VALUES[np.asarray(codes, dtype=np.uint8)] * \
        np.asarray(scale, dtype=np.float32).astype(np.float64)[:, None]


def decode_e2m1(codes) -> np.ndarray:
    """FP4 E2M1 codes (low 4 bits of each value) -> float64 values."""
    c = np.asarray(codes, dtype=np.uint8).astype(np.int64) & 15
    sign = np.where(c >> 3, -1.0, 1.0)
    e = (c >> 1) & 3
    m = (c & 1).astype(np.float64)
    v = np.where(e == 0, m / 2.0, (1.0 + m / 2.0) * np.exp2(e - 1.0))
    return sign * v


def decode_e8m0(codes) -> np.ndarray:
    """E8M0 scale bytes -> float64 2^(e - 127) (NaN for 255)."""
    e = np.asarray(codes, dtype=np.uint8).astype(np.int64)
    return np.where(e == 255, np.nan, np.exp2(e - 127.0))


_E2M1_VALUES = None


def dequant_mx(packed, scales) -> np.ndarray:
    """Weights of one MXFP4 matrix, float64 [rows, K] (exact): packed codes [rows, K / 2]
    (element 2c in the low nibble of byte c), E8M0 scales [rows, K / 32]."""
    global _E2M1_VALUES
    if _E2M1_VALUES is None:
        _E2M1_VALUES = decode_e2m1(np.arange(16, dtype=np.uint8))
    b = np.asarray(packed, dtype=np.uint8)
    rows, half = b.shape
    codes = np.empty((rows, 2 * half), dtype=np.uint8)
    codes[:, 0::2] = b & 15
    codes[:, 1::2] = b >> 4
    scale = decode_e8m0(scales)
    assert scale.shape == (rows, 2 * half // 32), "one scale per 32 elements of a row"
    return _E2M1_VALUES[codes] * np.repeat(scale, 32, axis=1)


def _as_f64(w) -> np.ndarray:
    w = np.asarray(w)
    return bf16_to_f64(w) if w.dtype == np.uint16 else w.astype(np.float64)


def expert_ffn(x, w1, w3, w2) -> np.ndarray:
    """SwiGLU expert applied to the rows of x (float64 [t,d]) -> float64 [t,d]; the weights
    are bf16 bit patterns (uint16) or float64 values."""
    W1 = _as_f64(w1)
    W3 = _as_f64(w3)
    W2 = _as_f64(w2)
    a = x @ W1.T
    b = x @ W3.T
    return (silu(a) * b) @ W2.T


def router_logits(x_bits, wg_bits) -> np.ndarray:
    """h = W_g x for every token (Section 2.2): float64 [T, N] from bf16 x [T,d] and
    W_g [N,d]."""
    return bf16_to_f64(x_bits) @ bf16_to_f64(wg_bits).T


def moe_forward(x_bits, ids, w, expert, rows=None, local=None, shared=()) -> np.ndarray:
    """y[i] = sum_r w[i,r] * E_{ids[i,r]}(x_i) + sum_s E^s_s(x_i) for the tokens in ``rows``
    (default: all); the second sum runs over the always-on shared experts of Section 2.1.

    ``expert(e)`` returns the bf16 bit arrays (w1 [f,d], w3 [f,d], w2 [d,f]) of expert e;
    ``shared`` is a sequence of such triples.  With ``local`` (a set of experts, those one
    GPU group hosts under expert parallelism, Section 5) only the terms of those routed
    experts are summed: that group's share of y.
    Returns float64 [len(rows), d].
    """
    X = bf16_to_f64(x_bits)
    ids = np.asarray(ids)
    w = np.asarray(w, dtype=np.float64)
    rows = list(range(X.shape[0])) if rows is None else [int(i) for i in rows]
    y = np.zeros((len(rows), X.shape[1]), dtype=np.float64)
    by_expert: dict[int, list[tuple[int, int]]] = {}
    for p, i in enumerate(rows):
        for r in range(ids.shape[1]):
            if local is None or int(ids[i, r]) in local:
                by_expert.setdefault(int(ids[i, r]), []).append((p, r))
    for e in sorted(by_expert):
        pairs = by_expert[e]
        w1, w3, w2 = expert(e)
        out = expert_ffn(X[[rows[p] for p, _ in pairs]], w1, w3, w2)
        for q, (p, r) in enumerate(pairs):
            y[p] += w[rows[p], r] * out[q]
    for w1, w3, w2 in shared:
        y += expert_ffn(X[rows], w1, w3, w2)
    return y


def combine(outputs, ids, w, d, rows=None, local=None) -> np.ndarray:
    """The routed sum of Section 2.1 from expert outputs on every token of the batch:
    y[i] = sum_r w[i,r] * outputs[ids[i,r]][i], ranks r in order, for the tokens in ``rows``
    (default: all).  ``outputs[e]`` is float64 [T, d], expert e applied to every token
    (expert_ffn over all rows of x); with ``local`` only those experts' terms are summed.
    Returns float64 [len(rows), d]."""
    ids = np.asarray(ids)
    w = np.asarray(w, dtype=np.float64)
    rows = list(range(ids.shape[0])) if rows is None else [int(i) for i in rows]
    y = np.zeros((len(rows), d), dtype=np.float64)
    for p, i in enumerate(rows):
        for r in range(ids.shape[1]):
            e = int(ids[i, r])
            if local is None or e in local:
                y[p] += w[i, r] * outputs[e][i]
    return y
