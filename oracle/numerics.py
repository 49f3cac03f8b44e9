"""fp32 numerics of the gates (oracle side).

The paper writes the gate of a chosen expert as exp(h_i) / sum_{j in T} exp(h_j)
(Section 2.2) but fixes no floating-point recipe.  Selection is a discrete
decision taken on sums of these gates, so both implementations evaluate them in
the same fp32 steps, each one an IEEE round-to-nearest-even operation:

exp_ref(x), for x <= 0 (always the case here: x = h - max h):
  * x < -80                        -> 0.0
  * n = rint(x * log2(e))          (fp32 multiply, ties to even)
  * r = (x - n*ln2_hi) - n*ln2_lo  (Cody-Waite two-constant reduction; ln2_hi keeps
                                    15 significant bits so n*ln2_hi is exact)
  * p = Taylor polynomial of degree 7 with coefficients 1/i! (fp32), Horner form,
        separate multiply and add (no fused multiply-add)
  * result = p * 2^n (exact scaling)
  Accuracy: within 2 ulp of the float64 exponential on [-80, 0] (tested).

softmax over a ranked list h_0 >= h_1 >= ... (rank order):
  * m = h_0; e_r = exp_ref(h_r - m)
  * Z = ((e_0 + e_1) + e_2) + ...  sequential in rank order
  * g_r = e_r / Z  (correctly rounded division)
"""
from __future__ import annotations

import math

import numpy as np

F32 = np.float32

LOG2E = F32(1.0 / math.log(2.0))
LN2_HI = F32(0.693145751953125)                 # 0x3f317200
LN2_LO = F32(math.log(2.0) - 0.693145751953125)
TAYLOR = [F32(1.0 / math.factorial(i)) for i in range(8)]
UNDERFLOW = F32(-80.0)


def exp_ref(x) -> np.ndarray:
    """Elementwise fp32 exp for x <= 0, following the recipe in the module docstring."""
    x = np.asarray(x, dtype=F32)
    if np.any(np.isnan(x)) or np.any(x > 0):
        raise ValueError("exp_ref: defined for finite x <= 0")
    n = np.rint(x * LOG2E)
    r = (x - n * LN2_HI) - n * LN2_LO
    p = TAYLOR[7]
    for i in range(6, -1, -1):
        p = p * r + TAYLOR[i]
    out = np.ldexp(p.astype(F32), n.astype(np.int32)).astype(F32)
    return np.where(x < UNDERFLOW, F32(0.0), out).astype(F32)


def seq_sum(values) -> F32:
    """fp32 sum taken strictly left to right, starting from +0.0."""
    z = F32(0.0)
    for v in values:
        z = F32(z + F32(v))
    return z


def softmax_ranked(h_ranked) -> np.ndarray:
    """Gates of a list of logits given in rank order (largest first), fp32."""
    h = np.asarray(h_ranked, dtype=F32)
    if h.size == 0:
        return h.copy()
    e = exp_ref(h - h[0])
    z = seq_sum(e)
    return (e / z).astype(F32)


def softmax_dense(h_row) -> np.ndarray:
    """Softmax over all experts of one token (dense-gate reading), fp32.

    m = max over the row; sum taken in ascending expert index.
    """
    h = np.asarray(h_row, dtype=F32)
    e = exp_ref(h - h.max())
    z = seq_sum(e)
    return (e / z).astype(F32)
