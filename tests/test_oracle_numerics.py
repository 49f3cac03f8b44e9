"""Pins of the oracle's fp32 gate numerics against float64 mathematics (Section 2.2 gates)."""
import math

import numpy as np
import pytest

from oracle.numerics import exp_ref, seq_sum, softmax_dense, softmax_ranked

F32 = np.float32


def _ulps(got, ref):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    ulp = np.spacing(np.abs(ref).astype(F32)).astype(np.float64)
    return np.abs(got - ref) / ulp


def test_exp_ref_within_2ulp_dense_grid():
    x = np.linspace(-80.0, 0.0, 800001).astype(F32)
    rng = np.random.default_rng(1)
    x = np.concatenate([x, -np.abs(rng.standard_normal(200000) * 8).astype(F32),
                        -rng.random(100000).astype(F32) * F32(1e-3)])
    x = x[x >= F32(-80.0)]
    err = _ulps(exp_ref(x), np.exp(x.astype(np.float64)))
    assert err.max() <= 2.0, (err.max(), x[err.argmax()])


def test_exp_ref_special_values():
    assert exp_ref(F32(0.0)) == F32(1.0)
    assert exp_ref(F32(-0.0)) == F32(1.0)
    assert exp_ref(F32(-80.5)) == F32(0.0)
    assert exp_ref(F32(-1000.0)) == F32(0.0)
    assert exp_ref(F32(-80.0)) > 0
    # exp(-ln 2) = 1/2 to within an ulp
    assert abs(float(exp_ref(F32(-math.log(2.0)))) - 0.5) <= 2 ** -24
    with pytest.raises(ValueError):
        exp_ref(F32(0.5))
    with pytest.raises(ValueError):
        exp_ref(F32(np.nan))


def test_exp_ref_monotone():
    x = np.sort(np.linspace(-80.0, 0.0, 200001).astype(F32))
    y = exp_ref(x)
    assert np.all(np.diff(y.astype(np.float64)) >= 0)


def test_seq_sum_is_left_to_right():
    # (1e8 + 1) - 1e8 == 0 in fp32 left to right; a pairwise or reordered sum gives 1
    assert seq_sum([F32(1e8), F32(1.0), F32(-1e8)]) == F32(0.0)
    assert seq_sum([F32(1.0), F32(1e8), F32(-1e8)]) == F32(0.0)
    assert seq_sum([F32(1e8), F32(-1e8), F32(1.0)]) == F32(1.0)
    assert seq_sum([]) == F32(0.0)


def _softmax_rel_bound(h, n_terms):
    """Relative error bound of the fp32 recipe against the exact softmax.

    fl(h_r - m) is off by at most |h_r - m| 2^-24 (relative change of exp),
    exp_ref adds at most 2 ulp (< 2^-22 relative), the sequential sum adds at
    most (n-1) 2^-24 on top of its terms' errors, the division 2^-24.
    """
    x = float(np.max(np.abs(h.astype(np.float64) - float(np.max(h)))))
    per_term = x * 2.0 ** -24 + 2.0 ** -22
    return 2 * per_term + (n_terms + 1) * 2.0 ** -24


@pytest.mark.parametrize("k", [1, 2, 4, 8, 32])
def test_softmax_ranked_matches_float64(k):
    rng = np.random.default_rng(k)
    for _ in range(300):
        h = np.sort(rng.standard_normal(k).astype(F32) * F32(3))[::-1]
        g = softmax_ranked(h)
        e = np.exp(h.astype(np.float64) - float(h[0]))
        ref = e / e.sum()
        rel = np.abs(g.astype(np.float64) - ref) / ref
        assert rel.max() <= _softmax_rel_bound(h, k)
        assert np.all(np.diff(g.astype(np.float64)) <= 0)           # non-increasing in rank
        assert abs(float(np.sum(g.astype(np.float64))) - 1.0) <= k * 2 ** -23


def test_softmax_ranked_single_and_ties():
    assert softmax_ranked([F32(3.0)])[0] == F32(1.0)
    g = softmax_ranked([F32(0.5)] * 4)
    assert np.all(g == F32(0.25))
    # a gap beyond the underflow point gives exact zeros
    g = softmax_ranked([F32(0.0), F32(-100.0)])
    assert g[0] == F32(1.0) and g[1] == F32(0.0)


def test_softmax_sums_in_the_stated_order():
    """Convention pin: the denominator is summed in rank order (ranked) / index order (dense).

    With e_0 = 1 and two terms e in (2^-25, 2^-24): left to right 1 + e rounds back to 1
    twice, so Z = 1 and g_0 = 1 exactly; summing the small terms first gives Z = 1 + 2^-23.
    """
    x = F32(-16.64)
    e = float(exp_ref(x))
    assert 2.0 ** -25 < e < 2.0 ** -24
    g = softmax_ranked([F32(0.0), x, x])
    assert g[0] == F32(1.0)
    gd = softmax_dense([x, x, F32(0.0)])          # index order: small terms first
    assert gd[2] == F32(1.0) / F32(1.0 + 2.0 ** -23) and gd[2] < F32(1.0)


def test_softmax_dense_matches_float64():
    rng = np.random.default_rng(7)
    for N in (8, 16, 128, 256):
        h = rng.standard_normal(N).astype(F32) * F32(2)
        g = softmax_dense(h)
        e = np.exp(h.astype(np.float64) - float(h.max()))
        ref = e / e.sum()
        rel = np.abs(g.astype(np.float64) - ref) / ref
        assert rel.max() <= _softmax_rel_bound(h, N)


def test_scores_sum_tokens_in_ascending_order():
    """s_j = sum_i g_ij is summed one token at a time in ascending token order (Eq. (2) in
    fp32).  Hand-derived: expert A's gates are fp32(1/3), 1/4, fp32(1/6) in token order, so
    ((1/3 + 1/4) + 1/6) = 0.75000006 (0x3F400001) while the reverse order gives exactly 0.75,
    which expert B (lower index) has too; with a total budget whose last slot goes to one of
    them, the ascending order selects A, and the reverse order would select B."""
    from helpers import score_order_case
    from oracle import route as R
    h, k, M, A, B = score_order_case()
    third, sixth = F32(1) / F32(3), F32(1) / F32(6)          # correctly rounded quotients
    assert third == F32(0.3333333432674408) and sixth == F32(0.1666666716337204)
    asc = F32(F32(third + F32(0.25)) + sixth)
    rev = F32(F32(sixth + F32(0.25)) + third)
    assert asc.view(np.uint32) == 0x3F400001 and rev == F32(0.75)
    r = R.route(h, k, 0, M)
    assert r.scores[A].view(np.uint32) == asc.view(np.uint32)
    assert r.scores[B] == F32(0.75)
    assert r.sel_list == [A, 3, 4, 5, 6, 7]
