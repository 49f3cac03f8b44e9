"""Pins for Algorithm 1's threshold rule in the oracle (Section 3.4): from S_0, add the best
remaining expert while f(S) < tau * f(E), f(S) = sum of the scores of S (Eq. (2)).

* hand-worked cases, and two hand-derived fp32 cases where the summation order decides
  the stopping point (f(E) in index order; f(S) from the starting set in ranking order);
* brute force in exact rationals: the set is a smallest superset of S_0 reaching the
  threshold, and the best of its size (Corollary 3.2);
* the same routing as the fixed budget |S| (reduction), nested sets in tau, tau = 0 and
  tau > 1, the hierarchical selection without per-request picks equal to the flat one.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest

import workloads as W
from oracle import route as R

F32 = np.float32


def test_hand_worked_thresholds():
    s = np.array([0.5, 0.3, 0.15, 0.05], dtype=F32)
    assert R.greedy_threshold(s, set(), 0.4, range(4)) == {0}
    assert R.greedy_threshold(s, set(), 0.7, range(4)) == {0, 1}          # 0.5 < 0.7 <= 0.8
    assert R.greedy_threshold(s, set(), 0.9, range(4)) == {0, 1, 2}       # 0.8 < 0.9 <= 0.95
    assert R.greedy_threshold(s, set(), 0.0, range(4)) == set()           # f(empty) = 0 >= 0
    assert R.greedy_threshold(s, {3}, 0.5, range(4)) == {0, 3}            # 0.05 < 0.5 <= 0.55
    assert R.greedy_threshold(s, {0, 1, 2}, 0.1, range(4)) == {0, 1, 2}   # start is never cut
    assert R.greedy_threshold(s, set(), 2.0, [1, 2]) == {1, 2}            # candidates run out


def test_total_score_is_summed_in_index_order():
    # f(E) in index order: (1 + 2^-24) rounds to 1, + 2^-24 rounds to 1 again: f(E) = 1.
    # With tau = 1 the first pick (1.0) already reaches it.  Summed smallest first,
    # f(E) would be 1 + 2^-23 and no fp32 prefix of the picks would ever reach it.
    e = F32(2.0 ** -24)
    s = np.array([1.0, e, e], dtype=F32)
    assert R.greedy_threshold(s, set(), 1.0, range(3)) == {0}


def test_start_set_is_summed_in_ranking_order():
    # scores 1, 2^-24, 2^-24, 1: f(E) = 2 (index order), tau = 0.5 + 2^-24 gives the target
    # 1 + 2^-23.  S_0 = {0, 1, 2} summed by score (1 first) stays at 1 < target, so expert 3
    # joins; summed smallest first it would be 1 + 2^-23 and S would stop at S_0.
    e = F32(2.0 ** -24)
    s = np.array([1.0, e, e, 1.0], dtype=F32)
    tau = F32(0.5) + F32(2.0 ** -24)
    assert float(tau) == 0.5 + 2.0 ** -24
    assert R.greedy_threshold(s, {0, 1, 2}, float(tau), range(4)) == {0, 1, 2, 3}


def test_target_is_one_fp32_product():
    # tau = fp32(1/3) = 11184811 * 2^-25 and f(E) = 3: the exact product 1 + 2^-25 rounds to
    # 1.0 in fp32, so the first expert (score 1) already reaches it; in float64 it would not.
    tau = float(F32(1.0 / 3.0))
    assert tau == 11184811 * 2.0 ** -25
    s = np.array([1.0, 1.0, 1.0], dtype=F32)
    assert R.greedy_threshold(s, set(), tau, range(3)) == {0}


def _exact(S, s):
    return sum((Fraction(float(s[j])) for j in S), Fraction(0))


@pytest.mark.parametrize("N", [5, 7, 9])
def test_brute_force_smallest_superset(N):
    rng = np.random.default_rng(N)
    checked = 0
    for trial in range(150):
        s = rng.choice(np.array([0.0, 0.05, 0.1, 0.25, 0.3, 0.6, 1.2], dtype=F32), N)
        cand = [j for j in range(N) if rng.random() < 0.85]
        S0 = set(j for j in cand if rng.random() < 0.2)
        tau = float(rng.uniform(0.05, 1.0))
        S = R.greedy_threshold(s, S0, tau, cand)
        target = Fraction(tau) * _exact(range(N), s)
        # skip cases within fp32 rounding of the threshold
        near = [abs(_exact(T, s) - target) for n in range(N + 1)
                for T in itertools.combinations(cand, n) if S0 <= set(T)]
        if min(near) < Fraction(1, 10 ** 5):
            continue
        checked += 1
        ok = [set(T) for n in range(N + 1) for T in itertools.combinations(cand, n)
              if S0 <= set(T) and _exact(T, s) >= target]
        if not ok:                                  # unreachable: every candidate is taken
            assert S == set(cand) | S0
            continue
        m = min(len(T) for T in ok)
        assert len(S) == m and _exact(S, s) >= target, (trial, s, S0, tau, S)
        same = [set(T) for T in itertools.combinations(cand, m) if S0 <= set(T)]
        assert _exact(S, s) == max(_exact(T, s) for T in same)
    assert checked > 100


def test_same_routing_as_the_fixed_budget_of_that_size():
    for seed in range(12):
        h = W.logits_domains(16, 64, 4, seed)
        for tau in (0.4, 0.7, 0.9):
            t = R.route(h, 4, 1, 0, R.THRESHOLD, tau=tau)
            m = t.n_selected
            if m < max(4, t.n_warmup):
                continue
            b = R.route(h, 4, 1, m, R.TOTAL)
            assert np.array_equal(t.sel_mask, b.sel_mask)
            assert np.array_equal(t.ids, b.ids)
            assert np.array_equal(t.w.view(np.uint32), b.w.view(np.uint32))


def test_nested_in_tau_and_limits():
    for seed in range(10):
        h = W.logits_domains(24, 128, 6, seed)
        prev = None
        for tau in (0.0, 0.2, 0.5, 0.8, 0.95, 1.5):
            r = R.route(h, 8, 1, 0, R.THRESHOLD, tau=tau)
            S = set(r.sel_list)
            if prev is not None:
                assert prev <= S
            prev = S
        U = set(int(e) for e in r.vanilla_ids.reshape(-1))
        assert prev == U                                  # tau > 1: every candidate
        r0 = R.route(h, 8, 1, 0, R.THRESHOLD, tau=0.0)    # tau = 0: S_0, topped up to k
        S0 = set(int(e) for e in r0.vanilla_ids[:, :1].reshape(-1))
        assert S0 <= set(r0.sel_list) and r0.n_selected == max(len(S0), 8)


def test_hierarchical_without_request_picks_is_flat():
    for seed in range(8):
        h, off = W.logits_spec(4, 4, 64, 4, seed)
        for tau in (0.5, 0.85):
            a = R.select_hier(h, off, 8, 1, 0, 0, R.THRESHOLD, tau=tau)
            b = R.route(h, 8, 1, 0, R.THRESHOLD, tau=tau)
            assert np.array_equal(a.sel_mask, b.sel_mask)
            assert np.array_equal(a.ids, b.ids)


def test_threshold_needs_tau():
    h = W.logits_domains(4, 16, 2, 0)
    for bad in (None, -0.1, float("nan")):
        with pytest.raises(ValueError):
            R.route(h, 2, 1, 0, R.THRESHOLD, tau=bad)
