"""Pins for the expert-parallel selection of the oracle (Section 5, Eq. (5), Algorithms 5-6).

* hand-worked cases that fix each reading of Algorithm 5 (cap per group, exhausted group,
  the loop condition tested per round, warm-up experts never cut);
* brute force of Eq. (5): with no warm-up and at least m_g candidates on every group the
  result is a maximiser of f(S) under MaxLoad(S) <= m_g, in exact rationals, and meets the
  balance bound MaxLoad(S) = ceil(|S| / G) of Section 5.1;
* an independent closed form of the rounds (each group's picks are its best min(R, a_g)
  candidates, R the number of rounds the loop runs);
* reductions: one group is the flat total-budget selection, one expert per group with
  m_g = 1 is plain top-k routing;
* invariants on random batches.
"""
import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

import workloads as W
from oracle import route as R


# ----------------------------------------------------------------------------- hand-worked

S8 = np.array([0.9, 0.8, 0.1, 0.05, 0.5, 0.4, 0.3, 0.0], dtype=np.float32)
G8 = [0, 0, 0, 0, 1, 1, 1, 1]


def test_two_groups_take_turns():
    # round 1: group 0 takes 0 (0.9), group 1 takes 4 (0.5); round 2: 1 (0.8) and 5 (0.4)
    assert R.gpu_aware_greedy(S8, G8, 2, 2, set(), range(8)) == {0, 1, 4, 5}


def test_warmup_over_the_cap_is_kept_and_counts():
    # S_0 = {0, 2, 3} puts 3 > m_g = 2 experts on group 0: it takes no more; group 1 takes
    # 4, then |S| = 4 = m_g * G ends the loop.  MaxLoad 3 > ceil(4 / 2): the balance bound
    # of Section 5.1 needs S_0 to be empty.
    S = R.gpu_aware_greedy(S8, G8, 2, 2, {0, 2, 3}, range(8))
    assert S == {0, 2, 3, 4}
    assert max(R.group_loads(S, G8, 2)) == 3 > math.ceil(len(S) / 2)


def test_exhausted_group_is_skipped_and_others_stop_at_the_cap():
    # Candidates {0..4}: group 1 has only expert 4.  m_g = 3: rounds add {0, 4}, {1}, {2};
    # the fourth round adds nothing (group 0 at its cap, group 1 empty) and ends the loop.
    S = R.gpu_aware_greedy(S8, G8, 2, 3, set(), [0, 1, 2, 3, 4])
    assert S == {0, 1, 2, 4}


def test_a_started_round_runs_over_all_groups():
    # G = 3, m_g = 2, S_0 = {0, 1, 2} on group 0 (load 3).  |S| = 3 < 6: round 1 adds the
    # best of groups 1 and 2 (|S| = 5 < 6); round 2 adds the next best of groups 1 and 2,
    # so |S| ends at 7 > m_g * G.
    s = np.array([0.1, 0.2, 0.3, 0.05, 0.9, 0.8, 0.7, 0.6, 0.5], dtype=np.float32)
    g = [0, 0, 0, 0, 1, 1, 2, 2, 2]
    S = R.gpu_aware_greedy(s, g, 3, 2, {0, 1, 2}, range(9))
    assert S == {0, 1, 2, 4, 5, 6, 7}


def test_ties_go_to_the_lower_index():
    s = np.array([0.5, 0.5, 0.5, 0.5], dtype=np.float32)
    assert R.gpu_aware_greedy(s, [0, 1, 0, 1], 2, 1, set(), range(4)) == {0, 1}


def test_zero_budget_keeps_only_the_warmup():
    assert R.gpu_aware_greedy(S8, G8, 2, 0, {5}, range(8)) == {5}


# ----------------------------------------------------------------------------- brute force

def _f(S, s):
    return sum((Fraction(float(s[j])) for j in S), Fraction(0))


@pytest.mark.parametrize("N,G", [(6, 2), (6, 3), (8, 2), (8, 4), (9, 3)])
def test_brute_force_eq5_without_warmup(N, G):
    rng = np.random.default_rng(100 + N * 10 + G)
    for trial in range(60):
        # a few distinct values so that ties are common
        s = rng.choice(np.array([0.0, 0.125, 0.25, 0.3, 0.75, 1.5], dtype=np.float32), N)
        groups = list(rng.permutation([g for g in range(G) for _ in range(N // G)]))
        m_g = int(rng.integers(1, N // G + 1))
        S = R.gpu_aware_greedy(s, groups, G, m_g, set(), range(N))
        best = max(_f(T, s) for n in range(N + 1) for T in itertools.combinations(range(N), n)
                   if max(R.group_loads(T, groups, G)) <= m_g)
        assert _f(S, s) == best, (trial, s, groups, m_g, S)
        assert len(S) == m_g * G
        assert max(R.group_loads(S, groups, G)) == math.ceil(len(S) / G)


# ----------------------------------------------------------------------------- closed form

def _rounds_closed_form(s, groups, G, m_g, S0, cand):
    """Group g can take a_g = min(m_g - |S_0 on g|, |candidates on g outside S_0|) experts,
    one per round; after R rounds the loop holds |S_0| + sum_g min(R, a_g) experts; it runs
    the fewest rounds that reach m_g * G, or all max_g a_g rounds if that total is never
    reached.  Group g's picks are its best min(R, a_g) candidates."""
    L0 = R.group_loads(S0, groups, G)
    own = [sorted((j for j in cand if groups[j] == g and j not in S0),
                  key=lambda j: (-float(s[j]), j)) for g in range(G)]
    a = [max(0, min(m_g - L0[g], len(own[g]))) for g in range(G)]
    need = m_g * G - len(S0)
    rounds = 0
    while rounds < max(a, default=0) and sum(min(rounds, x) for x in a) < need:
        rounds += 1
    return set(S0).union(*[own[g][:min(rounds, a[g])] for g in range(G)])


def test_loop_matches_the_closed_form():
    rng = np.random.default_rng(7)
    for trial in range(400):
        N = int(rng.integers(1, 40))
        G = int(rng.integers(1, N + 1))
        groups = [int(v) for v in rng.integers(0, G, N)]
        s = rng.choice(np.array([0, 0.1, 0.2, 0.5, 1.0, 2.0], dtype=np.float32), N)
        cand = [j for j in range(N) if rng.random() < 0.7]
        S0 = set(j for j in cand if rng.random() < 0.2)
        m_g = int(rng.integers(0, 6))
        got = R.gpu_aware_greedy(s, groups, G, m_g, S0, cand)
        assert got == _rounds_closed_form(s, groups, G, m_g, S0, cand), trial


# ----------------------------------------------------------------------------- reductions

def _logits(N, T, seed):
    return W.logits_domains(T, N, 4, seed)


@pytest.mark.parametrize("score", ["topk", "dense"])
def test_one_group_is_the_flat_total_budget(score):
    for seed in range(20):
        h = _logits(32, 8, seed)
        for k, k0, m in [(2, 1, 8), (4, 1, 6), (4, 0, 4), (2, 2, 12)]:
            ep = R.select_ep(h, k, k0, m, [0] * 32, 1, score)
            if ep.n_warmup > m:
                continue
            flat = R.route(h, k, k0, m, R.TOTAL, score)
            assert np.array_equal(ep.sel_mask, flat.sel_mask)
            assert np.array_equal(ep.ids, flat.ids)
            assert np.array_equal(ep.w.view(np.uint32), flat.w.view(np.uint32))


def test_one_expert_per_group_is_vanilla():
    for seed in range(20):
        h = _logits(24, 6, seed)
        for k, k0 in [(2, 0), (3, 1), (4, 4)]:
            ep = R.select_ep(h, k, k0, 1, list(range(24)), 24)
            v = R.vanilla(h, k)
            assert np.array_equal(ep.sel_mask, v.sel_mask)
            assert np.array_equal(ep.ids, v.vanilla_ids)
            assert np.array_equal(ep.w.view(np.uint32), v.vanilla_gates.view(np.uint32))


def test_every_token_keeps_k_experts_when_the_groups_give_fewer():
    # m_g = 0 with no warm-up selects nothing in the loop: the best k candidates are added.
    h = _logits(32, 4, 3)
    ep = R.select_ep(h, 4, 0, 0, R.contiguous_groups(32, 4), 4)
    flat = R.route(h, 4, 0, 4, R.TOTAL)
    assert ep.n_selected == 4
    assert np.array_equal(ep.sel_mask, flat.sel_mask)


# ----------------------------------------------------------------------------- invariants

def test_invariants_random_batches():
    rng = np.random.default_rng(11)
    for trial in range(120):
        N = int(rng.choice([16, 32, 64]))
        G = int(rng.choice([2, 4, 8]))
        k = int(rng.choice([2, 4, 8]))
        k0 = int(rng.integers(0, 3))
        T = int(rng.integers(1, 12))
        m_g = int(rng.integers(0, 6))
        score = "dense" if trial % 5 == 0 else "topk"
        groups = R.contiguous_groups(N, G) if trial % 2 else [int(v) for v in rng.integers(0, G, N)]
        h = W.logits_iid(T, N, int(trial)) if trial % 3 else _logits(N, T, trial)
        r = R.select_ep(h, k, k0, m_g, groups, G, score)
        S = set(r.sel_list)
        S0 = set(int(e) for e in r.vanilla_ids[:, :k0].reshape(-1))
        cand = set(range(N)) if score == "dense" else set(int(e) for e in r.vanilla_ids.reshape(-1))
        assert S0 <= S <= cand
        loads = r.extra["loads"]
        assert sum(loads) == len(S) and loads == R.group_loads(S, groups, G)
        L0 = R.group_loads(S0, groups, G)
        filled = len(S) == min(k, len(cand)) and len(S) > len(S0)
        if not filled:
            assert all(loads[g] <= max(m_g, L0[g]) for g in range(G))
            assert len(S) <= max(len(S0), m_g * G + G - 1)
        for i in range(T):
            assert len(set(r.ids[i].tolist())) == k and set(r.ids[i].tolist()) <= S
            assert abs(float(np.sum(r.w[i], dtype=np.float64)) - 1.0) < 1e-6


def test_rejects_bad_groups():
    h = _logits(16, 4, 0)
    with pytest.raises(ValueError):
        R.select_ep(h, 2, 1, 2, [0] * 15, 2)
    with pytest.raises(ValueError):
        R.select_ep(h, 2, 1, 2, [0] * 15 + [2], 2)
    with pytest.raises(ValueError):
        R.contiguous_groups(16, 3)
