"""Pins of the oracle's selection and routing against what the paper and mathematics fix.

Independent references used here (none of them calls the oracle's own ranking,
greedy or softmax):
* the closed form for the expected number of activated experts (Section 1);
* brute force over expert subsets in exact integer arithmetic: the optimum of
  the per-layer proxy, Eq. (2), that Corollary 3.2 says the greedy reaches;
* numpy's stable argsort for every top-k (vanilla, warm-up, refinement);
* float64 softmax and float64 score sums (Section 2.2, Eq. (2));
* special cases that reduce to plain top-k routing, and the reductions of the
  hierarchical algorithm (Algorithms 3-4) to the flat one (Algorithm 2).
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import workloads as W
from oracle import route as R

F32 = np.float32


# ----------------------------------------------------------------------------- independent helpers

def np_topk(h_row, k, allowed=None):
    """Top-k by logit descending, lowest index first on ties, via numpy's stable argsort."""
    h = np.asarray(h_row, np.float64) + 0.0
    order = np.argsort(-h, kind="stable")
    if allowed is not None:
        allowed = set(int(a) for a in allowed)
        order = [j for j in order if int(j) in allowed]
    return [int(j) for j in order[:k]]


def exact_softmax(h_vals):
    h = np.asarray(h_vals, np.float64)
    e = np.exp(h - h.max())
    return e / e.sum()


def rel_bound(h_vals, n):
    x = float(np.max(np.asarray(h_vals, np.float64)) - np.min(np.asarray(h_vals, np.float64)))
    return 2 * (x * 2.0 ** -24 + 2.0 ** -22) + (n + 1) * 2.0 ** -24


def exact_scores(h, k, score_mode="topk", tokens=None):
    """float64 s_j = sum_i g_ij from float64 gates."""
    T, N = h.shape
    tokens = range(T) if tokens is None else tokens
    s = np.zeros(N)
    for i in tokens:
        if score_mode == "topk":
            top = np_topk(h[i], k)
            s[top] += exact_softmax(h[i, top])
        else:
            s += exact_softmax(h[i])
    return s


def as_int(values):
    """Exact integers v * 2^149 (every fp32 value is an integer multiple of 2^-149)."""
    out = np.empty(len(values), dtype=object)
    for j, v in enumerate(values):
        num, den = float(v).as_integer_ratio()
        out[j] = num * (2 ** 149 // den)
    return out


def brute_best(s_int, forced, pool, size):
    """max over S with forced <= S <= forced | pool, |S| == size, of sum_{j in S} s_int[j]."""
    free = sorted(pool - forced)
    need = size - len(forced)
    base = int(sum(int(s_int[j]) for j in forced))
    if need < 0 or need > len(free):
        return None
    if need == 0:
        return base
    combos = np.array(list(itertools.combinations(free, need)), dtype=np.int64)
    return base + int(s_int[combos].sum(axis=1).max())


def brute_best_subset_of(s_int, pool, size):
    pool = sorted(pool)
    combos = np.array(list(itertools.combinations(pool, size)), dtype=np.int64)
    return int(s_int[combos].sum(axis=1).max())


# ----------------------------------------------------------------------------- Section 1 closed form

def closed_form(N, k, B):
    return N * (1.0 - (1.0 - k / N) ** B)


def closed_form_sd(N, k, B):
    p0 = (1 - k / N) ** B
    p00 = (((N - k) * (N - k - 1)) / (N * (N - 1))) ** B
    var = N * p0 * (1 - p0) + N * (N - 1) * (p00 - p0 * p0)
    return math.sqrt(var)


def test_closed_form_matches_paper_printed_values(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "expected_activated_experts.json")))
    for case in g["cases"]:
        assert round(closed_form(g["N"], g["k"], case["B"])) == case["printed"]


@pytest.mark.parametrize("N,k,T,seeds", [(256, 8, 8, 1500), (256, 8, 32, 600), (16, 2, 8, 2000)])
def test_vanilla_union_matches_closed_form(N, k, T, seeds):
    """iid logits: each token's top-k is a uniform k-subset, so E|U| is the closed form."""
    sizes = []
    for seed in range(seeds):
        h = R.canonical(W.logits_iid(T, N, seed))
        ids = [R.ranked(h[i])[:k] for i in range(T)]
        sizes.append(len(set(e for row in ids for e in row)))
    mean = float(np.mean(sizes))
    mu = closed_form(N, k, T)
    sd = closed_form_sd(N, k, T)
    assert abs(mean - mu) <= 4 * sd / math.sqrt(seeds), (mean, mu, sd)
    assert abs(float(np.std(sizes)) - sd) <= 0.15 * sd


# ----------------------------------------------------------------------------- gating (Section 2.2)

@pytest.mark.parametrize("cfg", ["tiny", "qwen", "ds_t32", "spec"])
def test_vanilla_gating_against_argsort_and_float64(cfg):
    c = W.CONFIGS[cfg]
    for seed in range(4):
        h, _ = W.make_logits(c, seed)
        hc = R.canonical(h)
        ids, gates = R.vanilla_gating(hc, c["k"])
        for i in range(h.shape[0]):
            assert list(ids[i]) == np_topk(h[i], c["k"])
            ref = exact_softmax(h[i, ids[i]])
            rel = np.abs(gates[i].astype(np.float64) - ref) / ref
            assert rel.max() <= rel_bound(h[i, ids[i]], c["k"])


@pytest.mark.parametrize("score_mode", ["topk", "dense"])
def test_scores_against_float64(score_mode):
    for cfg in ("tiny", "qwen", "ds_t32"):
        c = W.CONFIGS[cfg]
        h, _ = W.make_logits(c, 3)
        r = R.route(h, c["k"], c["k0"], c["M"], R.TOTAL, score_mode)
        ref = exact_scores(h, c["k"], score_mode)
        # each gate is within ~2^-20 relative, then T sequential fp32 adds
        tol = (h.shape[0] + 8) * 2.0 ** -20 * np.maximum(ref, 1e-30) + 1e-30
        assert np.all(np.abs(r.scores.astype(np.float64) - ref) <= tol)
        if score_mode == "topk":
            assert np.all((r.scores > 0) == (ref > 0))


# ----------------------------------------------------------------------------- Eq. (2) / Cor. 3.2

def _greedy_is_optimal(h, k, k0, M, mode, score_mode="topk"):
    r = R.route(h, k, k0, M, mode, score_mode)
    T, N = h.shape
    S = set(r.sel_list)
    S0 = set(e for i in range(T) for e in np_topk(h[i], k0))
    U = set(e for i in range(T) for e in np_topk(h[i], k))
    cand = U if score_mode == "topk" else set(range(N))
    s_int = as_int(r.scores)
    m = r.budget_eff
    assert len(S) == m
    f = int(sum(int(s_int[j]) for j in S))
    if len(S0) <= m:
        # optimum of Eq. (2) over every subset of E of size m holding the warm-up set
        best = brute_best(s_int, S0, set(range(N)), m)
        assert S0 <= S and S <= cand
    else:
        best = brute_best_subset_of(s_int, S0, m)      # total budget cuts the warm-up set
        assert S <= S0
    assert f == best
    # tie rule: no unselected candidate beats, or ties with a lower index, a greedily added one
    added = S - S0 if len(S0) <= m else S
    pool = (cand - S) if len(S0) <= m else (S0 - S)
    for j in pool:
        for a in added:
            assert (r.scores[j], -j) < (r.scores[a], -a)
    return r


@pytest.mark.parametrize("k0", [0, 1, 2])
def test_greedy_reaches_bruteforce_optimum_tiny(k0):
    c = W.CONFIGS["tiny"]
    for seed in range(60):
        h, _ = W.make_logits(c, seed)
        for mode, M in ((R.TOTAL, 8), (R.TOTAL, 2), (R.TOTAL, 5), (R.EXTRA, 0), (R.EXTRA, 3)):
            _greedy_is_optimal(h, c["k"], k0, M, mode)


def test_greedy_reaches_bruteforce_optimum_dense_tiny():
    c = W.CONFIGS["tiny"]
    for seed in range(40):
        h, _ = W.make_logits(c, seed)
        for mode, M in ((R.TOTAL, 8), (R.EXTRA, 2)):
            _greedy_is_optimal(h, c["k"], 1, M, mode, "dense")


def test_greedy_equals_sorted_top_budget():
    """Corollary 3.2: greedy == sort by score and keep the top m (fixed start set)."""
    rng = np.random.default_rng(5)
    for _ in range(300):
        N = int(rng.integers(4, 40))
        s = (rng.integers(0, 6, N) / 4).astype(F32)          # many exact ties
        cand = sorted(int(j) for j in rng.choice(N, int(rng.integers(1, N + 1)), replace=False))
        start = set(int(j) for j in rng.choice(cand, int(rng.integers(0, len(cand) + 1)), replace=False))
        m = int(rng.integers(len(start), len(cand) + 1))
        S = R.greedy_select(s, start, m, cand)
        rest = sorted(set(cand) - start, key=lambda j: (-float(s[j]), j))
        assert S == start | set(rest[: m - len(start)])


def test_modularity_marginal_gain():
    """Proposition 3.1: f(S + e) - f(S) = s_e, checked in exact integers on oracle scores."""
    c = W.CONFIGS["tiny"]
    h, _ = W.make_logits(c, 11)
    r = R.route(h, c["k"], 1, 8)
    ref = exact_scores(h, c["k"])
    rng = np.random.default_rng(0)
    for _ in range(200):
        S = set(int(j) for j in rng.choice(16, int(rng.integers(0, 15)), replace=False))
        e = int(rng.choice(sorted(set(range(16)) - S)))
        fS = sum(ref[j] for j in S)
        fSe = sum(ref[j] for j in S | {e})
        assert abs((fSe - fS) - ref[e]) <= 1e-12


# ----------------------------------------------------------------------------- Algorithm 2 invariants

def _check_routing(h, r, k, k0, M, mode, score_mode, offsets=None):
    T, N = h.shape
    S = set(r.sel_list)
    U = set(e for i in range(T) for e in np_topk(h[i], k))
    S0 = set(e for i in range(T) for e in np_topk(h[i], k0))
    assert r.n_vanilla_union == len(U)
    assert r.n_warmup == len(S0)
    if mode == R.TOTAL:
        assert len(S) <= M
    assert len(S) == r.budget_eff
    if T > 0:
        assert len(S) >= k
    if score_mode == "topk":
        assert S <= U
    if len(S0) <= r.budget_eff:
        assert S0 <= S
    for i in range(T):
        ids = [int(e) for e in r.ids[i]]
        assert len(set(ids)) == k and set(ids) <= S
        assert ids == np_topk(h[i], k, S)                                  # refinement
        ref = exact_softmax(h[i, ids])
        rel = np.abs(r.w[i].astype(np.float64) - ref) / ref
        assert rel.max() <= rel_bound(h[i, ids], k)
        assert np.all(np.diff(r.w[i].astype(np.float64)) <= 0)
        assert abs(float(r.w[i].astype(np.float64).sum()) - 1.0) <= k * 2.0 ** -23


@pytest.mark.parametrize("cfg", ["tiny", "mixtral", "qwen", "ds_t8", "ds_t32", "ds_iid_t32"])
@pytest.mark.parametrize("score_mode", ["topk", "dense"])
def test_route_invariants(cfg, score_mode):
    c = W.CONFIGS[cfg]
    for seed in range(3):
        h, _ = W.make_logits(c, seed)
        for k0 in (0, 1, 2):
            k0 = min(k0, c["k"])
            for M in c["M_sweep"]:
                for mode in (R.TOTAL, R.EXTRA):
                    r = R.route(h, c["k"], k0, M, mode, score_mode)
                    _check_routing(h, r, c["k"], k0, M, mode, score_mode)


def test_budget_sets_are_nested():
    c = W.CONFIGS["ds_t32"]
    h, _ = W.make_logits(c, 2)
    prev = None
    for M in range(8, 120, 3):
        S = set(R.route(h, 8, 1, M).sel_list)
        if prev is not None:
            assert prev <= S
        prev = S


def test_extra_budget_zero_is_warmup_only():
    """Paper setting (m_l = 0, k0): the selected set is exactly the warm-up set (when >= k)."""
    c = W.CONFIGS["qwen"]
    for seed in range(6):
        h, _ = W.make_logits(c, seed)
        for k0 in (1, 2):
            r = R.route(h, c["k"], k0, 0, R.EXTRA)
            S0 = set(e for i in range(h.shape[0]) for e in np_topk(h[i], k0))
            if len(S0) >= c["k"]:
                assert set(r.sel_list) == S0


def test_large_budget_is_vanilla_topk():
    """M >= |U|: XShare reduces to plain top-k routing, gates bit for bit."""
    for cfg in ("tiny", "qwen", "ds_t32", "mixtral"):
        c = W.CONFIGS[cfg]
        h, _ = W.make_logits(c, 1)
        for k0 in (0, 1, c["k"]):
            r = R.route(h, c["k"], k0, c["N"], R.TOTAL)
            assert set(r.sel_list) == set(e for i in range(h.shape[0]) for e in np_topk(h[i], c["k"]))
            assert np.array_equal(r.ids, r.vanilla_ids)
            assert np.array_equal(r.w.view(np.uint32), r.vanilla_gates.view(np.uint32))


def test_single_token_selects_its_topk():
    c = W.CONFIGS["ds_t8"]
    h = W.logits_domains(1, 256, 8, 4)
    for M in (8, 24, 200):
        r = R.route(h, 8, 1, M)
        assert r.sel_list == sorted(np_topk(h[0], 8))


def test_empty_batch():
    h = np.zeros((0, 16), F32)
    for mode in (R.TOTAL, R.EXTRA):
        for sm in ("topk", "dense"):
            r = R.route(h, 2, 1, 8, mode, sm)
            assert r.n_selected == 0 and r.ids.shape == (0, 2)
    r = R.select_hier(h, [0], 2, 1, 2, 8)
    assert r.n_selected == 0


def test_ties_and_signed_zero():
    rng = np.random.default_rng(3)
    for _ in range(40):
        h = (np.round(rng.standard_normal((16, 32)) * 2) / 4).astype(F32)   # quarter steps: many ties
        h[rng.random(h.shape) < 0.2] = F32(-0.0)
        h[rng.random(h.shape) < 0.2] = F32(0.0)
        for mode, M in ((R.TOTAL, 10), (R.EXTRA, 3)):
            r = R.route(h, 4, 1, M, mode)
            _check_routing(h, r, 4, 1, M, mode, "topk")
            hp = h + F32(0.0)                 # all +0.0
            r2 = R.route(hp, 4, 1, M, mode)
            assert np.array_equal(r.sel_mask, r2.sel_mask) and np.array_equal(r.ids, r2.ids)
    h = np.zeros((4, 8), F32)
    r = R.route(h, 2, 1, 4)
    assert r.sel_list == [0, 1] and np.all(r.ids == [0, 1]) and np.all(r.w == F32(0.5))


def test_gate_underflow_keeps_candidates():
    """A top-k expert whose gate underflows to 0 stays a candidate with score 0."""
    h = np.full((2, 8), -300.0, F32)
    h[0, 0], h[0, 5] = 0.0, -150.0          # expert 5: second for token 0, gate underflows
    h[1, 1], h[1, 6] = 0.0, -150.0          # expert 6: second for token 1, gate underflows
    r = R.route(h, 2, 0, 3)
    assert r.scores[5] == 0 and r.scores[6] == 0
    assert r.n_vanilla_union == 4
    assert r.sel_list == [0, 1, 5]           # zero-score tie resolved to the lower index
    assert list(r.ids[0]) == [0, 5] and list(r.ids[1]) == [1, 0]


def test_invalid_parameters_raise():
    h = W.logits_iid(4, 16, 0)
    with pytest.raises(ValueError):
        R.route(h, 17, 0, 20)
    with pytest.raises(ValueError):
        R.route(h, 4, 5, 20)
    with pytest.raises(ValueError):
        R.route(h, 4, 1, 3, R.TOTAL)
    bad = h.copy()
    bad[0, 0] = np.nan
    with pytest.raises(ValueError):
        R.route(bad, 2, 1, 8)
    with pytest.raises(ValueError):
        R.select_hier(h, [0, 2, 2, 4], 2, 1, 2, 8)
    with pytest.raises(ValueError):
        R.select_hier(h, [0, 3], 2, 1, 2, 8)


# ----------------------------------------------------------------------------- Algorithms 3 + 4

@pytest.mark.parametrize("score_mode", ["topk", "dense"])
def test_hier_single_request_equals_flat(score_mode):
    """R = 1: per-request picks are the flat greedy's first m_r picks (same scores)."""
    for cfg in ("tiny", "qwen", "ds_t32"):
        c = W.CONFIGS[cfg]
        h, _ = W.make_logits(c, 4)
        T = h.shape[0]
        for k0 in (0, 1, 2):
            for m_r in (0, 3, 6):
                for m in (0, 5):
                    a = R.select_hier(h, [0, T], c["k"], k0, m_r, m, R.EXTRA, score_mode)
                    b = R.route(h, c["k"], k0, m_r + m, R.EXTRA, score_mode)
                    assert np.array_equal(a.sel_mask, b.sel_mask)
                    assert np.array_equal(a.ids, b.ids)
                    assert np.array_equal(a.w.view(np.uint32), b.w.view(np.uint32))
                for M in c["M_sweep"]:
                    a = R.select_hier(h, [0, T], c["k"], k0, m_r, M, R.TOTAL, score_mode)
                    b = R.route(h, c["k"], k0, M, R.TOTAL, score_mode)
                    assert np.array_equal(a.sel_mask, b.sel_mask)


def test_hier_one_token_requests_is_vanilla():
    """Each request one token, k0 + m_r = k, m = 0: every S_r is the token's top-k, S = U."""
    c = W.CONFIGS["ds_t32"]
    h, _ = W.make_logits(c, 6)
    T = h.shape[0]
    for k0 in (0, 1, 3, 8):
        r = R.select_hier(h, list(range(T + 1)), 8, k0, 8 - k0, 0, R.EXTRA)
        assert np.array_equal(r.ids, r.vanilla_ids)
        assert r.n_selected == r.n_vanilla_union


def test_hier_per_request_picks_against_float64():
    """Algorithm 3: the m_r added experts of request r top its own float64 score sum."""
    c = W.CONFIGS["spec"]
    for seed in range(3):
        h, off = W.make_logits(c, seed)
        hc = R.canonical(h)
        vids, vg = R.vanilla_gating(hc, 8)
        G = R.gate_matrix(hc, vids, vg, "topk")
        for r in range(len(off) - 1):
            toks = range(off[r], off[r + 1])
            S0r, add = R.per_request_select(hc, G, vids, toks, 1, 4, "topk")
            assert S0r == set(e for i in toks for e in np_topk(h[i], 1))
            sr = exact_scores(h, 8, "topk", toks)
            pool = set(e for i in toks for e in np_topk(h[i], 8)) - S0r
            assert add <= pool and len(add) == min(4, len(pool))
            for a in add:
                for j in pool - add:
                    assert sr[a] >= sr[j] * (1 - 1e-5)


def test_hier_spec_invariants_and_bruteforce_final_stage():
    c = W.CONFIGS["spec"]
    for seed in range(4):
        h, off = W.make_logits(c, seed)
        for mode, M in ((R.TOTAL, 64), (R.TOTAL, 40), (R.EXTRA, 0), (R.EXTRA, 8)):
            r = R.select_hier(h, off, 8, 1, 4, M, mode)
            _check_routing(h, r, 8, 1, M, mode, "topk", off)
            S = set(r.sel_list)
            # recompute the union of the per-request sets independently
            S_batch = set()
            for q in range(len(off) - 1):
                toks = range(off[q], off[q + 1])
                S0r = set(e for i in toks for e in np_topk(h[i], 1))
                sr = exact_scores(h, 8, "topk", toks)
                pool = sorted(set(e for i in toks for e in np_topk(h[i], 8)) - S0r,
                              key=lambda j: (-sr[j], j))
                S_batch |= S0r | set(pool[:4])
            assert r.extra["per_request_union"] == len(S_batch)
            if len(S_batch) <= r.budget_eff:
                assert S_batch <= S
                # final GreedySelect: S maximises the batch score among supersets of S_batch
                free = sorted(S - S_batch)
                others = sorted(set(e for i in range(64) for e in np_topk(h[i], 8)) - S)
                if free and others:
                    assert min(r.scores[j] for j in free) >= max(r.scores[j] for j in others)


def test_hier_bruteforce_tiny_groups():
    """Tiny request-grouped batches: the final set is the best superset of the S_r union."""
    for seed in range(40):
        h, off = W.logits_spec(3, 3, 16, 2, seed)
        for m in (0, 1, 3):
            r = R.select_hier(h, off, 2, 1, 1, m, R.EXTRA)
            S = set(r.sel_list)
            T = h.shape[0]
            S_batch = set()
            for q in range(3):
                toks = range(off[q], off[q + 1])
                S0r = set(e for i in toks for e in np_topk(h[i], 1))
                sr = exact_scores(h, 2, "topk", toks)
                pool = sorted(set(e for i in toks for e in np_topk(h[i], 2)) - S0r,
                              key=lambda j: (-sr[j], j))
                S_batch |= S0r | set(pool[:1])
            U = set(e for i in range(T) for e in np_topk(h[i], 2))
            s_int = as_int(r.scores)
            best = brute_best(s_int, S_batch, U, r.budget_eff)
            assert S_batch <= S and int(sum(int(s_int[j]) for j in S)) == best
