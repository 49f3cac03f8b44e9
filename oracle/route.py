"""Expert selection and routing (oracle side).

Follows, step by step:
* Section 2.2 -- top-k gating: the k largest logits of a token, gates given by a
  softmax renormalised over those k;
* Section 3.2, Eq. (2) -- per-layer proxy: the score of expert j is the sum over
  the batch of its gates, s_j = sum_i g_ij;
* Section 3.4, Algorithm 1 -- greedy selection, here with the fixed budget the
  paper says it uses in practice instead of the threshold;
* Section 3.4, Algorithm 2 -- warm-up S_0 (top-k0 of every token), greedy
  selection, refinement (each token routed to its top-k inside the set);
* Section 4.1, Eqs. (3)-(4), Algorithms 3 and 4 -- per-request warm-up plus the
  m_r best experts of each request by its own score, union over requests, then
  the batch-level greedy and the same refinement;
* Section 5, Eq. (5), Algorithms 5 and 6 -- experts partitioned over G GPU groups;
  after the warm-up, rounds in which every group in turn adds its best remaining
  expert, then the same refinement.

Readings of what the paper leaves open (each one is listed with its reason in
the design notes of the repository):
* gates for the scores are the top-k-sparse renormalised gates of Section 2.2
  ("topk" mode, default); "dense" mode uses the softmax over all N experts;
* refinement ranks a token's experts by its logits (monotone in the softmax);
* ranking key everywhere is (value descending, expert index ascending); logits
  are canonicalised with h + 0.0 so that -0.0 and +0.0 compare equal;
* budget "total": |S| <= M (requires M >= k); budget "extra": M experts are
  added beyond the warm-up set (beyond the union of the per-request sets in the
  hierarchical case), which is how the paper's tables use m_l; budget
  "threshold": Algorithm 1's own stopping rule, add experts while
  f(S) < tau * f(E), in fp32: f(E) sums every s_j in index order, f(S) starts
  with the starting set in ranking order (priority, score descending, index
  ascending) and adds each pick; tau * f(E) is one fp32 product; the starting
  set is never cut and the loop also stops when no candidate is left;
* candidates: in "topk" mode only experts some token (some token of the
  request, for per-request picks) has in its top-k; in "dense" mode all experts
  (none when the batch is empty);
* the effective set size is clamped up to k so that every token keeps exactly k
  experts; if the starting set is larger than a total budget it is cut by
  priority (warm-up first, then per-request picks), score descending, index
  ascending;
* batch scores are always the sum over all tokens in ascending token order, so
  the hierarchical scores of Eq. (4) equal the flat ones bit for bit;
* GPU groups (Algorithm 5): the per-group budget m_g is also a cap, as in the
  constraint of Eq. (5): a group whose load (warm-up experts included) has reached
  m_g adds nothing more; a group with no candidate left is skipped (the argmax of
  Algorithm 5 is over an empty set there); the loop condition |S| < m_g * G is
  tested before each round, so a started round runs over all groups, and a round
  that adds nothing ends the loop; the warm-up set is never cut; if fewer than k
  experts result, the best remaining candidates are added regardless of group.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from .numerics import F32, seq_sum, softmax_dense, softmax_ranked

TOTAL = "total"
EXTRA = "extra"
THRESHOLD = "threshold"
TOPK = "topk"
DENSE = "dense"


@dataclass
class Routing:
    sel_mask: np.ndarray          # uint8 [N], 1 = expert in S
    ids: np.ndarray               # int32 [T,k], rank order
    w: np.ndarray                 # fp32 [T,k]
    scores: np.ndarray            # fp32 [N], batch scores s_j
    vanilla_ids: np.ndarray       # int32 [T,k], plain top-k
    vanilla_gates: np.ndarray     # fp32 [T,k]
    n_vanilla_union: int
    n_warmup: int
    budget_eff: int
    extra: dict = field(default_factory=dict)

    @property
    def sel_list(self) -> list[int]:
        return [int(j) for j in np.flatnonzero(self.sel_mask)]

    @property
    def n_selected(self) -> int:
        return int(self.sel_mask.sum())

    @property
    def n_active(self) -> int:
        return len(set(int(e) for e in self.ids.reshape(-1)))


# ----------------------------------------------------------------------------- ranking

def canonical(h) -> np.ndarray:
    """fp32 logits with -0.0 mapped to +0.0; rejects NaN and infinities."""
    h = np.asarray(h, dtype=F32)
    if not np.all(np.isfinite(h)):
        raise ValueError("logits must be finite")
    return (h + F32(0.0)).astype(F32)


def ranked(h_row, allowed=None) -> list[int]:
    """Experts in rank order (logit descending, index ascending), optionally restricted."""
    js = range(len(h_row)) if allowed is None else allowed
    return sorted((int(j) for j in js), key=lambda j: (-float(h_row[j]), j))


# ----------------------------------------------------------------------------- gates and scores

def vanilla_gating(h, k: int):
    """Section 2.2: per token the top-k experts (rank order) and their renormalised gates."""
    T = h.shape[0]
    ids = np.zeros((T, k), dtype=np.int32)
    gates = np.zeros((T, k), dtype=F32)
    for i in range(T):
        top = ranked(h[i])[:k]
        ids[i] = top
        gates[i] = softmax_ranked(h[i, top])
    return ids, gates


def gate_matrix(h, ids, gates, score_mode: str) -> np.ndarray:
    """G[T,N] fp32: the gates g_ij that enter the scores (zeros outside the top-k in topk mode)."""
    T, N = h.shape
    G = np.zeros((T, N), dtype=F32)
    for i in range(T):
        if score_mode == TOPK:
            G[i, ids[i]] = gates[i]
        elif score_mode == DENSE:
            G[i] = softmax_dense(h[i])
        else:
            raise ValueError(score_mode)
    return G


def scores_over(G, tokens) -> np.ndarray:
    """s_j = sum over the given tokens of g_ij, added one token at a time in the given order."""
    s = np.zeros(G.shape[1], dtype=F32)
    for i in tokens:
        s = (s + G[i]).astype(F32)
    return s


# ----------------------------------------------------------------------------- greedy

def greedy_order(scores, start, candidates, priority=None) -> list[int]:
    """The order in which Algorithm 1's greedy takes experts under the objective of Eq. (2).

    f(S) = sum of s_j over S is modular (Proposition 3.1): adding e to any set raises f by
    exactly s_e.  So the argmax of every greedy step is the best remaining candidate by score
    whatever was taken before, and the greedy takes the candidates in one fixed order, score
    descending, lowest index first on equal scores (Corollary 3.2).  The starting set comes
    first, in (priority ascending, score descending, index ascending) order: the order in
    which a budget smaller than the starting set cuts it.
    """
    pri = priority or {}
    start = set(int(j) for j in start)
    head = sorted(start, key=lambda j: (pri.get(j, 0), -float(scores[j]), j))
    rest = sorted(set(int(e) for e in candidates) - start, key=lambda e: (-float(scores[e]), e))
    return head + rest


def greedy_select(scores, start, budget: int, candidates, priority=None) -> set[int]:
    """Algorithm 1 with a fixed budget (Section 3.4): the first ``budget`` experts of the
    greedy order, or all of them if there are fewer; a starting set larger than the budget
    is cut by the order's key."""
    return set(greedy_order(scores, start, candidates, priority)[:max(int(budget), 0)])


def greedy_threshold(scores, start, tau: float, candidates, priority=None) -> set[int]:
    """Algorithm 1's own stopping rule: the shortest prefix of the greedy order that holds
    the whole starting set and reaches f(S) >= tau * f(E), f(S) = sum of the scores in S
    (Eq. (2)); every candidate if no prefix reaches it.  All in fp32: f(E) adds every s_j in
    index order, f(S) adds the prefix's scores in order, tau * f(E) is one product."""
    scores = np.asarray(scores, dtype=F32)
    f_E = F32(0.0)
    for j in range(len(scores)):                       # f(E), index order
        f_E = F32(f_E + scores[j])
    target = F32(F32(tau) * f_E)
    order = greedy_order(scores, start, candidates, priority)
    n_start = len(set(int(j) for j in start))
    f_S = F32(0.0)
    for m, j in enumerate(order):
        if m >= n_start and not f_S < target:          # order[:m] reaches the target
            return set(order[:m])
        f_S = F32(f_S + scores[j])
    return set(order)


def _effective_budget(base: int, n_cand: int, k: int) -> int:
    return max(min(base, n_cand), min(k, n_cand))


def _check(h, k, k0, M, budget_mode, score_mode, tau=None):
    T, N = h.shape
    if not 1 <= k <= N:
        raise ValueError("need 1 <= k <= N")
    if not 0 <= k0 <= k:
        raise ValueError("need 0 <= k0 <= k")
    if M < 0:
        raise ValueError("need M >= 0")
    if budget_mode == TOTAL and M < k:
        raise ValueError("a total budget must be >= k")
    if budget_mode not in (TOTAL, EXTRA, THRESHOLD) or score_mode not in (TOPK, DENSE):
        raise ValueError("unknown mode")
    if budget_mode == THRESHOLD and (tau is None or not np.isfinite(tau) or tau < 0):
        raise ValueError("the threshold mode needs a finite tau >= 0")


# ----------------------------------------------------------------------------- refinement

def refine(h, S, k: int):
    """Route every token to its top-k experts inside S, gates renormalised over those k."""
    T = h.shape[0]
    allowed = sorted(S)
    ids = np.zeros((T, k), dtype=np.int32)
    w = np.zeros((T, k), dtype=F32)
    for i in range(T):
        top = ranked(h[i], allowed)[:k]
        ids[i] = top
        w[i] = softmax_ranked(h[i, top])
    return ids, w


# ----------------------------------------------------------------------------- Algorithm 2

def route(h, k: int, k0: int, M: int, budget_mode: str = TOTAL,
          score_mode: str = TOPK, tau: float | None = None) -> Routing:
    """Batch-aware expert selection for one layer (Algorithm 2; Algorithm 1's threshold
    rule instead of the budget with budget_mode "threshold")."""
    h = canonical(h)
    _check(h, k, k0, M, budget_mode, score_mode, tau)
    T, N = h.shape
    vids, vg = vanilla_gating(h, k)
    G = gate_matrix(h, vids, vg, score_mode)
    s = scores_over(G, range(T))

    union = set(int(e) for e in vids.reshape(-1))
    S0 = set(int(e) for e in vids[:, :k0].reshape(-1))            # warm-up
    if T == 0:
        cand = set()
    else:
        cand = union if score_mode == TOPK else set(range(N))
    if budget_mode == THRESHOLD:
        S = greedy_threshold(s, S0, tau, sorted(cand))
        m_eff = max(len(S), min(k, len(cand)))
        S = greedy_select(s, S, m_eff, sorted(cand))               # every token keeps k
    else:
        base = M if budget_mode == TOTAL else len(S0) + M
        m_eff = _effective_budget(base, len(cand), k)
        S = greedy_select(s, S0, m_eff, sorted(cand))
    ids, w = refine(h, S, k)
    mask = np.zeros(N, dtype=np.uint8)
    mask[sorted(S)] = 1
    return Routing(mask, ids, w, s, vids, vg, len(union), len(S0), m_eff)


# ----------------------------------------------------------------------------- Algorithms 3 + 4

def check_offsets(offsets, T: int) -> list[int]:
    o = [int(v) for v in offsets]
    if len(o) < 1 or o[0] != 0 or o[-1] != T or any(b <= a for a, b in zip(o, o[1:])):
        raise ValueError("request offsets must satisfy 0 = o_0 < o_1 < ... < o_R = T")
    return o


def per_request_select(h, G, vids, tokens, k0: int, m_r: int, score_mode: str):
    """Algorithm 3 for one request: (S_0(r), added experts) with the request's own scores."""
    N = h.shape[1]
    S0_r = set(int(e) for i in tokens for e in vids[i, :k0])
    s_r = scores_over(G, tokens)
    if score_mode == TOPK:
        pool = set(int(e) for i in tokens for e in vids[i])
    else:
        pool = set(range(N))
    rest = sorted(pool - S0_r, key=lambda j: (-float(s_r[j]), j))
    return S0_r, set(rest[:m_r])


def select_hier(h, offsets, k: int, k0: int, m_r: int, M: int,
                budget_mode: str = TOTAL, score_mode: str = TOPK,
                tau: float | None = None) -> Routing:
    """Speculative-decoding-aware selection (Algorithm 4 calling Algorithm 3 per request)."""
    h = canonical(h)
    _check(h, k, k0, M, budget_mode, score_mode, tau)
    if m_r < 0:
        raise ValueError("need m_r >= 0")
    T, N = h.shape
    o = check_offsets(offsets, T)
    vids, vg = vanilla_gating(h, k)
    G = gate_matrix(h, vids, vg, score_mode)
    s = scores_over(G, range(T))                                   # Eq. (4) == flat score

    S0 = set()
    added = set()
    for r in range(len(o) - 1):
        S0_r, add_r = per_request_select(h, G, vids, range(o[r], o[r + 1]), k0, m_r, score_mode)
        S0 |= S0_r
        added |= add_r
    S_batch = S0 | added                                           # union of the S_r
    union = set(int(e) for e in vids.reshape(-1))
    if T == 0:
        cand = set()
    else:
        cand = union if score_mode == TOPK else set(range(N))
    priority = {j: (0 if j in S0 else 1) for j in S_batch}
    if budget_mode == THRESHOLD:
        S = greedy_threshold(s, S_batch, tau, sorted(cand), priority)
        m_eff = max(len(S), min(k, len(cand)))
        S = greedy_select(s, S, m_eff, sorted(cand), priority)
    else:
        base = M if budget_mode == TOTAL else len(S_batch) + M
        m_eff = _effective_budget(base, len(cand), k)
        S = greedy_select(s, S_batch, m_eff, sorted(cand), priority)
    ids, w = refine(h, S, k)
    mask = np.zeros(N, dtype=np.uint8)
    mask[sorted(S)] = 1
    return Routing(mask, ids, w, s, vids, vg, len(union), len(S0), m_eff,
                   extra=dict(per_request_union=len(S_batch), tier1=len(added - S0)))


# ----------------------------------------------------------------------------- Algorithms 5 + 6

def contiguous_groups(N: int, G: int) -> list[int]:
    """Expert j lives on GPU group j // (N / G) (equal contiguous blocks)."""
    if G < 1 or N % G:
        raise ValueError("contiguous groups need G >= 1 dividing N")
    return [j // (N // G) for j in range(N)]


def group_loads(S, groups, G: int) -> list[int]:
    """Load_g(S) = |S intersected with E_g| for every group (Section 5.1)."""
    load = [0] * G
    for j in S:
        load[groups[j]] += 1
    return load


def gpu_aware_greedy(scores, groups, G: int, m_g: int, S0, candidates) -> set[int]:
    """Algorithm 5: starting from S_0, rounds over the groups; each group adds the
    candidate of largest marginal gain (= its score, Proposition 3.1) among its own
    experts not yet in S, while |S| < m_g * G at the start of a round."""
    S = set(int(j) for j in S0)
    load = group_loads(S, groups, G)
    while len(S) < m_g * G:
        added = 0
        for g in range(G):
            if load[g] >= m_g:                       # Eq. (5): MaxLoad(S) <= m_g
                continue
            rest = [int(e) for e in candidates if groups[int(e)] == g and int(e) not in S]
            if not rest:                             # no candidate left on this group
                continue
            e_star = max(rest, key=lambda e: (float(scores[e]), -e))
            S.add(e_star)
            load[g] += 1
            added += 1
        if added == 0:
            break
    return S


def check_groups(groups, N: int, G: int) -> list[int]:
    gr = [int(v) for v in groups]
    if G < 1 or len(gr) != N or any(not 0 <= v < G for v in gr):
        raise ValueError("every expert needs a group in [0, G)")
    return gr


def select_ep(h, k: int, k0: int, m_g: int, groups, G: int,
              score_mode: str = TOPK) -> Routing:
    """Expert-parallelism-aware selection (Algorithm 6 calling Algorithm 5)."""
    h = canonical(h)
    _check(h, k, k0, k, TOTAL, score_mode)
    if m_g < 0:
        raise ValueError("need m_g >= 0")
    T, N = h.shape
    gr = check_groups(groups, N, G)
    vids, vg = vanilla_gating(h, k)
    G_mat = gate_matrix(h, vids, vg, score_mode)
    s = scores_over(G_mat, range(T))

    union = set(int(e) for e in vids.reshape(-1))
    S0 = set(int(e) for e in vids[:, :k0].reshape(-1))            # warm-up
    if T == 0:
        cand = set()
    else:
        cand = union if score_mode == TOPK else set(range(N))
    S = gpu_aware_greedy(s, gr, G, m_g, S0, sorted(cand))
    if len(S) < min(k, len(cand)):                                 # every token keeps k
        S = greedy_select(s, S, min(k, len(cand)), sorted(cand))
    ids, w = refine(h, S, k)
    mask = np.zeros(N, dtype=np.uint8)
    mask[sorted(S)] = 1
    loads = group_loads(S, gr, G)
    vloads = group_loads(union, gr, G)
    return Routing(mask, ids, w, s, vids, vg, len(union), len(S0), min(m_g * G, N),
                   extra=dict(loads=loads, max_load=max(loads) if loads else 0,
                              vanilla_loads=vloads, vanilla_max_load=max(vloads)))


def vanilla(h, k: int) -> Routing:
    """Plain top-k routing expressed as Algorithm 2 with every candidate kept."""
    N = np.asarray(h).shape[1]
    return route(h, k, 0, N, EXTRA, TOPK)
