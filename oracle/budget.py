"""Global expert budget over the MoE layers of a forward pass (oracle side).

TEST INFRASTRUCTURE ONLY: only the tests may import this module.

Section 3.2: the L MoE layers share one budget K of activated experts,
sum_l |S_l| <= K, and the practical algorithm splits it uniformly, m_l = K / L.
The paper does not say where the remainder of K / L goes.  Reading: every layer
gets floor(K / L) and the first K mod L layers one more, so the budgets sum to
exactly K and differ by at most one.

The running totals a pass keeps (layers, sum |S_l|, sum of the experts whose
weights are streamed, sum |U_l|, calls that selected nothing, largest |S_l|)
are plain sums over the per-layer selections.
"""
from __future__ import annotations


def uniform_budgets(K: int, L: int) -> list[int]:
    """m_l for l = 0..L-1: floor(K / L), plus one for the first K mod L layers."""
    if L < 1 or K < 0:
        raise ValueError("need L >= 1 and K >= 0")
    q, r = divmod(K, L)
    return [q + (1 if l < r else 0) for l in range(L)]


LEDGER_FIELDS = ("layers", "selected", "active", "vanilla_union", "invalid", "max_selected")


def ledger(routings) -> dict:
    """Totals over the per-layer selections (oracle Routing objects, or None for a call
    whose request offsets were invalid and that therefore selected nothing)."""
    out = dict.fromkeys(LEDGER_FIELDS, 0)
    for r in routings:
        out["layers"] += 1
        if r is None:
            out["invalid"] += 1
            continue
        out["selected"] += r.n_selected
        out["active"] += r.n_active
        out["vanilla_union"] += r.n_vanilla_union
        out["max_selected"] = max(out["max_selected"], r.n_selected)
    return out
