"""Global budget over the layers of a pass (Section 3.2) on the GPU: the per-layer budgets
m_l = K / L from xshare_layer_budgets, each layer's selection bit-exact against the oracle,
and the device ledger's running totals equal to the oracle's sums over the same layers."""
import numpy as np
import pytest
import torch

import workloads as W
from helpers import DEV, assert_ffn_close, assert_route_equal, expert_fetcher, say
from oracle import budget as B
from oracle import ffn as OF
from oracle import route as OR

pytestmark = pytest.mark.gpu


def _ledger(t):
    from paper_2602_07265_amd import xshare as X
    return {k: v for k, v in X.ledger_dict(t).items()}


def test_pass_of_deepseek_layers_selection_only():
    from paper_2602_07265_amd import xshare as X
    T, N, k, L, K = 32, 256, 8, 6, 250
    m = X.layer_budgets(K, L)
    assert m == B.uniform_budgets(K, L)
    led = X.new_ledger(DEV)
    refs = []
    for l in range(L):
        say(f"budget case deepseek selection layer {l} m_l={m[l]}")
        h = W.logits_domains(T, N, 8, 100 + l)
        res = X.route(torch.from_numpy(h).to(DEV), k, 1, m[l], ledger=led)
        torch.cuda.synchronize()
        ref = OR.route(h, k, 1, m[l])
        assert_route_equal({key: v.cpu().numpy() for key, v in res.items()}, ref, f"layer {l}")
        refs.append(ref)
    got = _ledger(led)
    assert got == B.ledger(refs), (got, B.ledger(refs))
    assert got["selected"] <= K


def test_budget_below_k_per_layer_is_reported():
    # K / L < k: every layer still selects at least k experts, and the ledger shows the
    # pass exceeding K
    from paper_2602_07265_amd import xshare as X
    T, N, k, L, K = 16, 64, 4, 5, 12
    m = X.layer_budgets(K, L)
    led = X.new_ledger(DEV)
    refs = []
    for l in range(L):
        h = W.logits_domains(T, N, 4, 200 + l)
        say(f"budget case small layer {l} m_l={m[l]}")
        X.route(torch.from_numpy(h).to(DEV), k, 1, max(m[l], k), ledger=led)
        refs.append(OR.route(h, k, 1, max(m[l], k)))
    torch.cuda.synchronize()
    got = _ledger(led)
    assert got == B.ledger(refs)
    assert got["selected"] >= k * L > K


def test_ledger_through_the_layer_entry_points():
    from paper_2602_07265_amd import xshare as X
    T, N, k, d, f = 12, 32, 4, 128, 256
    m = X.layer_budgets(30, 3)
    led = X.new_ledger(DEV)
    refs = []
    for l in range(3):
        say(f"budget case moe_forward layer {l} m_l={m[l]}")
        h = W.logits_domains(T, N, 3, 300 + l)
        x = W.activations(T, d, 300 + l, DEV)
        w1, w3, w2 = W.expert_weights(N, d, f, 300 + l, DEV)
        res = X.moe_forward(x, torch.from_numpy(h).to(DEV), w1, w3, w2, k, 1, m[l], ledger=led)
        torch.cuda.synchronize()
        ref = OR.route(h, k, 1, m[l])
        assert_route_equal({key: v.cpu().numpy() for key, v in res.items() if key != "y"}, ref,
                           f"moe layer {l}")
        y_ref = OF.moe_forward(W.bf16_bits(x), ref.ids, ref.w, expert_fetcher(w1, w3, w2))
        assert_ffn_close(OF.bf16_to_f64(W.bf16_bits(res["y"])), y_ref, f"moe layer {l}")
        refs.append(ref)
    # an expert-parallel selection and a hierarchical call with invalid device-side offsets
    # (it selects nothing) add to the same ledger
    h = W.logits_domains(T, N, 3, 400)
    say("budget case expert-parallel selection and invalid offsets")
    X.select_ep(torch.from_numpy(h).to(DEV), X.GroupMap(4, None, device=DEV), k, 1, 3,
                ledger=led)
    refs.append(OR.select_ep(h, k, 1, 3, OR.contiguous_groups(N, 4), 4))
    bad = torch.tensor([0, 5, 5, T], dtype=torch.int32, device=DEV)   # empty request
    X.select_hier(torch.from_numpy(h).to(DEV), bad, k, 1, 1, 8, ledger=led)
    refs.append(None)
    torch.cuda.synchronize()
    assert _ledger(led) == B.ledger(refs)
