"""Pins of the oracle's MoE layer output (Section 2.1, SwiGLU experts)."""
import math

import numpy as np
import torch

import workloads as W
from oracle import ffn as O
from oracle import route as R


def f32_to_bf16_bits(a):
    """Exact bf16 patterns of values that are already bf16-representable."""
    b = np.asarray(a, np.float32).view(np.uint32)
    assert np.all((b & 0xFFFF) == 0)
    return (b >> 16).astype(np.uint16)


def test_bf16_to_f64_exact():
    vals = np.array([0.0, -0.0, 1.0, -2.5, 0.0078125, 3.0e38, -1.1754944e-38], np.float32)
    t = torch.tensor(vals).to(torch.bfloat16)
    bits = t.view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(O.bf16_to_f64(bits), t.to(torch.float64).numpy())


def test_silu():
    assert O.silu(0.0) == 0.0
    assert abs(O.silu(30.0) - 30.0) < 1e-10
    assert abs(O.silu(-30.0)) < 1e-10
    assert abs(O.silu(1.0) - 1.0 / (1.0 + math.exp(-1.0))) < 1e-15


def _perm_expert(rng, d, f):
    """W1/W3 rows pick one input component, W2 rows pick one hidden component."""
    p1, p3 = rng.integers(0, d, f), rng.integers(0, d, f)
    s2 = rng.integers(0, f, d)
    a = rng.choice([0.5, 1.0, -2.0, 0.25], f)
    b = rng.choice([1.0, -0.5, 2.0], f)
    c = rng.choice([1.0, -1.0, 0.75], d)
    W1 = np.zeros((f, d), np.float32)
    W3 = np.zeros((f, d), np.float32)
    W2 = np.zeros((d, f), np.float32)
    W1[np.arange(f), p1] = a
    W3[np.arange(f), p3] = b
    W2[np.arange(d), s2] = c
    closed = lambda x: c * (lambda z: z / (1 + np.exp(-z)))(a[s2] * x[p1[s2]]) * (b[s2] * x[p3[s2]])
    return (f32_to_bf16_bits(W1), f32_to_bf16_bits(W3), f32_to_bf16_bits(W2)), closed


def test_closed_form_permutation_experts():
    """E(x)_n = c_n silu(a_s x_p1(s)) b_s x_p3(s), s = s2(n): catches a transposed operand."""
    rng = np.random.default_rng(0)
    d, f, N, T, k = 12, 20, 5, 6, 2
    experts, closed = zip(*[_perm_expert(rng, d, f) for _ in range(N)])
    x = rng.choice([0.5, -1.0, 1.5, 2.0, -0.25], (T, d)).astype(np.float32)
    xb = f32_to_bf16_bits(x)
    ids = np.array([rng.choice(N, k, replace=False) for _ in range(T)], np.int32)
    w = rng.random((T, k)).astype(np.float32)
    y = O.moe_forward(xb, ids, w, lambda e: experts[e])
    for i in range(T):
        ref = sum(float(w[i, r]) * closed[ids[i, r]](x[i].astype(np.float64)) for r in range(k))
        assert np.allclose(y[i], ref, rtol=1e-13, atol=1e-13)


def test_dense_gate_formulation_on_tiny_workload():
    """y = sum over ALL experts of G[:, e] * E_e(X) with a dense gate matrix (zeros elsewhere)."""
    c = W.CONFIGS["tiny"]
    h, _ = W.make_logits(c, 0)
    r = R.route(h, c["k"], 1, c["M"])
    x = W.bf16_bits(W.activations(c["T"], c["d"], 0))
    ws = [tuple(W.bf16_bits(W.expert_matrix(e, m, c["d"], c["f"], 0)) for m in ("w1", "w3", "w2"))
          for e in range(c["N"])]
    y = O.moe_forward(x, r.ids, r.w, lambda e: ws[e])
    G = np.zeros((c["T"], c["N"]))
    for i in range(c["T"]):
        G[i, r.ids[i]] = r.w[i]
    X = O.bf16_to_f64(x)
    dense = np.zeros_like(y)
    for e in range(c["N"]):
        W1, W3, W2 = (O.bf16_to_f64(m) for m in ws[e])
        a = np.einsum("fd,td->tf", W1, X)
        b = np.einsum("fd,td->tf", W3, X)
        dense += G[:, e:e + 1] * np.einsum("df,tf->td", W2, a / (1 + np.exp(-a)) * b)
    assert np.allclose(y, dense, rtol=1e-12, atol=1e-14)
    # a subset of rows gives the same rows
    sub = O.moe_forward(x, r.ids, r.w, lambda e: ws[e], rows=[5, 1])
    assert np.allclose(sub, y[[5, 1]], rtol=1e-12, atol=1e-15)
    # the routed sum from every expert's output on all tokens (combine) is the dense form too,
    # for all rows, a subset, and one group's experts (the dense form over those experts only)
    outs = {e: O.expert_ffn(X, *ws[e]) for e in range(c["N"])}
    assert np.allclose(O.combine(outs, r.ids, r.w, c["d"]), dense, rtol=1e-12, atol=1e-14)
    assert np.allclose(O.combine(outs, r.ids, r.w, c["d"], rows=[6, 0]), dense[[6, 0]],
                       rtol=1e-12, atol=1e-14)
    mine = {int(e) for e in r.ids[0][:1]}
    part = np.zeros_like(dense)
    for e in mine:
        part += G[:, e:e + 1] * outs[e]
    assert np.allclose(O.combine(outs, r.ids, r.w, c["d"], local=mine), part, rtol=1e-12,
                       atol=1e-14)


def test_group_shares_sum_to_the_layer():
    """Expert parallelism: the shares of the G groups (dense formulation restricted to each
    group's experts) add up to the whole layer output."""
    c = W.CONFIGS["tiny"]
    h, _ = W.make_logits(c, 2)
    G = 4
    groups = R.contiguous_groups(c["N"], G)
    r = R.select_ep(h, c["k"], 1, 2, groups, G)
    x = W.bf16_bits(W.activations(c["T"], c["d"], 2))
    ws = [tuple(W.bf16_bits(W.expert_matrix(e, m, c["d"], c["f"], 2)) for m in ("w1", "w3", "w2"))
          for e in range(c["N"])]
    y = O.moe_forward(x, r.ids, r.w, lambda e: ws[e])
    X = O.bf16_to_f64(x)
    total = np.zeros_like(y)
    for g in range(G):
        mine = {e for e in range(c["N"]) if groups[e] == g}
        share = O.moe_forward(x, r.ids, r.w, lambda e: ws[e], local=mine)
        dense = np.zeros_like(y)
        for e in sorted(mine):
            W1, W3, W2 = (O.bf16_to_f64(m) for m in ws[e])
            gate = np.array([sum(float(r.w[i, q]) for q in range(c["k"]) if r.ids[i, q] == e)
                             for i in range(c["T"])])
            a, b = X @ W1.T, X @ W3.T
            dense += gate[:, None] * ((a / (1 + np.exp(-a)) * b) @ W2.T)
        assert np.allclose(share, dense, rtol=1e-12, atol=1e-14)
        total += share
    assert np.allclose(total, y, rtol=1e-12, atol=1e-14)


def test_router_logits_closed_forms():
    """h = W_g x (Section 2.2): one-hot router rows read out columns of x (a transposed
    operand fails since N != d), and a pure-Python dot product on a tiny case."""
    import torch
    T, d, N = 5, 12, 7
    x = W.activations(T, d, 3)
    eye = torch.zeros((N, d), dtype=torch.bfloat16)
    cols = [3, 0, 11, 5, 5, 8, 1]
    for j, c in enumerate(cols):
        eye[j, c] = 1.0
    h = O.router_logits(W.bf16_bits(x), W.bf16_bits(eye))
    X = O.bf16_to_f64(W.bf16_bits(x))
    assert np.array_equal(h, X[:, cols])
    wg = W.router_weights(N, d, 3)
    Wg = O.bf16_to_f64(W.bf16_bits(wg))
    h = O.router_logits(W.bf16_bits(x), W.bf16_bits(wg))
    for i in range(T):
        for j in range(N):
            ref = 0.0
            for q in range(d):
                ref += float(X[i, q]) * float(Wg[j, q])
            assert abs(h[i, j] - ref) <= 1e-12 * (1 + abs(ref))


def test_shared_expert_is_an_always_routed_expert_with_weight_one():
    """Section 2.1: the shared term equals routing every token to that expert with gate 1."""
    c = W.CONFIGS["tiny"]
    h, _ = W.make_logits(c, 4)
    r = R.route(h, c["k"], 1, c["M"])
    x = W.bf16_bits(W.activations(c["T"], c["d"], 4))
    ws = [tuple(W.bf16_bits(W.expert_matrix(e, m, c["d"], c["f"], 4)) for m in ("w1", "w3", "w2"))
          for e in range(c["N"])]
    sh = [tuple(W.bf16_bits(m[e]) for m in W.shared_weights(2, c["d"], c["f"], 4))
          for e in range(2)]
    base = O.moe_forward(x, r.ids, r.w, lambda e: ws[e])
    both = O.moe_forward(x, r.ids, r.w, lambda e: ws[e], shared=sh)
    ones = np.ones((c["T"], 1))
    alone = sum(O.moe_forward(x, np.zeros((c["T"], 1), np.int32), ones, lambda e, t=t: t)
                for t in sh)
    assert np.allclose(both - base, alone, rtol=1e-12, atol=1e-14)
    # one SwiGLU of width 2f equals two of width f holding its halves (the hidden units are
    # independent), which is how a wider shared expert maps onto experts of width f
    wide = tuple(np.concatenate(p, axis=1 if i == 2 else 0) for i, p in enumerate(zip(*sh)))
    X = O.bf16_to_f64(x)
    assert np.allclose(O.expert_ffn(X, *wide), O.expert_ffn(X, *sh[0]) + O.expert_ffn(X, *sh[1]),
                       rtol=1e-12, atol=1e-14)


def test_domain_activations_carry_the_routing_structure():
    """Tokens of one domain share most of their hidden state, so the router's logits of two
    such tokens are strongly correlated; iid activations give uncorrelated logits."""
    T, d, N, Q = 48, 512, 128, 6
    x = W.bf16_bits(W.activations_domains(T, d, Q, 1))
    wg = W.bf16_bits(W.router_weights(N, d, 1))
    h = O.router_logits(x, wg)
    dom = W._rng(W._S_X, 2, T, d, Q, 1).integers(0, Q, T)
    same = [np.corrcoef(h[i], h[j])[0, 1] for i in range(T) for j in range(i) if dom[i] == dom[j]]
    diff = [np.corrcoef(h[i], h[j])[0, 1] for i in range(T) for j in range(i) if dom[i] != dom[j]]
    assert np.mean(same) > 0.6 and abs(np.mean(diff)) < 0.2
    assert 1.2 < h.std() < 2.0
