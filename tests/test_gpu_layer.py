"""The whole layer of Section 2.1 on the GPU: router logits h = W_g x, selection on those
logits, the routed experts and the always-on shared experts.

* router logits within the fp32 accumulation bound of the exact dot product,
  |h - h_exact| <= d * 2^-24 * sum_q |x_q W_q|, and bit-identical across calls;
* the selection made inside xshare_moe_layer equals the oracle's selection on the logits
  the layer reports (bit for bit), and those logits equal xshare_router_logits';
* y within 2e-2 * RMS of the float64 oracle (routed terms plus shared terms).
"""
import numpy as np
import pytest
import torch

import workloads as W
from helpers import (DEV, OracleOutputs, assert_ffn_close, assert_route_equal, bf16_weights_of,
                     expert_fetcher, say)
from oracle import ffn as OF
from oracle import route as OR

pytestmark = pytest.mark.gpu



def _router_inputs(T, d, N, seed, Q=4):
    x = W.activations_domains(T, d, Q, seed, DEV)
    wg = W.router_weights(N, d, seed, DEV)
    return x, wg


def test_router_logits_within_the_accumulation_bound():
    from paper_2602_07265_amd import xshare as X
    for T, d, N in [(8, 64, 16), (1, 256, 8), (37, 512, 200), (64, 2048, 128), (32, 7168, 256),
                    (100, 1024, 64), (300, 256, 40)]:
        say(f"router case T={T} d={d} N={N}")
        x, wg = _router_inputs(T, d, N, 0)
        h = X.router_logits(x, wg)
        h2 = X.router_logits(x, wg)
        torch.cuda.synchronize()
        assert torch.equal(h.view(torch.int32), h2.view(torch.int32)), "not deterministic"
        xb, wb = W.bf16_bits(x), W.bf16_bits(wg)
        ref = OF.router_logits(xb, wb)
        mag = np.abs(OF.bf16_to_f64(xb)) @ np.abs(OF.bf16_to_f64(wb)).T
        err = np.abs(h.cpu().numpy().astype(np.float64) - ref)
        bound = d * 2.0 ** -24 * mag * (1 + 1e-6) + 1e-30
        assert np.all(err <= bound), f"max err/bound {np.max(err / bound):.3f}"
        say(f"  max |err| / (d u sum|xw|) = {np.max(err / bound):.3e}")


def _layer(T, N, k, d, f, n_shared, seed, k0=1, M=None, mode="total", tau=0.0, offsets=None,
           m_r=0, rows=None, label=""):
    from paper_2602_07265_amd import xshare as X
    M = M if M is not None else max(k, N // 4)
    x, wg = _router_inputs(T, d, N, seed)
    w1, w3, w2 = W.expert_weights(N, d, f, seed, DEV)
    sh = W.shared_weights(n_shared, d, f, seed, DEV) if n_shared else None
    say(f"layer case {label} T={T} N={N} k={k} d={d} f={f} shared={n_shared} M={M} {mode}"
        f"{'' if offsets is None else ' hier'}")
    res = X.moe_layer(x, wg, w1, w3, w2, k, k0, M, mode, shared=sh, tau=tau,
                      req_offsets=None if offsets is None else list(offsets),
                      per_request_budget=m_r)
    torch.cuda.synchronize()
    logits = res["logits"].cpu().numpy()
    alone = X.router_logits(x, wg).cpu().numpy()
    assert np.array_equal(logits.view(np.uint32), alone.view(np.uint32)), \
        f"{label}: the layer's logits differ from xshare_router_logits"
    got = {key: v.cpu().numpy() for key, v in res.items() if key not in ("y", "logits")}
    if offsets is None:
        ref = OR.route(logits, k, k0, M, mode, tau=tau if mode == "threshold" else None)
    else:
        ref = OR.select_hier(logits, offsets, k, k0, m_r, M, mode)
    assert_route_equal(got, ref, label)
    rows = list(range(T)) if rows is None else list(rows)
    shared_bits = [] if sh is None else [tuple(W.bf16_bits(m[s]) for m in sh)
                                         for s in range(n_shared)]
    y_ref = OracleOutputs(x, bf16_weights_of(w1, w3, w2), shared_bits).y(ref.ids, ref.w, rows)
    y_gpu = OF.bf16_to_f64(W.bf16_bits(res["y"]))[rows]
    assert np.all(np.isfinite(y_gpu))
    assert_ffn_close(y_gpu, y_ref, label, f" |S|={got['stats'][0]}")
    return res


def test_layer_small_shapes():
    for T, N, k, d, f, ns in [(8, 16, 2, 64, 128, 1), (24, 32, 4, 128, 256, 2),
                              (37, 40, 4, 96, 160, 0), (1, 16, 2, 64, 32, 1),
                              (70, 24, 3, 128, 96, 3)]:
        _layer(T, N, k, d, f, ns, 0, label=f"T{T} N{N}")


def test_layer_modes():
    _layer(24, 32, 4, 128, 256, 1, 1, k0=0, M=6, mode="extra", label="extra")
    _layer(24, 32, 4, 128, 256, 1, 1, mode="threshold", tau=0.8, label="threshold")
    _layer(24, 32, 4, 128, 256, 1, 1, M=32, label="every candidate")
    off = [0, 4, 8, 12, 16, 20, 24]
    _layer(24, 32, 4, 128, 256, 1, 1, M=12, offsets=off, m_r=2, label="hier")


def test_layer_split_reductions_with_shared_experts():
    # few wide experts: gate/up splits d and down splits f; the shared expert's rows take
    # the same split path
    _layer(16, 8, 2, 1024, 256, 1, 2, M=2, label="split gate/up")
    _layer(16, 8, 2, 128, 1024, 2, 2, M=2, label="split down")


def test_moe_forward_with_shared_experts_from_given_logits():
    from paper_2602_07265_amd import xshare as X
    c = W.CONFIGS["qwen"]
    T, N, k, d, f = c["T"], c["N"], c["k"], c["d"], c["f"]
    h, _ = W.make_logits(c, 3)
    x = W.activations(T, d, 3, DEV)
    w1, w3, w2 = W.expert_weights(N, d, f, 3, DEV)
    sh = W.shared_weights(4, d, f, 3, DEV)
    say("shared case qwen T=64 with 4 shared experts (a 4f-wide shared expert)")
    res = X.moe_forward(x, torch.from_numpy(h).to(DEV), w1, w3, w2, k, 1, 32, shared=sh)
    torch.cuda.synchronize()
    ref = OR.route(h, k, 1, 32)
    got = {key: v.cpu().numpy() for key, v in res.items() if key != "y"}
    assert_route_equal(got, ref, "qwen shared")
    y_ref = OF.moe_forward(W.bf16_bits(x), ref.ids, ref.w, expert_fetcher(w1, w3, w2),
                           shared=[tuple(W.bf16_bits(m[s]) for m in sh) for s in range(4)])
    assert_ffn_close(OF.bf16_to_f64(W.bf16_bits(res["y"])), y_ref, "qwen shared")


def test_layer_deepseek():
    # DeepSeek-R1 shape with its one shared expert, T = 32, total budget 48, all rows: 49
    # expert slots, so the gate/up launch's last slot runs apart, split along d
    res = _layer(32, 256, 8, 7168, 2048, 1, 0, M=48, label="deepseek")
    assert int(res["stats"][1]) <= 48
    torch.cuda.empty_cache()


def test_full_layer_generators_identical_on_gpu_and_cpu():
    for fn, args in [(W.activations_domains, (9, 96, 3, 5)), (W.router_weights, (40, 96, 5))]:
        a = fn(*args, device=DEV).cpu()
        b = fn(*args, device="cpu")
        assert torch.equal(a.view(torch.int16), b.view(torch.int16)), fn.__name__
    ga = W.shared_weights(2, 64, 32, 7, DEV)
    gb = W.shared_weights(2, 64, 32, 7, "cpu")
    for a, b in zip(ga, gb):
        assert torch.equal(a.cpu().view(torch.int16), b.view(torch.int16))
