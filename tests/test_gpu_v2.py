"""xshare_moe_forward_v2 (one argument struct) against the fixed-signature layer calls it
stands behind: identical outputs bit for bit, for every weight format, the hierarchical and
expert-parallel selections, shared experts, and logits computed from w_gate."""
import numpy as np
import pytest
import torch

import workloads as W
from helpers import DEV, say

pytestmark = pytest.mark.gpu


def _same(a, b, label):
    for key in ("y", "sel_mask", "ids", "w", "stats", "logits"):
        if key in a or key in b:
            ta, tb = a[key], b[key]
            if ta.dtype == torch.bfloat16:
                ta, tb = ta.view(torch.int16), tb.view(torch.int16)
            assert torch.equal(ta, tb), f"{label}: {key} differs"


def test_v2_equals_the_fixed_calls():
    from paper_2602_07265_amd import xshare as X
    c = W.CONFIGS["qwen"]
    T, N, k, d, f = c["T"], c["N"], c["k"], c["d"], c["f"]
    h, _ = W.make_logits(c, 0)
    hd = torch.from_numpy(h).to(DEV)
    x = W.activations(T, d, 0, DEV)
    w = W.expert_weights(N, d, f, 0, DEV)
    say("v2 case bf16 flat / threshold / dense")
    for M, mode, score, tau in [(32, "total", "topk", 0.0), (0, "threshold", "topk", 0.8),
                                (6, "extra", "dense", 0.0)]:
        a = X.moe_forward(x, hd, *w, k, 1, M, mode, score, tau=tau)
        b = X.moe_forward_v2(x, k, 1, M, mode, score, logits=hd, weights=w, tau=tau)
        torch.cuda.synchronize()
        _same(a, b, f"bf16 {mode} {score}")
    say("v2 case hierarchical")
    off = [0, 16, 32, 48, 64]
    a = X.moe_forward(x, hd, *w, k, 1, 32, req_offsets=off, per_request_budget=2)
    b = X.moe_forward_v2(x, k, 1, 32, logits=hd, weights=w, req_offsets=off,
                         per_request_budget=2)
    torch.cuda.synchronize()
    _same(a, b, "hierarchical")
    say("v2 case expert-parallel share")
    gm = X.GroupMap(8, None, local_group=3, device=DEV)
    a = X.moe_forward(x, hd, *w, k, 1, 4, groups=gm)
    b = X.moe_forward_v2(x, k, 1, 4, logits=hd, weights=w, groups=gm)
    torch.cuda.synchronize()
    _same(a, b, "ep share")
    say("v2 case shared experts and the router GEMM")
    sh = W.shared_weights(2, d, f, 0, DEV)
    wg = W.router_weights(N, d, 0, DEV)
    a = X.moe_forward(x, hd, *w, k, 1, 32, shared=sh)
    b = X.moe_forward_v2(x, k, 1, 32, logits=hd, weights=w, shared=sh)
    torch.cuda.synchronize()
    _same(a, b, "shared")
    a = X.moe_layer(x, wg, *w, k, 1, 32, shared=sh)
    b = X.moe_forward_v2(x, k, 1, 32, w_gate=wg, weights=w, shared=sh, logits_out=True)
    torch.cuda.synchronize()
    _same(a, b, "layer")
    say("v2 case FP8 and MXFP4 weights")
    q = W.expert_weights_fp8(N, d, f, 0, DEV)
    a = X.moe_forward_fp8(x, hd, *q, k, 1, 32)
    b = X.moe_forward_v2(x, k, 1, 32, logits=hd, weights=q[:3], scales=q[3:],
                         weight_format="fp8")
    torch.cuda.synchronize()
    _same(a, b, "fp8")
    q = X.mx_tiled(W.expert_weights_mxfp4(N, d, f, 0, DEV))
    a = X.moe_forward_mxfp4(x, hd, *q, k, 1, 32)
    b = X.moe_forward_v2(x, k, 1, 32, logits=hd, weights=q[:3], scales=q[3:],
                         weight_format="mxfp4")
    torch.cuda.synchronize()
    _same(a, b, "mxfp4")
    assert int(b["stats"][0]) == 32
