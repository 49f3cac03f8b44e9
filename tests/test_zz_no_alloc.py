"""The no-allocation entry point (xshare_moe_forward_noalloc) against xshare_moe_forward.

Same kernels, same plan: the routing must be identical bit for bit and y too (which is
stricter than the oracle's tolerance).  Two calls in a row, the second with a smaller
input, so the second runs on the scratch the first one left behind; then a call beyond the
scratch's size is refused before anything is enqueued, and the empty batch.
"""
import numpy as np
import pytest
import torch

import workloads as W
from helpers import DEV, say

pytestmark = pytest.mark.gpu


def _outs(T, N, k):
    return dict(sel_mask=torch.empty(N, dtype=torch.uint8, device=DEV),
                ids=torch.empty((T, k), dtype=torch.int32, device=DEV),
                w=torch.empty((T, k), dtype=torch.float32, device=DEV),
                stats=torch.empty(8, dtype=torch.int32, device=DEV))


def _same(cfg, seed, M, weights, label):
    from paper_2602_07265_amd import xshare as X
    T, N, k, d = cfg["T"], cfg["N"], cfg["k"], cfg["d"]
    h, _ = W.make_logits(cfg, seed)
    x = W.activations(T, d, seed, DEV)
    hd = torch.from_numpy(h).to(DEV)
    p = X.params(N, k, 1, M)
    need = X.moe_workspace_bytes(T, d, cfg["f"], p)
    say(f"noalloc case {label} T={T} N={N} d={d} f={cfg['f']} M={M} workspace {need} B")
    assert 0 < need <= X.NOALLOC_SCRATCH_BYTES
    got = X.moe_forward_noalloc(x, hd, *weights, k, 1, M, out=_outs(T, N, k))
    ref = X.moe_forward(x, hd, *weights, k, 1, M)
    torch.cuda.synchronize()
    for key in ("sel_mask", "ids", "w", "stats"):
        assert torch.equal(got[key], ref[key]), f"{label}: {key} differs"
    assert torch.equal(got["y"].view(torch.int16), ref["y"].view(torch.int16)), \
        f"{label}: y differs"
    assert int(got["stats"][0]) > 0 and bool(torch.isfinite(got["y"].float()).all())


def test_noalloc_equals_the_workspace_entry_point():
    from paper_2602_07265_amd import xshare as X
    c32, c8 = W.CONFIGS["ds_t32"], W.CONFIGS["ds_t8"]
    say("generating the DeepSeek-shaped expert weights (22.5 GB)")
    weights = W.expert_weights(c32["N"], c32["d"], c32["f"], 0, DEV)
    _same(c32, 0, 48, weights, "DeepSeek T=32 M=48")
    _same(c8, 1, 24, weights, "DeepSeek T=8 M=24 (smaller, after the larger)")
    # beyond the scratch: refused on the host, nothing enqueued
    T, N, k, d, f = 512, 256, 8, 7168, 2048
    assert X.moe_workspace_bytes(T, d, f, X.params(N, k, 1, 48)) > X.NOALLOC_SCRATCH_BYTES
    x = torch.zeros((T, d), dtype=torch.bfloat16, device=DEV)
    hd = torch.zeros((T, N), dtype=torch.float32, device=DEV)
    with pytest.raises(X.XShareError) as e:
        X.moe_forward_noalloc(x, hd, *weights, k, 1, 48)
    assert e.value.status == X.EWORKSPACE
    del weights
    torch.cuda.empty_cache()


def test_noalloc_small_and_empty():
    from paper_2602_07265_amd import xshare as X
    c = W.CONFIGS["qwen"]
    weights = W.expert_weights(c["N"], c["d"], c["f"], 0, DEV)
    _same(c, 0, 32, weights, "Qwen T=64 M=32")
    tiny = dict(c, T=5)
    _same(tiny, 2, 16, weights, "Qwen T=5 M=16")
    say("noalloc case empty batch")
    x0 = torch.empty((0, c["d"]), dtype=torch.bfloat16, device=DEV)
    r = X.moe_forward_noalloc(x0, torch.empty((0, c["N"]), device=DEV), *weights, 8, 1, 32,
                              out=_outs(0, c["N"], 8))
    torch.cuda.synchronize()
    assert r["y"].shape == (0, c["d"]) and int(r["sel_mask"].sum()) == 0
