"""MoE layer parity on the GPU: y within 2e-2 * RMS of the float64 oracle (Section 2.1).

The oracle routes independently (bit-exact routing is asserted too) and evaluates the
SwiGLU experts in float64 from the same bf16 inputs.  Every workload shape of the layer is
compared on all of its token rows: the DeepSeek-R1 shape at T = 8 and T = 32 with budgets
24, 48 and 96 (domain logits) and 48 (iid logits), the speculative 16 x 4 batch, the
Mixtral and Qwen-MoE shapes.  The oracle evaluates each routed expert once on every token
of a batch and the budgets' routings share those outputs.
"""
import numpy as np
import pytest
import torch

import workloads as W
from helpers import (DEV, OracleOutputs, assert_ffn_close, assert_route_equal, bf16_weights_of,
                     make_layer, oracle_route, say)
from oracle import ffn as OF

pytestmark = pytest.mark.gpu


def _run(cfg, seed, k0, M, mode="total", score="topk", rows=None, m_r=0, layer=None,
         oracle=None, label=""):
    from paper_2602_07265_amd import xshare as X
    h, off, x, w1, w3, w2 = layer if layer is not None else make_layer(cfg, seed)
    hier = cfg.get("logits") == "spec"
    say(f"ffn case {label} T={cfg['T']} N={cfg['N']} d={cfg['d']} f={cfg['f']} k0={k0} M={M} "
        f"{mode} {score}{' hier' if hier else ''}")
    res = X.moe_forward(x, torch.from_numpy(h).to(DEV), w1, w3, w2, cfg["k"], k0, M, mode, score,
                        req_offsets=list(off) if hier else None, per_request_budget=m_r)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in res.items() if k != "y"}
    ref = oracle_route(h, cfg["k"], k0, M, mode, score, off if hier else None, m_r)
    assert_route_equal(got, ref, label)
    rows = list(range(cfg["T"])) if rows is None else rows
    if oracle is None:
        oracle = OracleOutputs(x, bf16_weights_of(w1, w3, w2))
    y_ref = oracle.y(ref.ids, ref.w, rows)
    y_gpu = OF.bf16_to_f64(W.bf16_bits(res["y"]))[rows]
    assert_ffn_close(y_gpu, y_ref, label, f", |S|={got['stats'][0]} active={got['stats'][1]} "
                     f"|U|={got['stats'][2]}, {len(rows)} rows")
    return res, ref


@pytest.fixture(scope="module")
def ds_weights():
    """The DeepSeek-R1-shaped layer's expert weights (N=256, d=7168, f=2048, seed 0): the
    T = 8, T = 32 and speculative workloads draw the same weights for seed 0."""
    say("generating the DeepSeek-shaped expert weights (22.5 GB)")
    w = W.expert_weights(256, 7168, 2048, 0, DEV)
    yield w
    del w
    torch.cuda.empty_cache()


def _ds_layer(cfg, seed, weights):
    h, off = W.make_logits(cfg, seed)
    x = W.activations(cfg["T"], cfg["d"], seed, DEV)
    return (h, off, x, *weights)


def test_ffn_tiny_all_modes():
    c = W.CONFIGS["tiny"]
    for seed in range(4):
        layer = make_layer(c, seed)
        for k0, M, mode, score in [(1, 8, "total", "topk"), (0, 2, "total", "topk"),
                                   (2, 0, "extra", "topk"), (1, 8, "total", "dense"),
                                   (0, 16, "extra", "topk")]:
            _run(c, seed, k0, M, mode, score, layer=layer, label=f"tiny/s{seed}")


def test_ffn_ragged_shapes():
    for T, N, k, d, f, M in [(37, 40, 4, 96, 160, 20), (1, 16, 2, 64, 32, 2),
                             (70, 24, 3, 128, 96, 24), (5, 8, 8, 32, 64, 8)]:
        c = dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=3)
        _run(c, 0, 1, M, label=f"ragged T{T} d{d} f{f}")


def test_ffn_largest_batches():
    """The size limits: T * k = 8192 (token, slot) rows, and T = 4096 tokens; many tokens per
    expert, so the GEMMs loop over several 32-token passes."""
    for T, N, k, d, f, M in [(1024, 64, 8, 64, 64, 24), (4096, 16, 2, 32, 64, 4)]:
        c = dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=4)
        _run(c, 0, 1, M, label=f"largest T{T} k{k}")


def test_ffn_many_rows_per_expert():
    """Few experts holding many rows each: the GEMMs stage up to 32 token rows per pass in
    LDS, so these cases run passes of 32 rows followed by ragged ones (1-8, 9-16, 17-24,
    25-32 rows), with 128- and 64-element steps, a rotated down pass and blocks whose last
    waves lie past f or d."""
    for T, N, k, d, f, M in [(70, 8, 4, 256, 512, 4), (40, 6, 3, 384, 192, 3),
                             (20, 4, 2, 192, 320, 2), (45, 8, 2, 320, 256, 3)]:
        c = dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=2)
        _run(c, 0, 1, M, label=f"many rows T{T} d{d} f{f} M{M}")


def test_ffn_edge_shapes():
    """Top-1 and top-32 routing, the largest expert count (N = 1024), a budget of exactly
    k, a budget above N, and one expert per token."""
    for T, N, k, d, f, M, label in [(24, 16, 1, 128, 256, 4, "k=1"),
                                    (8, 64, 32, 64, 128, 40, "k=32"),
                                    (16, 1024, 8, 64, 64, 64, "N=1024"),
                                    (8, 32, 4, 128, 128, 4, "M=k"),
                                    (12, 64, 4, 96, 64, 200, "M>N"),
                                    (9, 9, 1, 64, 96, 9, "N=9 k=1")]:
        c = dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=3)
        _run(c, 0, 1, M, label=label)


def test_ffn_split_reduction():
    """Few, wide experts: the down GEMM splits f into 8, 8, 4 and 2 parts and the gate/up
    GEMM splits d into 8 and 4 parts (partials summed in split order); within tolerance."""
    for T, N, k, d, f, M in [(16, 8, 2, 128, 1024, 2), (8, 16, 2, 64, 2048, 3),
                             (40, 12, 3, 96, 512, 12), (16, 8, 2, 1024, 256, 4),
                             (24, 16, 4, 512, 384, 16)]:
        c = dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=2)
        _run(c, 0, 1, M, label=f"split T{T} d{d} f{f} M{M}")


def test_ffn_persistent_down_multi_pass():
    """The persistent seven-tile down launch (448 output rows per block, one block per CU)
    on experts that hold more than 32 routed rows, so a unit runs in several passes of up
    to 32 H rows, and blocks with one and with two units: N=64, k=8, T=64, d=7168 (16
    column blocks), f=256; budgets 16 and 32 make one and two whole rounds of 256 blocks."""
    c = dict(N=64, k=8, d=7168, f=256, T=64, logits="domains", Q=4)
    layer = make_layer(c, 2)
    oracle = OracleOutputs(layer[2], bf16_weights_of(*layer[3:]))
    for M in (16, 32):
        _, ref = _run(c, 2, 1, M, layer=layer, oracle=oracle, label=f"persistent down M{M}")
        rows = np.bincount(ref.ids.ravel(), minlength=c["N"])
        assert rows.max() > 32, f"M{M}: no expert above 32 rows ({rows.max()})"


def test_ffn_qwen_full():
    c = W.CONFIGS["qwen"]
    layer = make_layer(c, 0)
    for M in c["M_sweep"]:
        _run(c, 0, 1, M, layer=layer, label=f"qwen M{M}")
    _run(c, 0, 0, c["N"], "extra", layer=layer, label="qwen vanilla")


def test_ffn_mixtral():
    c = W.CONFIGS["mixtral"]
    _run(c, 0, 1, 5, label="mixtral")
    torch.cuda.empty_cache()


def test_ffn_deepseek_t32(ds_weights):
    """The headline shape at every budget of its sweep, all 32 rows; M = 96 exceeds |U| on
    some batches, so the whole union is selected there.  The iid control batch shares x."""
    c = W.CONFIGS["ds_t32"]
    layer = _ds_layer(c, 0, ds_weights)
    oracle = OracleOutputs(layer[2], bf16_weights_of(*ds_weights))
    for M in c["M_sweep"]:
        _run(c, 0, 1, M, layer=layer, oracle=oracle, label=f"ds_t32 M{M}")
    ci = W.CONFIGS["ds_iid_t32"]
    _run(ci, 0, 1, 48, layer=(*W.make_logits(ci, 0), *layer[2:]), oracle=oracle,
         label="ds_iid_t32 M48")


def test_ffn_deepseek_t8(ds_weights):
    """T = 8: the narrow down GEMM shape (few rows per expert); M = 48 and 96 reach |U|."""
    c = W.CONFIGS["ds_t8"]
    layer = _ds_layer(c, 0, ds_weights)
    oracle = OracleOutputs(layer[2], bf16_weights_of(*ds_weights))
    for M in c["M_sweep"]:
        _run(c, 0, 1, M, layer=layer, oracle=oracle, label=f"ds_t8 M{M}")
    ci = W.CONFIGS["ds_iid_t8"]
    _run(ci, 0, 1, 48, layer=(*W.make_logits(ci, 0), *layer[2:]), oracle=oracle,
         label="ds_iid_t8 M48")


def test_ffn_deepseek_one_token(ds_weights):
    """A single decoding token at the DeepSeek shape: S is its own top-k."""
    c = dict(W.CONFIGS["ds_t8"], T=1)
    layer = _ds_layer(c, 3, ds_weights)
    for M in (8, 48):
        _run(c, 3, 1, M, layer=layer, label=f"ds T=1 M{M}")


def test_ffn_spec_hier(ds_weights):
    """The speculative 16 x 4 batch, all 64 rows: hierarchical selection with m_r = 4 under a
    total budget of 64, and the paper's (k0, m, m_r) = (1, 0, 4) as an extra budget of 0."""
    c = W.CONFIGS["spec"]
    layer = _ds_layer(c, 0, ds_weights)
    oracle = OracleOutputs(layer[2], bf16_weights_of(*ds_weights))
    _run(c, 0, 1, 64, m_r=4, layer=layer, oracle=oracle, label="spec M64")
    _run(c, 0, 1, 0, "extra", m_r=4, layer=layer, oracle=oracle, label="spec extra 0")


def test_ffn_reads_only_selected_experts_and_is_deterministic():
    """Unselected experts' weights replaced by NaN: y must not change by a single bit."""
    from paper_2602_07265_amd import xshare as X
    c = W.CONFIGS["qwen"]
    h, _, x, w1, w3, w2 = make_layer(c, 1)
    hd = torch.from_numpy(h).to(DEV)
    say("ffn case poisoned unselected experts")
    a = X.moe_forward(x, hd, w1, w3, w2, 8, 1, 32)
    b = X.moe_forward(x, hd, w1, w3, w2, 8, 1, 32)
    torch.cuda.synchronize()
    assert torch.equal(a["y"].view(torch.int16), b["y"].view(torch.int16))
    unused = torch.ones(c["N"], dtype=torch.bool, device=DEV)
    unused[a["ids"].long().reshape(-1)] = False
    nan = torch.tensor(float("nan"), dtype=torch.bfloat16, device=DEV)
    for m in (w1, w3, w2):
        m[unused] = nan
    p = X.moe_forward(x, hd, w1, w3, w2, 8, 1, 32)
    torch.cuda.synchronize()
    assert int(unused.sum()) > 0
    assert torch.equal(a["y"].view(torch.int16), p["y"].view(torch.int16))


def test_ffn_empty_batch():
    from paper_2602_07265_amd import xshare as X
    say("ffn case empty batch")
    x = torch.empty((0, 64), dtype=torch.bfloat16, device=DEV)
    w1 = torch.zeros((16, 128, 64), dtype=torch.bfloat16, device=DEV)
    w2 = torch.zeros((16, 64, 128), dtype=torch.bfloat16, device=DEV)
    res = X.moe_forward(x, torch.empty((0, 16), device=DEV), w1, w1, w2, 2, 1, 8)
    torch.cuda.synchronize()
    assert res["y"].shape == (0, 64) and int(res["sel_mask"].sum()) == 0


def test_generator_identical_on_gpu_and_cpu():
    say("generator cpu/gpu")
    a = W.expert_matrix(3, "w2", 96, 64, 7, "cpu")
    b = W.expert_matrix(3, "w2", 96, 64, 7, DEV).cpu()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
