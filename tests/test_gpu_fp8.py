"""MoE layer with FP8 expert weights on the GPU (OCP E4M3FN codes, one fp32 scale per output
row): selection bit-exact, y within 2e-2 * RMS of the float64 oracle evaluated on the same
codes and scales (decoded exactly), so quantization error is not part of the comparison."""
import numpy as np
import pytest
import torch

import workloads as W
from helpers import DEV, OracleOutputs, assert_ffn_close, assert_route_equal, oracle_route, say
from oracle import ffn as OF

pytestmark = pytest.mark.gpu



def _fetch(q1, q3, q2, s1, s3, s2):
    """Expert e's weights, decoded and scaled exactly (float64), for OracleOutputs."""
    return lambda e: tuple(OF.dequant_rows(q[e].cpu().numpy(), s[e].cpu().numpy())
                           for q, s in ((q1, s1), (q3, s3), (q2, s2)))


def _run(cfg, seed, k0, M, mode="total", weights=None, rows=None, offsets=None, m_r=0,
         groups=None, local=None, label=""):
    from paper_2602_07265_amd import xshare as X
    T, N, k, d, f = cfg["T"], cfg["N"], cfg["k"], cfg["d"], cfg["f"]
    h = W.make_logits(cfg, seed)[0] if offsets is None else cfg["h"]
    x = W.activations(T, d, seed, DEV)
    wts = weights if weights is not None else W.expert_weights_fp8(N, d, f, seed, DEV)
    say(f"fp8 case {label} T={T} N={N} k={k} d={d} f={f} k0={k0} M={M} {mode}")
    gm = None if groups is None else X.GroupMap(groups, None, local_group=local, device=DEV)
    res = X.moe_forward_fp8(x, torch.from_numpy(h).to(DEV), *wts, k, k0, M, mode,
                            req_offsets=None if offsets is None else list(offsets),
                            per_request_budget=m_r, groups=gm)
    torch.cuda.synchronize()
    got = {key: v.cpu().numpy() for key, v in res.items() if key != "y"}
    if groups is None:
        ref = oracle_route(h, k, k0, M, mode, offsets=offsets, m_r=m_r)
        assert_route_equal(got, ref, label)
        mine = None
    else:
        from oracle import route as OR
        gr = OR.contiguous_groups(N, groups)
        ref = OR.select_ep(h, k, k0, M, gr, groups)
        assert np.array_equal(got["ids"], ref.ids), label
        mine = None if local is None or local < 0 else {e for e in range(N) if gr[e] == local}
    rows = list(range(T)) if rows is None else rows
    y_ref = OracleOutputs(x, _fetch(*wts)).y(ref.ids, ref.w, rows, local=mine)
    y_gpu = OF.bf16_to_f64(W.bf16_bits(res["y"]))[rows]
    assert np.all(np.isfinite(y_gpu))
    if mine is not None:
        hit = np.array([bool(set(ref.ids[i].tolist()) & mine) for i in rows])
        assert not np.any(y_gpu[~hit])
        y_gpu, y_ref = y_gpu[hit], y_ref[hit]
        if not len(y_ref):
            return res
    assert_ffn_close(y_gpu, y_ref, label)
    return res


def test_fp8_tiny_and_ragged():
    c = W.CONFIGS["tiny"]
    for seed in range(3):
        for k0, M, mode in [(1, 8, "total"), (0, 2, "total"), (2, 0, "extra")]:
            _run(c, seed, k0, M, mode, label=f"tiny/s{seed}")
    for T, N, k, d, f, M in [(37, 40, 4, 96, 160, 20), (1, 16, 2, 64, 32, 2),
                             (70, 24, 3, 128, 96, 24), (5, 8, 8, 32, 64, 8)]:
        _run(dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=3), 0, 1, M,
             label=f"ragged T{T} d{d} f{f}")


def test_fp8_many_rows_per_expert():
    """Few experts holding many rows each: passes of 32 staged token rows, then ragged ones
    (1-8, 9-16, 17-24, 25-32 rows), with blocks whose last waves lie past f or d."""
    for T, N, k, d, f, M in [(70, 8, 4, 256, 512, 4), (40, 6, 3, 384, 192, 3),
                             (20, 4, 2, 192, 320, 2), (45, 8, 2, 320, 256, 3)]:
        _run(dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=2), 0, 1, M,
             label=f"many rows T{T} d{d} f{f} M{M}")


def test_fp8_largest_batches():
    """The size limits: T * k = 8192 (token, slot) rows, and T = 4096 tokens; experts with
    hundreds of rows, so the GEMMs loop over many staged 32-row passes."""
    for T, N, k, d, f, M in [(1024, 64, 8, 64, 64, 24), (4096, 16, 2, 64, 64, 4)]:
        _run(dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=4), 0, 1, M,
             label=f"largest T{T} k{k}")


def test_fp8_every_code():
    """Weights cycling through every finite E4M3FN code (both signs, subnormals, 448) with
    power-of-two scales: the kernels' hardware decode must agree with the format."""
    N, k, d, f, T = 8, 2, 64, 128, 12
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)
    rng = np.random.default_rng(3)

    def mat(r, c):
        return torch.from_numpy(rng.permutation(np.resize(codes, r * c)).reshape(r, c)).to(DEV)

    q1 = torch.stack([mat(f, d) for _ in range(N)])
    q3 = torch.stack([mat(f, d) for _ in range(N)])
    q2 = torch.stack([mat(d, f) for _ in range(N)])
    s1 = torch.full((N, f), 2.0 ** -12, device=DEV)
    s3 = torch.full((N, f), 2.0 ** -12, device=DEV)
    s2 = torch.full((N, d), 2.0 ** -10, device=DEV)
    c = dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=2)
    _run(c, 0, 1, 4, weights=(q1, q3, q2, s1, s3, s2), label="every code")


def test_fp8_split_reductions():
    for T, N, k, d, f, M in [(16, 8, 2, 1024, 256, 4), (16, 8, 2, 128, 1024, 2),
                             (24, 16, 4, 512, 384, 16)]:
        _run(dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=2), 0, 1, M,
             label=f"split T{T} d{d} f{f}")


def test_fp8_qwen_full_and_deepseek():
    c = W.CONFIGS["qwen"]
    _run(c, 0, 1, 32, label="qwen M32")
    c = W.CONFIGS["ds_t32"]
    wts = W.expert_weights_fp8(c["N"], c["d"], c["f"], 0, DEV)
    _run(c, 0, 1, 48, weights=wts, label="ds_t32 M48")
    _run(c, 1, 1, 24, weights=wts, label="ds_t32 M24")
    # 49 experts: 784 two-tile gate/up blocks, one slot past three rounds of 256 when one
    # block fits per CU (that slot then runs apart, split along d)
    _run(c, 2, 1, 49, weights=wts, label="ds_t32 M49")
    del wts
    torch.cuda.empty_cache()


def test_fp8_group_share_and_hierarchical():
    c = dict(N=32, k=4, d=128, f=256, T=24, logits="domains", Q=3)
    wts = W.expert_weights_fp8(32, 128, 256, 2, DEV)
    for local in (-1, 0, 3):
        _run(c, 2, 1, 3, groups=4, local=local, weights=wts, label=f"group share {local}")
    h, off = W.logits_spec(4, 4, 32, 2, 0)
    cs = dict(N=32, k=4, d=128, f=256, T=16, h=h)
    _run(cs, 0, 1, 12, offsets=off, m_r=2, weights=W.expert_weights_fp8(32, 128, 256, 0, DEV),
         label="hierarchical")


def test_fp8_deterministic_and_empty():
    from paper_2602_07265_amd import xshare as X
    c = W.CONFIGS["tiny"]
    h, _ = W.make_logits(c, 5)
    x = W.activations(c["T"], c["d"], 5, DEV)
    wts = W.expert_weights_fp8(c["N"], c["d"], c["f"], 5, DEV)
    hd = torch.from_numpy(h).to(DEV)
    say("fp8 case determinism and empty batch")
    a = X.moe_forward_fp8(x, hd, *wts, 2, 1, 8)["y"]
    b = X.moe_forward_fp8(x, hd, *wts, 2, 1, 8)["y"]
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    x0 = torch.empty((0, c["d"]), dtype=torch.bfloat16, device=DEV)
    r = X.moe_forward_fp8(x0, torch.empty((0, c["N"]), device=DEV), *wts, 2, 1, 8)
    torch.cuda.synchronize()
    assert r["y"].shape == (0, c["d"]) and int(r["sel_mask"].sum()) == 0
