"""MoE layer with MXFP4 expert weights on the GPU (E2M1 codes, one E8M0 scale per 32 inputs
of a row): selection bit-exact, y within 2e-2 * RMS of the float64 oracle evaluated on the
same codes and scales (decoded exactly), so quantization error is not part of the
comparison."""
import numpy as np
import pytest
import torch

import workloads as W
from helpers import DEV, OracleOutputs, assert_ffn_close, assert_route_equal, oracle_route, say
from oracle import ffn as OF

pytestmark = pytest.mark.gpu



def _fetch(q1, q3, q2, e1, e3, e2):
    """Expert e's weights, decoded and scaled exactly (float64), for OracleOutputs."""
    return lambda e: tuple(OF.dequant_mx(q[e].cpu().numpy(), s[e].cpu().numpy())
                           for q, s in ((q1, e1), (q3, e3), (q2, e2)))


def _run(cfg, seed, k0, M, mode="total", weights=None, rows=None, offsets=None, m_r=0,
         groups=None, local=None, label=""):
    from paper_2602_07265_amd import xshare as X
    T, N, k, d, f = cfg["T"], cfg["N"], cfg["k"], cfg["d"], cfg["f"]
    h = W.make_logits(cfg, seed)[0] if offsets is None else cfg["h"]
    x = W.activations(T, d, seed, DEV)
    wts = weights if weights is not None else W.expert_weights_mxfp4(N, d, f, seed, DEV)
    say(f"mxfp4 case {label} T={T} N={N} k={k} d={d} f={f} k0={k0} M={M} {mode}")
    gm = None if groups is None else X.GroupMap(groups, None, local_group=local, device=DEV)
    res = X.moe_forward_mxfp4(x, torch.from_numpy(h).to(DEV), *X.mx_tiled(wts), k, k0, M, mode,
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


def test_mxfp4_tiny_and_ragged():
    c = W.CONFIGS["tiny"]
    for seed in range(3):
        for k0, M, mode in [(1, 8, "total"), (0, 2, "total"), (2, 0, "extra")]:
            _run(c, seed, k0, M, mode, label=f"tiny/s{seed}")
    # d, f of 96 / 160 run one 32-element group per step, 64 two, 128 four
    for T, N, k, d, f, M in [(37, 40, 4, 96, 160, 20), (1, 16, 2, 64, 32, 2),
                             (70, 24, 3, 128, 96, 24), (5, 8, 8, 32, 64, 8)]:
        _run(dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=3), 0, 1, M,
             label=f"ragged T{T} d{d} f{f}")


def test_mxfp4_many_rows_per_expert():
    """Few experts holding many rows each: the GEMMs stage up to 32 token rows per pass in
    LDS, so these cases run passes of 32 rows followed by ragged ones (1-8, 9-16, 17-24,
    25-32 rows), with 512-, 256-, 128- and 64-element steps and blocks whose last waves lie
    past f or d."""
    for T, N, k, d, f, M in [(70, 8, 4, 256, 512, 4), (40, 6, 3, 384, 192, 3),
                             (20, 4, 2, 192, 320, 2), (45, 8, 2, 320, 256, 3),
                             (33, 4, 2, 512, 160, 2), (21, 6, 3, 1024, 256, 3)]:
        _run(dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=2), 0, 1, M,
             label=f"many rows T{T} d{d} f{f} M{M}")


def test_mxfp4_largest_batches():
    """The size limits: T * k = 8192 (token, slot) rows, and T = 4096 tokens; experts with
    hundreds of rows, so the GEMMs loop over many staged 32-row passes."""
    for T, N, k, d, f, M in [(1024, 64, 8, 64, 64, 24), (4096, 16, 2, 64, 64, 4)]:
        _run(dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=4), 0, 1, M,
             label=f"largest T{T} k{k}")


def test_mx_scales_tile_layout():
    """xshare_mx_scales_tile against the layout written out with numpy, byte for byte:
    tiled[m][r / 16][c / 8][r % 16][c % 8] = scales[m][r][c], 127 past a row's last block
    (k = 96 and 288 end in a partial granule of 8 blocks)."""
    from paper_2602_07265_amd import xshare as X
    rng = np.random.default_rng(11)
    for n, rows, k in [(3, 32, 256), (2, 48, 96), (1, 16, 288), (2, 64, 7168)]:
        say(f"mx scale tiling n={n} rows={rows} k={k}")
        sc = rng.integers(0, 255, size=(n, rows, k // 32), dtype=np.uint8)
        got = X.tile_mx_scales(torch.from_numpy(sc).to(DEV)).cpu().numpy()
        G = (k + 255) // 256
        want = np.full((n, rows // 16, G, 16, 8), 127, dtype=np.uint8)
        for m in range(n):
            for r in range(rows):
                for c in range(k // 32):
                    want[m, r // 16, c // 8, r % 16, c % 8] = sc[m, r, c]
        assert np.array_equal(got, want), (n, rows, k)


@pytest.mark.parametrize("d,f", [(128, 128), (1024, 1280), (1280, 768), (2048, 512)])
def test_mxfp4_every_code_and_varied_scales(d, f):
    """Weight bytes cycling through all 256 pairs of E2M1 codes, block scales drawn from
    2^-14 .. 2^-6: the kernels' hardware decode and scaling must agree with the format.
    The GEMMs read each step's scale bytes from the tiled layout (granules of 256 inputs):
    d, f of 1024-2048 are whole granules, 1280 and 768 have 5 and 3, 128 half of one, and
    512 is split across blocks."""
    N, k, T = 8, 2, 12
    rng = np.random.default_rng(4 + d + f)

    def codes(r, c):
        return torch.from_numpy(rng.permutation(np.resize(np.arange(256, dtype=np.uint8),
                                                          r * c)).reshape(r, c)).to(DEV)

    def scales(r, c):
        return torch.from_numpy(rng.integers(113, 122, size=(r, c), dtype=np.uint8)).to(DEV)

    q1 = torch.stack([codes(f, d // 2) for _ in range(N)])
    q3 = torch.stack([codes(f, d // 2) for _ in range(N)])
    q2 = torch.stack([codes(d, f // 2) for _ in range(N)])
    e1 = torch.stack([scales(f, d // 32) for _ in range(N)])
    e3 = torch.stack([scales(f, d // 32) for _ in range(N)])
    e2 = torch.stack([scales(d, f // 32) for _ in range(N)])
    c = dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=2)
    _run(c, 0, 1, 4, weights=(q1, q3, q2, e1, e3, e2), label=f"every code d{d} f{f}")


def test_mxfp4_split_reductions():
    for T, N, k, d, f, M in [(16, 8, 2, 1024, 256, 4), (16, 8, 2, 128, 1024, 2),
                             (24, 16, 4, 512, 384, 16)]:
        _run(dict(N=N, k=k, d=d, f=f, T=T, logits="domains", Q=2), 0, 1, M,
             label=f"split T{T} d{d} f{f}")


def test_mxfp4_qwen_full_and_deepseek():
    c = W.CONFIGS["qwen"]
    _run(c, 0, 1, 32, label="qwen M32")
    c = W.CONFIGS["ds_t32"]
    wts = W.expert_weights_mxfp4(c["N"], c["d"], c["f"], 0, DEV)
    _run(c, 0, 1, 48, weights=wts, label="ds_t32 M48")
    _run(c, 1, 1, 24, weights=wts, label="ds_t32 M24")
    # 49 experts: 784 two-tile gate/up blocks, one slot past three rounds of 256 when one
    # block fits per CU (that slot then runs apart, split along d)
    _run(c, 2, 1, 49, weights=wts, label="ds_t32 M49")
    del wts
    torch.cuda.empty_cache()


def test_mxfp4_group_share_and_hierarchical():
    c = dict(N=32, k=4, d=128, f=256, T=24, logits="domains", Q=3)
    wts = W.expert_weights_mxfp4(32, 128, 256, 2, DEV)
    for local in (-1, 0, 3):
        _run(c, 2, 1, 3, groups=4, local=local, weights=wts, label=f"group share {local}")
    h, off = W.logits_spec(4, 4, 32, 2, 0)
    cs = dict(N=32, k=4, d=128, f=256, T=16, h=h)
    _run(cs, 0, 1, 12, offsets=off, m_r=2,
         weights=W.expert_weights_mxfp4(32, 128, 256, 0, DEV), label="hierarchical")


def test_mxfp4_deterministic_and_empty():
    from paper_2602_07265_amd import xshare as X
    c = W.CONFIGS["tiny"]
    h, _ = W.make_logits(c, 5)
    x = W.activations(c["T"], c["d"], 5, DEV)
    wts = W.expert_weights_mxfp4(c["N"], c["d"], c["f"], 5, DEV)
    hd = torch.from_numpy(h).to(DEV)
    say("mxfp4 case determinism and empty batch")
    tiled = X.mx_tiled(wts)
    a = X.moe_forward_mxfp4(x, hd, *tiled, 2, 1, 8)["y"]
    b = X.moe_forward_mxfp4(x, hd, *tiled, 2, 1, 8)["y"]
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    x0 = torch.empty((0, c["d"]), dtype=torch.bfloat16, device=DEV)
    r = X.moe_forward_mxfp4(x0, torch.empty((0, c["N"]), device=DEV), *tiled, 2, 1, 8)
    torch.cuda.synchronize()
    assert r["y"].shape == (0, c["d"]) and int(r["sel_mask"].sum()) == 0
