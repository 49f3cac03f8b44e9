"""Out-of-bounds checks of the kernels at their real launch shapes, with guard bytes.

Every buffer the library writes (selection outputs, y, the workspace) sits between two
4 KB guards filled with 0xA5 that must survive the call; every buffer it reads (logits, x,
the expert weights, FP8 / MXFP4 scales) sits between guards of 0xFF bytes, which are NaN
in fp32, bf16, E4M3FN and E8M0, so a read past either end would reach the results, which
are then compared with the oracle as in the parity tests.  The cases reach the selection
modes (flat, hierarchical, GPU groups, dense scores, threshold), the largest expert count
and batch, and the GEMM launch variants: split reductions of both GEMMs, the gate/up tail
launch, the persistent down grid with multi-pass units, and the FP8 and MXFP4 passes.
"""
import numpy as np
import pytest
import torch

import workloads as W
from helpers import (DEV, OracleOutputs, assert_ffn_close, assert_route_equal,
                     bf16_weights_of, oracle_route, say)
from oracle import ffn as OF

pytestmark = pytest.mark.gpu

GUARD = 4096          # bytes on each side; a multiple of 256 keeps every view aligned
OUT_FILL = 0xA5       # around written buffers
IN_FILL = 0xFF        # around read buffers: NaN in every float format the library reads


class Guarded:
    """A device buffer of `nbytes` between two guards of `fill` bytes."""

    def __init__(self, nbytes, fill):
        self.n, self.fill = int(nbytes), fill
        self.base = torch.full((self.n + 2 * GUARD,), fill, dtype=torch.uint8, device=DEV)

    def view(self, dtype, shape):
        return self.base[GUARD:GUARD + self.n].view(dtype).view(shape)

    def intact(self):
        return bool((self.base[:GUARD] == self.fill).all()) and \
            bool((self.base[GUARD + self.n:] == self.fill).all())


def guarded_input(t):
    g = Guarded(t.numel() * t.element_size(), IN_FILL)
    v = g.view(t.dtype, tuple(t.shape))
    v.copy_(t)
    return g, v


def guarded_output(dtype, shape):
    n = int(np.prod(shape)) * torch.empty((), dtype=dtype).element_size()
    g = Guarded(n, OUT_FILL)
    return g, g.view(dtype, tuple(shape))


def guarded_workspace(nbytes):
    g = Guarded(max(int(nbytes), 256), OUT_FILL)
    return g, g.view(torch.uint8, (g.n,))


def assert_guards(label, written, read):
    for name, g in written.items():
        assert g.intact(), f"{label}: a write reached the guard of {name}"
    for name, g in read.items():
        assert g.intact(), f"{label}: the read-only guard of {name} changed"


def _route_case(label, h, k, k0, M, mode="total", score="topk", offsets=None, m_r=0, tau=0.0):
    from paper_2602_07265_amd import xshare as X
    T, N = h.shape
    say(f"guards route {label} T={T} N={N} k={k} k0={k0} M={M} {mode} {score}")
    gl, logits = guarded_input(torch.from_numpy(np.ascontiguousarray(h)).to(DEV))
    outs = {"sel_mask": guarded_output(torch.uint8, (N,)), "ids": guarded_output(torch.int32, (T, k)),
            "w": guarded_output(torch.float32, (T, k)), "stats": guarded_output(torch.int32, (8,))}
    p = X.params(N, k, k0, M, mode, score, m_r, tau)
    gw, ws = guarded_workspace(X.route_workspace_bytes(T, p))
    out = {key: v for key, (_, v) in outs.items()}
    if offsets is None:
        res = X.route(logits, k, k0, M, mode, score, tau=tau, out=out, workspace=ws)
    else:
        res = X.select_hier(logits, list(int(v) for v in offsets), k, k0, m_r, M, mode, score,
                            tau=tau, out=out, workspace=ws)
    torch.cuda.synchronize()
    assert_guards(label, {**{key: g for key, (g, _) in outs.items()}, "workspace": gw},
                  {"logits": gl})
    got = {key: v.cpu().numpy() for key, v in res.items()}
    ref = oracle_route(h, k, k0, M, mode, score, offsets, m_r, tau if mode == "threshold" else None)
    assert_route_equal(got, ref, label)


def test_route_guards():
    for T, N, k, M in [(37, 40, 4, 20), (32, 256, 8, 48), (16, 1024, 8, 64), (4096, 16, 2, 4),
                       (1, 8, 8, 8)]:
        c = dict(N=N, k=k, T=T, logits="domains", Q=4)
        h = W.make_logits(c, 1)[0]
        _route_case(f"flat T{T} N{N}", h, k, 1, M)
    c = dict(N=256, k=8, T=32, logits="domains", Q=8)
    h = W.make_logits(c, 2)[0]
    _route_case("dense", h, 8, 1, 48, score="dense")
    _route_case("extra k0=0", h, 8, 0, 16, mode="extra")
    _route_case("threshold", h, 8, 1, 0, mode="threshold", tau=0.8)
    cs = W.CONFIGS["spec"]
    hs, off = W.make_logits(cs, 0)
    _route_case("hier m_r=4", hs, cs["k"], 1, 64, offsets=off, m_r=4)


def test_select_ep_guards():
    from paper_2602_07265_amd import xshare as X
    from oracle import route as OR
    T, N, k, G, mg = 32, 256, 8, 8, 5
    h = W.make_logits(dict(N=N, k=k, T=T, logits="domains", Q=8), 3)[0]
    say(f"guards select_ep T={T} N={N} G={G} m_g={mg}")
    gl, logits = guarded_input(torch.from_numpy(h).to(DEV))
    gm = X.GroupMap(G, None, device=DEV)
    outs = {"sel_mask": guarded_output(torch.uint8, (N,)), "ids": guarded_output(torch.int32, (T, k)),
            "w": guarded_output(torch.float32, (T, k)), "stats": guarded_output(torch.int32, (8,))}
    p = X.params(N, k, 1, mg, "per_group")
    gw, ws = guarded_workspace(X.route_workspace_bytes(T, p))
    res = X.select_ep(logits, gm, k, 1, mg, out={key: v for key, (_, v) in outs.items()},
                      workspace=ws)
    torch.cuda.synchronize()
    assert_guards("select_ep", {**{key: g for key, (g, _) in outs.items()}, "workspace": gw},
                  {"logits": gl})
    ref = OR.select_ep(h, k, 1, mg, OR.contiguous_groups(N, G), G)
    assert np.array_equal(res["ids"].cpu().numpy(), ref.ids)
    assert np.array_equal(res["sel_mask"].cpu().numpy(), ref.sel_mask)


def _moe_case(label, cfg, seed, M, fmt="bf16"):
    from paper_2602_07265_amd import xshare as X
    T, N, k, d, f = cfg["T"], cfg["N"], cfg["k"], cfg["d"], cfg["f"]
    say(f"guards moe {fmt} {label} T={T} N={N} k={k} d={d} f={f} M={M}")
    h = W.make_logits(cfg, seed)[0]
    gl, logits = guarded_input(torch.from_numpy(h).to(DEV))
    gx, x = guarded_input(W.activations(T, d, seed, DEV))
    if fmt == "bf16":
        wts = W.expert_weights(N, d, f, seed, DEV)
        fetch = bf16_weights_of(*wts)
        fwd = X.moe_forward
    elif fmt == "fp8":
        wts = W.expert_weights_fp8(N, d, f, seed, DEV)
        q1, q3, q2, s1, s3, s2 = wts
        fetch = lambda e: tuple(OF.dequant_rows(q[e].cpu().numpy(), s[e].cpu().numpy())
                                for q, s in ((q1, s1), (q3, s3), (q2, s2)))
        fwd = X.moe_forward_fp8
    else:
        base = W.expert_weights_mxfp4(N, d, f, seed, DEV)
        q1, q3, q2, e1, e3, e2 = base
        fetch = lambda e: tuple(OF.dequant_mx(q[e].cpu().numpy(), s[e].cpu().numpy())
                                for q, s in ((q1, e1), (q3, e3), (q2, e2)))
        wts = X.mx_tiled(base)
        fwd = X.moe_forward_mxfp4
    gw_in = [guarded_input(t) for t in wts]
    gy, y = guarded_output(torch.bfloat16, (T, d))
    need = (X.moe_workspace_bytes(T, d, f, X.params(N, k, 1, M)))
    gws, ws = guarded_workspace(need)
    res = fwd(x, logits, *[v for _, v in gw_in], k, 1, M, y=y, workspace=ws)
    torch.cuda.synchronize()
    assert_guards(f"{fmt} {label}", {"y": gy, "workspace": gws},
                  {"logits": gl, "x": gx, **{f"weights[{i}]": g for i, (g, _) in enumerate(gw_in)}})
    ref = oracle_route(h, k, 1, M)
    assert_route_equal({key: v.cpu().numpy() for key, v in res.items() if key != "y"}, ref, label)
    y_ref = OracleOutputs(x, fetch).y(ref.ids, ref.w)
    assert_ffn_close(OF.bf16_to_f64(W.bf16_bits(res["y"])), y_ref, f"{fmt} {label}")
    return res


def _cfg(T, N, k, d, f, Q=3):
    return dict(T=T, N=N, k=k, d=d, f=f, logits="domains", Q=Q)


def test_moe_guards_bf16_launch_variants():
    _moe_case("tiny", _cfg(8, 16, 2, 64, 128), 0, 8)
    _moe_case("ragged", _cfg(37, 40, 4, 96, 160), 1, 20)
    _moe_case("down split", _cfg(16, 8, 2, 128, 1024, 2), 0, 2)
    _moe_case("gate/up split", _cfg(16, 8, 2, 1024, 256, 2), 0, 4)
    _moe_case("many rows", _cfg(70, 8, 4, 256, 512, 2), 0, 4)


def test_moe_guards_bf16_tail_and_persistent():
    """A gate/up launch of one full round of one-tile blocks and one slot more (the tail
    launch and its finish pass), and the persistent seven-tile down grid with units of
    more than 32 rows."""
    _moe_case("gate/up tail", _cfg(32, 16, 4, 2048, 4096, 3), 0, 9)
    torch.cuda.empty_cache()
    _moe_case("persistent down", _cfg(64, 64, 8, 7168, 256, 4), 2, 16)
    torch.cuda.empty_cache()


def test_moe_guards_low_precision():
    for fmt in ("fp8", "mxfp4"):
        _moe_case("small", _cfg(16, 8, 2, 256, 512), 0, 4, fmt)
        _moe_case("ragged", _cfg(37, 24, 4, 512, 256), 1, 12, fmt)
        _moe_case("down split", _cfg(16, 8, 2, 256, 2048, 2), 0, 2, fmt)
