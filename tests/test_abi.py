"""The C-ABI library: it loads, exports every declared symbol, and validates on the host.

Every call below fails validation, so it returns before any HIP call: these tests run
without a GPU.  Fake non-null device pointers are never dereferenced.
"""
import ctypes
import os
import re
import subprocess

import pytest

from paper_2602_07265_amd import xshare as X

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "xshare.h")
FAKE = ctypes.c_void_p(1 << 20)        # 16-byte aligned, never dereferenced
FAKE_ODD = ctypes.c_void_p((1 << 20) + 2)


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(xshare_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert {"xshare_route", "xshare_select_hier", "xshare_select_ep", "xshare_moe_forward",
            "xshare_moe_forward_fp8", "xshare_moe_forward_mxfp4", "xshare_moe_layer",
            "xshare_router_logits", "xshare_layer_budgets"} <= set(names)
    lib = X.lib()
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", X.LIB_PATH], capture_output=True,
                         text=True).stdout
    exported = set(re.findall(r" T (xshare_\w+)", out))
    assert set(names) <= exported
    assert X.version().count(".") == 2


def test_status_strings():
    assert X.status_string(0) == "ok"
    for s in (1, 2, 3, 4):
        assert X.status_string(s) and X.status_string(s) != "unknown status"
    assert X.status_string(99) == "unknown status"


def test_workspace_sizes():
    p = X.params(256, 8, 1, 48)
    a = X.route_workspace_bytes(32, p)
    b = X.route_workspace_bytes(64, p)
    assert a > 0 and a % 256 == 0 and b >= a
    dense = X.params(256, 8, 1, 48, "total", "dense")
    assert X.route_workspace_bytes(32, dense) >= a + 32 * 256 * 4
    m = X.moe_workspace_bytes(32, 7168, 2048, p)
    # H (bf16 [T k, f]) and per-slot outputs (fp32 [T k, d]) dominate
    assert m >= a + 32 * 8 * (2048 * 2 + 7168 * 4)
    assert X.route_workspace_bytes(0, p) > 0
    assert X.route_workspace_bytes(32, X.params(256, 300, 1, 48)) == 0
    assert X.moe_workspace_bytes(32, 0, 2048, p) == 0


def _route(p, T=8, ws=FAKE, ws_bytes=1 << 30, logits=FAKE, mask=FAKE, ids=FAKE, w=FAKE):
    return X.lib().xshare_route(logits, T, ctypes.byref(p), mask, ids, w, None, ws, ws_bytes,
                                None)


@pytest.mark.parametrize("kw,status", [
    (dict(n_experts=0), X.EINVAL),
    (dict(top_k=0), X.EINVAL),
    (dict(top_k=17), X.EINVAL),            # k > N
    (dict(warmup_k0=3), X.EINVAL),         # k0 > k
    (dict(warmup_k0=-1), X.EINVAL),
    (dict(budget=1), X.EINVAL),            # total budget < k
    (dict(budget=-1, budget_mode=1), X.EINVAL),
    (dict(budget_mode=2), X.EINVAL),       # per-group budget without groups
    (dict(budget_mode=4), X.EINVAL),
    (dict(budget_mode=3, threshold=-0.5), X.EINVAL),
    (dict(budget_mode=3, threshold=float("nan")), X.EINVAL),
    (dict(budget_mode=3, threshold=float("inf")), X.EINVAL),
    (dict(budget_mode=3, threshold=0.8, budget=0), X.EWORKSPACE),   # valid: fails on ws
    (dict(score_mode=5), X.EINVAL),
    (dict(n_experts=2048, top_k=8, budget=64), X.EUNSUPPORTED),
    (dict(n_experts=64, top_k=33, budget=64), X.EUNSUPPORTED),
])
def test_route_parameter_validation(kw, status):
    base = dict(n_experts=16, top_k=2, warmup_k0=1, budget=8, budget_mode=0, score_mode=0,
                per_request_budget=0, threshold=0.0, ledger=None)
    base.update(kw)
    p = X.RouteParams(*[base[f] for f, _ in X.RouteParams._fields_])
    assert _route(p, ws=None) == status             # valid parameters stop at the workspace


def test_route_size_and_pointer_validation():
    p = X.params(16, 2, 1, 8)
    assert _route(p, T=-1) == X.EINVAL
    assert _route(p, T=4097) == X.EUNSUPPORTED
    assert _route(X.params(16, 4, 1, 8), T=4096) == X.EUNSUPPORTED    # T k > 8192
    assert _route(p, logits=None) == X.EINVAL
    assert _route(p, mask=None) == X.EINVAL
    assert _route(p, ids=None) == X.EINVAL
    assert _route(p, ws=None) == X.EWORKSPACE
    assert _route(p, ws_bytes=X.route_workspace_bytes(8, p) - 1) == X.EWORKSPACE
    assert X.lib().xshare_route(FAKE, 8, None, FAKE, FAKE, FAKE, None, FAKE, 1 << 30,
                                None) == X.EINVAL


def test_select_hier_offset_validation():
    p = X.params(16, 2, 1, 8, per_request_budget=2)
    L = X.lib()

    def call(host, R, T=8, dev=FAKE, pp=p):
        arr = None if host is None else (ctypes.c_int32 * len(host))(*host)
        return L.xshare_select_hier(FAKE, T, dev, arr, R, ctypes.byref(pp), FAKE, FAKE, FAKE, None,
                                    None, 0, None)

    assert call([0, 4, 4, 8], 3) == X.EINVAL        # empty request
    assert call([0, 5, 4, 8], 3) == X.EINVAL        # decreasing
    assert call([1, 4, 8], 2) == X.EINVAL           # must start at 0
    assert call([0, 4, 7], 2) == X.EINVAL           # must end at T
    assert call(None, 9) == X.EINVAL                # more requests than tokens
    assert call(None, 0) == X.EINVAL                # no request for a non-empty batch
    assert call(None, 2, dev=None) == X.EINVAL
    assert call([0, 4, 8], 2, pp=X.params(16, 2, 1, 8, per_request_budget=-1)) == X.EINVAL
    assert call([0, 4, 8], 2) == X.EWORKSPACE       # valid offsets; fails on the workspace


def test_moe_forward_validation():
    p = X.params(16, 2, 1, 8)
    L = X.lib()

    def call(d=64, f=128, x=FAKE, y=FAKE, ws=None, T=8):
        return L.xshare_moe_forward(x, FAKE, T, d, f, FAKE, FAKE, FAKE, ctypes.byref(p), None,
                                    None, 0, None, None, y, None, None, None, None, ws, 1 << 30,
                                    None, None)

    assert call(d=48) == X.EUNSUPPORTED
    assert call(f=100) == X.EUNSUPPORTED
    assert call(d=0) == X.EINVAL
    assert call(x=None) == X.EINVAL
    assert call(x=FAKE_ODD) == X.EINVAL             # 16-byte alignment of bf16 rows
    assert call(y=FAKE_ODD) == X.EINVAL
    assert call() == X.EWORKSPACE


def test_binding_refuses_cpu_tensors():
    import torch
    with pytest.raises(ValueError):
        X.route(torch.zeros(4, 16), 2, 1, 8)


def _ep(G, local=-1, host=None, dev=None):
    arr = None if host is None else (ctypes.c_int32 * len(host))(*host)
    lay = X.EpLayout(G, local, dev, None if arr is None else ctypes.addressof(arr))
    lay._keep = arr
    return lay


def test_select_ep_validation():
    L = X.lib()
    pg = X.params(16, 2, 1, 3, "per_group")

    def call(ep, pp=pg, ws=None):
        return L.xshare_select_ep(FAKE, 8, ctypes.byref(pp), None if ep is None else ctypes.byref(ep),
                                  FAKE, FAKE, FAKE, None, None, ws, 0 if ws is None else 1 << 30,
                                  None)

    assert call(None) == X.EINVAL                               # the layout is required
    assert call(_ep(4), pp=X.params(16, 2, 1, 8)) == X.EINVAL   # needs the per-group mode
    assert call(_ep(0)) == X.EINVAL
    assert call(_ep(17)) == X.EINVAL                            # more groups than experts
    assert call(_ep(3)) == X.EINVAL                             # 3 does not divide 16
    assert call(_ep(3, dev=1 << 20)) == X.EWORKSPACE            # any map on the device is fine
    assert call(_ep(2, host=[0] * 15 + [2], dev=1 << 20)) == X.EINVAL   # group id out of range
    assert call(_ep(2, host=[0, 1] * 8, dev=1 << 20)) == X.EWORKSPACE
    assert call(_ep(4), pp=X.params(16, 2, 1, -1, "per_group")) == X.EINVAL
    assert call(_ep(4)) == X.EWORKSPACE
    # the per-group mode is refused without groups
    assert _route(X.params(16, 2, 1, 8, "per_group")) == X.EINVAL


def test_moe_forward_ep_validation():
    L = X.lib()
    pg = X.params(16, 2, 1, 3, "per_group")

    def call(ep, pp=pg, offsets=None, R=0):
        return L.xshare_moe_forward(FAKE, FAKE, 8, 64, 128, FAKE, FAKE, FAKE, ctypes.byref(pp),
                                    offsets, None, R, None if ep is None else ctypes.byref(ep),
                                    None, FAKE, None, None, None, None, None, 1 << 30, None, None)

    assert call(_ep(4, local=4)) == X.EINVAL                    # local group out of range
    assert call(_ep(4, local=-2)) == X.EINVAL
    assert call(_ep(4, local=3)) == X.EWORKSPACE
    assert call(_ep(4), offsets=FAKE, R=2) == X.EUNSUPPORTED    # not with request offsets
    assert call(None, pp=pg) == X.EINVAL                        # per-group mode needs groups
    full = X.moe_workspace_bytes(32, 7168, 2048, X.params(256, 8, 1, 5, "per_group"), _ep(8))
    share = X.moe_workspace_bytes(32, 7168, 2048, X.params(256, 8, 1, 5, "per_group"),
                                  _ep(8, 0))
    assert full > 0 and share > 0
    assert X.moe_workspace_bytes(32, 7168, 2048, X.params(256, 8, 1, 5, "per_group"), None) == 0


def test_router_and_layer_validation():
    L = X.lib()
    assert X.lib().xshare_router_workspace_bytes(32, 7168, 256) > 0
    assert X.lib().xshare_router_workspace_bytes(32, 100, 256) == 0     # d % 32
    assert X.lib().xshare_router_workspace_bytes(32, 7168, 2000) == 0   # N > 1024

    def router(T=8, d=64, N=16, x=FAKE, wg=FAKE, out=FAKE):
        return L.xshare_router_logits(x, wg, T, d, N, out, None, 0, None)

    assert router(d=48) == X.EUNSUPPORTED
    assert router(N=0) == X.EINVAL
    assert router(N=2048) == X.EUNSUPPORTED
    assert router(x=None) == X.EINVAL
    assert router(x=FAKE_ODD) == X.EINVAL
    assert router(T=0) == X.OK                       # empty batch: nothing to do
    assert router(T=64, d=7168, N=256) == X.EWORKSPACE   # needs the partial sums

    p = X.params(16, 2, 1, 8)

    def layer(shared=None, ep=None, wg=FAKE, ws=None):
        return L.xshare_moe_layer(FAKE, wg, 8, 64, 128, FAKE, FAKE, FAKE,
                                  None if shared is None else ctypes.byref(shared),
                                  ctypes.byref(p if ep is None else pg), None, None, 0,
                                  None if ep is None else ctypes.byref(ep), FAKE, None, None,
                                  None, None, None, ws, 1 << 30, None, None)

    pg = X.params(16, 2, 1, 3, "per_group")
    assert layer() == X.EWORKSPACE
    assert layer(wg=None) == X.EINVAL
    assert layer(wg=FAKE_ODD) == X.EINVAL
    assert layer(X.SharedExperts(-1, None, None, None)) == X.EINVAL
    assert layer(X.SharedExperts(65, 1 << 20, 1 << 20, 1 << 20)) == X.EUNSUPPORTED
    assert layer(X.SharedExperts(1, None, 1 << 20, 1 << 20)) == X.EINVAL
    assert layer(X.SharedExperts(1, (1 << 20) + 2, 1 << 20, 1 << 20)) == X.EINVAL
    assert layer(X.SharedExperts(1, 1 << 20, 1 << 20, 1 << 20)) == X.EWORKSPACE
    assert layer(X.SharedExperts(1, 1 << 20, 1 << 20, 1 << 20), _ep(4, 1)) == X.EUNSUPPORTED
    q = X.params(256, 8, 1, 48)
    no = X.moe_workspace_bytes(32, 7168, 2048, q)
    one = X.moe_workspace_bytes(32, 7168, 2048, q, None, X.SharedExperts(1, 0, 0, 0))
    assert one >= no + 32 * (2048 * 2 + 7168 * 4)     # H and Y rows of the shared expert
    assert X.layer_workspace_bytes(32, 7168, 2048, q) > no


def test_moe_forward_fp8_validation():
    L = X.lib()
    p = X.params(16, 2, 1, 8)

    def call(q1=FAKE, q3=FAKE, q2=FAKE, s1=FAKE, s3=FAKE, s2=FAKE, d=64, f=128, T=8):
        return L.xshare_moe_forward_fp8(FAKE, FAKE, T, d, f, q1, q3, q2, s1, s3, s2,
                                        ctypes.byref(p), None, None, 0, None, FAKE, None, None,
                                        None, None, None, 1 << 30, None, None)

    assert call() == X.EWORKSPACE
    assert call(q1=None) == X.EINVAL
    assert call(q2=None) == X.EINVAL
    assert call(s3=None) == X.EINVAL                 # scales are required
    assert call(q3=FAKE_ODD) == X.EINVAL             # 16-byte alignment
    assert call(d=40) == X.EUNSUPPORTED


def test_moe_forward_mxfp4_validation():
    L = X.lib()
    p = X.params(16, 2, 1, 8)

    def call(q1=FAKE, q3=FAKE, q2=FAKE, e1=FAKE, e3=FAKE, e2=FAKE, d=64, f=128, T=8):
        return L.xshare_moe_forward_mxfp4(FAKE, FAKE, T, d, f, q1, q3, q2, e1, e3, e2,
                                          ctypes.byref(p), None, None, 0, None, FAKE, None,
                                          None, None, None, None, 1 << 30, None, None)

    assert call() == X.EWORKSPACE
    assert call(q1=None) == X.EINVAL
    assert call(q2=None) == X.EINVAL
    assert call(e1=None) == X.EINVAL                 # block scales are required
    assert call(e2=None) == X.EINVAL
    assert call(q3=FAKE_ODD) == X.EINVAL             # 16-byte alignment of the codes
    assert call(e3=FAKE_ODD) == X.EINVAL             # scale rows: 16-byte alignment
    assert call(e2=ctypes.c_void_p((1 << 20) + 8)) == X.EINVAL
    assert call(d=48) == X.EUNSUPPORTED              # d, f multiples of 32
    assert call(f=80) == X.EUNSUPPORTED


def test_mx_scales_tile_validation():
    """The tiled MXFP4 scale layout: ceil(k / 256) granules of 8 bytes per row; rows a
    multiple of 16 and k of 32, checked before any HIP call."""
    L = X.lib()
    assert L.xshare_mx_scales_tiled_bytes(2, 32, 7168) == 2 * 32 * 28 * 8
    assert L.xshare_mx_scales_tiled_bytes(1, 16, 96) == 16 * 1 * 8      # one partial granule
    assert L.xshare_mx_scales_tiled_bytes(1, 16, 288) == 16 * 2 * 8
    assert L.xshare_mx_scales_tiled_bytes(-1, 16, 256) == 0
    assert L.xshare_mx_scales_tile(FAKE, FAKE, 1, 24, 256, None) == X.EINVAL   # rows % 16
    assert L.xshare_mx_scales_tile(FAKE, FAKE, 1, 32, 48, None) == X.EINVAL    # k % 32
    assert L.xshare_mx_scales_tile(None, FAKE, 1, 32, 64, None) == X.EINVAL
    assert L.xshare_mx_scales_tile(FAKE, None, 1, 32, 64, None) == X.EINVAL
    assert L.xshare_mx_scales_tile(None, None, 0, 32, 64, None) == X.OK        # nothing to do


def _args(**kw):
    """An xshare_layer_args for a bf16 layer with fake device pointers (never dereferenced:
    every call below stops in validation)."""
    p = X.params(16, 2, 1, 8)
    a = X.LayerArgs()
    a.struct_size = ctypes.sizeof(X.LayerArgs)
    a.T, a.d, a.f = 8, 64, 128
    a.x = a.logits = a.y = FAKE.value
    a.w1 = a.w3 = a.w2 = FAKE.value
    a.weight_format = X.WEIGHTS["bf16"]
    a.params = ctypes.pointer(p)
    a._keep = p
    for key, v in kw.items():
        setattr(a, key, v)
    return a


def test_layer_args_struct_matches_the_header():
    # offsets of the C struct (x86-64): size_t, three int32, pointers 8-aligned
    assert ctypes.sizeof(X.LayerArgs) == 232
    assert X.LayerArgs.weight_format.offset == 48 and X.LayerArgs.R.offset == 128
    src = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    end = src.index("} xshare_layer_args;")
    body = src[src.rindex("typedef struct {", 0, end) + len("typedef struct {"):end]
    names = re.findall(r"(\w+)(?:\s*,\s*(\w+))?(?:\s*,\s*(\w+))?;", body)
    fields = [n for group in names for n in group if n]
    assert fields == [f for f, _ in X.LayerArgs._fields_]


def test_moe_forward_v2_validation():
    L = X.lib()
    v2 = lambda a: L.xshare_moe_forward_v2(ctypes.byref(a))
    assert L.xshare_moe_forward_v2(None) == X.EINVAL
    assert v2(_args()) == X.EWORKSPACE                       # valid: fails on the workspace
    assert v2(_args(struct_size=ctypes.sizeof(X.LayerArgs) - 8)) == X.EINVAL
    assert v2(_args(w_gate=FAKE.value)) == X.EINVAL          # both logits and w_gate
    assert v2(_args(logits=None)) == X.EINVAL                # neither
    assert v2(_args(logits=None, w_gate=FAKE.value)) == X.EWORKSPACE
    assert v2(_args(weight_format=3)) == X.EINVAL
    assert v2(_args(weight_format=X.WEIGHTS["fp8"])) == X.EINVAL      # scales missing
    assert v2(_args(weight_format=X.WEIGHTS["fp8"], w1_scale=FAKE.value, w3_scale=FAKE.value,
                    w2_scale=FAKE.value)) == X.EWORKSPACE
    assert v2(_args(weight_format=X.WEIGHTS["mxfp4"], w1_scale=FAKE.value,
                    w3_scale=FAKE.value, w2_scale=FAKE_ODD.value)) == X.EINVAL   # alignment
    assert v2(_args(d=48)) == X.EUNSUPPORTED
    assert v2(_args(x=FAKE_ODD.value)) == X.EINVAL
    assert v2(_args(T=0, x=None, logits=None, y=None)) == X.EWORKSPACE   # empty batch: no inputs
    assert v2(_args(ws=FAKE.value, ws_bytes=16)) == X.EWORKSPACE
    sh = X.SharedExperts(1, 1 << 20, 1 << 20, 1 << 20)
    assert v2(_args(shared=ctypes.pointer(sh), weight_format=X.WEIGHTS["fp8"],
                    w1_scale=FAKE.value, w3_scale=FAKE.value,
                    w2_scale=FAKE.value)) == X.EUNSUPPORTED          # shared experts: bf16 only


def test_moe_forward_v2_workspace_equals_the_fixed_calls():
    L = X.lib()
    ws2 = lambda a: int(L.xshare_moe_forward_v2_workspace_bytes(ctypes.byref(a)))
    for T, N, k, M, d, f in [(32, 256, 8, 48, 7168, 2048), (8, 16, 2, 8, 64, 128),
                             (64, 128, 8, 32, 2048, 768)]:
        p = X.params(N, k, 1, M)
        a = _args(T=T, d=d, f=f, params=ctypes.pointer(p))
        assert ws2(a) == X.moe_workspace_bytes(T, d, f, p) > 0
        a = _args(T=T, d=d, f=f, params=ctypes.pointer(p), logits=None, w_gate=FAKE.value)
        assert ws2(a) == X.layer_workspace_bytes(T, d, f, p) > 0
    assert L.xshare_moe_forward_v2_workspace_bytes(None) == 0
    assert ws2(_args(struct_size=8)) == 0
    assert ws2(_args(d=0)) == 0


def test_stream_probe_validation():
    L = X.lib()
    call = lambda buf=FAKE, n=1 << 20, blocks=64, sink=FAKE, mode=0: L.xshare_probe_stream_read(
        buf, n, blocks, mode, sink, None)
    assert call(buf=None) == X.EINVAL
    assert call(buf=FAKE_ODD) == X.EINVAL
    assert call(n=0) == X.EINVAL
    assert call(n=(1 << 20) + 8) == X.EINVAL
    assert call(blocks=0) == X.EINVAL
    assert call(sink=None) == X.EINVAL
    assert call(mode=4) == X.EINVAL


def test_block_times_only_in_the_profiling_build():
    """The product library exports xshare_block_times but has no timeline: it returns
    EUNSUPPORTED before touching anything (so it can be called here, without a GPU)."""
    L = X.lib()
    assert L.xshare_block_times(FAKE, FAKE, FAKE, 0, None) == X.EUNSUPPORTED
    assert L.xshare_block_times(None, None, None, 1, None) == X.EUNSUPPORTED
