"""Python binding of libxshare.so (argument marshalling only).

Every computation runs in the HIP kernels behind the C ABI of include/xshare.h; this module
checks tensor devices/dtypes/shapes, carves nothing itself except the workspace tensor it
allocates when none is passed, and forwards raw device pointers plus the current HIP stream.
There is no fallback: if the library is not built or no GPU is present, calls raise.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libxshare.so")
# the profiling build (block timeline of the expert GEMMs, xshare_block_times)
TIMELINE_LIB_PATH = os.path.join(_HERE, "libxshare_timeline.so")
TIME_BLOCKS, TIME_SEQ_BLOCKS, TIME_SEQ_STRIDE = 16384, 1024, 33   # XSHARE_TIME_*

OK, EINVAL, EUNSUPPORTED, EWORKSPACE, EHIP = 0, 1, 2, 3, 4
BUDGET = {"total": 0, "extra": 1, "per_group": 2, "threshold": 3}
SCORE = {"topk": 0, "dense": 1}
N_STAGE_EVENTS = 5
NOALLOC_SCRATCH_BYTES = 64 << 20     # XSHARE_NOALLOC_SCRATCH_BYTES
STAGES = ("route", "gate_up", "down", "combine")


class RouteParams(ctypes.Structure):
    _fields_ = [
        ("n_experts", ctypes.c_int32),
        ("top_k", ctypes.c_int32),
        ("warmup_k0", ctypes.c_int32),
        ("budget", ctypes.c_int32),
        ("budget_mode", ctypes.c_int32),
        ("score_mode", ctypes.c_int32),
        ("per_request_budget", ctypes.c_int32),
        ("threshold", ctypes.c_float),
        ("ledger", ctypes.c_void_p),
    ]


class EpLayout(ctypes.Structure):
    _fields_ = [
        ("n_groups", ctypes.c_int32),
        ("local_group", ctypes.c_int32),
        ("expert_group", ctypes.c_void_p),
        ("host_expert_group", ctypes.c_void_p),
    ]


class SharedExperts(ctypes.Structure):
    _fields_ = [
        ("n_shared", ctypes.c_int32),
        ("w1", ctypes.c_void_p),
        ("w3", ctypes.c_void_p),
        ("w2", ctypes.c_void_p),
    ]


class LayerArgs(ctypes.Structure):
    """xshare_layer_args (include/xshare.h), the argument struct of xshare_moe_forward_v2."""
    _fields_ = [
        ("struct_size", ctypes.c_size_t),
        ("T", ctypes.c_int32), ("d", ctypes.c_int32), ("f", ctypes.c_int32),
        ("x", ctypes.c_void_p), ("logits", ctypes.c_void_p), ("w_gate", ctypes.c_void_p),
        ("weight_format", ctypes.c_int32),
        ("w1", ctypes.c_void_p), ("w3", ctypes.c_void_p), ("w2", ctypes.c_void_p),
        ("w1_scale", ctypes.c_void_p), ("w3_scale", ctypes.c_void_p),
        ("w2_scale", ctypes.c_void_p),
        ("params", ctypes.POINTER(RouteParams)),
        ("req_offsets", ctypes.c_void_p), ("host_offsets", ctypes.c_void_p),
        ("R", ctypes.c_int32),
        ("ep", ctypes.POINTER(EpLayout)), ("shared", ctypes.POINTER(SharedExperts)),
        ("y", ctypes.c_void_p), ("logits_out", ctypes.c_void_p), ("sel_mask", ctypes.c_void_p),
        ("topk_ids", ctypes.c_void_p), ("topk_w", ctypes.c_void_p), ("stats", ctypes.c_void_p),
        ("ws", ctypes.c_void_p), ("ws_bytes", ctypes.c_size_t),
        ("stage_events", ctypes.c_void_p),
        ("stream", ctypes.c_void_p),
    ]


WEIGHTS = {"bf16": 0, "fp8": 1, "mxfp4": 2}

STATS_FIELDS = ("n_selected", "n_active", "n_vanilla_union", "n_warmup", "n_start",
                "budget_eff", "max_group_load")


class XShareError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} ({status})")
        self.status = status


_lib = None
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_SZ = ctypes.c_size_t


def lib() -> ctypes.CDLL:
    """The loaded libxshare.so (raises if it was not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -m paper_2602_07265_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        L.xshare_route_workspace_bytes.argtypes = [_I32, ctypes.POINTER(RouteParams)]
        L.xshare_route_workspace_bytes.restype = _SZ
        L.xshare_moe_workspace_bytes.argtypes = [_I32, _I32, _I32, ctypes.POINTER(RouteParams),
                                                 ctypes.POINTER(EpLayout),
                                                 ctypes.POINTER(SharedExperts)]
        L.xshare_moe_workspace_bytes.restype = _SZ
        L.xshare_layer_workspace_bytes.argtypes = [_I32, _I32, _I32, ctypes.POINTER(RouteParams),
                                                   ctypes.POINTER(EpLayout),
                                                   ctypes.POINTER(SharedExperts)]
        L.xshare_layer_workspace_bytes.restype = _SZ
        L.xshare_router_workspace_bytes.argtypes = [_I32, _I32, _I32]
        L.xshare_router_workspace_bytes.restype = _SZ
        L.xshare_router_logits.argtypes = [_P, _P, _I32, _I32, _I32, _P, _P, _SZ, _P]
        L.xshare_router_logits.restype = ctypes.c_int
        L.xshare_moe_layer.argtypes = [_P, _P, _I32, _I32, _I32, _P, _P, _P,
                                       ctypes.POINTER(SharedExperts), ctypes.POINTER(RouteParams),
                                       _P, _P, _I32, ctypes.POINTER(EpLayout), _P, _P, _P, _P, _P,
                                       _P, _P, _SZ, _P, _P]
        L.xshare_moe_layer.restype = ctypes.c_int
        L.xshare_moe_forward_fp8.argtypes = [_P, _P, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P,
                                             ctypes.POINTER(RouteParams), _P, _P, _I32,
                                             ctypes.POINTER(EpLayout), _P, _P, _P, _P, _P, _P,
                                             _SZ, _P, _P]
        L.xshare_moe_forward_fp8.restype = ctypes.c_int
        L.xshare_moe_forward_mxfp4.argtypes = [_P, _P, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P,
                                             ctypes.POINTER(RouteParams), _P, _P, _I32,
                                             ctypes.POINTER(EpLayout), _P, _P, _P, _P, _P, _P,
                                             _SZ, _P, _P]
        L.xshare_moe_forward_mxfp4.restype = ctypes.c_int
        L.xshare_mx_scales_tiled_bytes.argtypes = [_I32, _I32, _I32]
        L.xshare_mx_scales_tiled_bytes.restype = _SZ
        L.xshare_mx_scales_tile.argtypes = [_P, _P, _I32, _I32, _I32, _P]
        L.xshare_mx_scales_tile.restype = ctypes.c_int
        L.xshare_route.argtypes = [_P, _I32, ctypes.POINTER(RouteParams), _P, _P, _P, _P, _P, _SZ,
                                   _P]
        L.xshare_route.restype = ctypes.c_int
        L.xshare_select_hier.argtypes = [_P, _I32, _P, _P, _I32, ctypes.POINTER(RouteParams), _P,
                                         _P, _P, _P, _P, _SZ, _P]
        L.xshare_select_hier.restype = ctypes.c_int
        L.xshare_select_ep.argtypes = [_P, _I32, ctypes.POINTER(RouteParams),
                                       ctypes.POINTER(EpLayout), _P, _P, _P, _P, _P, _P, _SZ, _P]
        L.xshare_select_ep.restype = ctypes.c_int
        L.xshare_moe_forward.argtypes = [_P, _P, _I32, _I32, _I32, _P, _P, _P,
                                         ctypes.POINTER(RouteParams), _P, _P, _I32,
                                         ctypes.POINTER(EpLayout), ctypes.POINTER(SharedExperts),
                                         _P, _P, _P, _P, _P, _P, _SZ, _P, _P]
        L.xshare_moe_forward.restype = ctypes.c_int
        L.xshare_moe_forward_noalloc.argtypes = [_P, _P, _I32, _I32, _I32, _P, _P, _P,
                                                 ctypes.POINTER(RouteParams), _P, _P, _I32,
                                                 ctypes.POINTER(EpLayout),
                                                 ctypes.POINTER(SharedExperts), _P, _P, _P, _P,
                                                 _P, _P, _P]
        L.xshare_moe_forward_noalloc.restype = ctypes.c_int
        L.xshare_moe_forward_v2.argtypes = [ctypes.POINTER(LayerArgs)]
        L.xshare_moe_forward_v2.restype = ctypes.c_int
        L.xshare_moe_forward_v2_workspace_bytes.argtypes = [ctypes.POINTER(LayerArgs)]
        L.xshare_moe_forward_v2_workspace_bytes.restype = _SZ
        L.xshare_probe_stream_read.argtypes = [_P, _SZ, _I32, _I32, _P, _P]
        L.xshare_probe_stream_read.restype = ctypes.c_int
        L.xshare_block_times.argtypes = [_P, _P, _P, _I32, _P]
        L.xshare_block_times.restype = ctypes.c_int
        L.xshare_status_string.argtypes = [_I32]
        L.xshare_status_string.restype = ctypes.c_char_p
        L.xshare_version.argtypes = []
        L.xshare_version.restype = ctypes.c_char_p
        L.xshare_layer_budgets.argtypes = [_I32, _I32, _P]
        L.xshare_layer_budgets.restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().xshare_status_string(int(status)).decode()


def version() -> str:
    return lib().xshare_version().decode()


def params(n_experts: int, top_k: int, warmup_k0: int, budget: int, budget_mode="total",
           score_mode="topk", per_request_budget: int = 0, threshold: float = 0.0,
           ledger=None) -> RouteParams:
    """``threshold`` is tau of the "threshold" budget mode (Algorithm 1's stopping rule);
    ``ledger`` an optional device int32 tensor of LEDGER_FIELDS' length that the call adds
    its counts to."""
    if ledger is not None:
        _dev(ledger, torch.int32, (len(LEDGER_FIELDS) + 2,), "ledger")
    return RouteParams(int(n_experts), int(top_k), int(warmup_k0), int(budget),
                       BUDGET[budget_mode] if isinstance(budget_mode, str) else int(budget_mode),
                       SCORE[score_mode] if isinstance(score_mode, str) else int(score_mode),
                       int(per_request_budget), float(threshold),
                       None if ledger is None else ledger.data_ptr())


LEDGER_FIELDS = ("layers", "selected", "active", "vanilla_union", "invalid", "max_selected")


def new_ledger(device="cuda") -> torch.Tensor:
    """A zeroed budget ledger (xshare_budget_ledger) in device memory."""
    return torch.zeros(len(LEDGER_FIELDS) + 2, dtype=torch.int32, device=device)


def ledger_dict(ledger: torch.Tensor) -> dict:
    return dict(zip(LEDGER_FIELDS, ledger.to("cpu").tolist()))


def layer_budgets(K: int, L: int) -> list:
    """Uniform per-layer budgets m_l for a global budget K over L layers (host call)."""
    m = (ctypes.c_int32 * max(int(L), 1))()
    _check(lib().xshare_layer_budgets(int(K), int(L), m), "xshare_layer_budgets")
    return [int(v) for v in m[:int(L)]]


def route_workspace_bytes(T: int, p: RouteParams) -> int:
    return int(lib().xshare_route_workspace_bytes(int(T), ctypes.byref(p)))


def moe_workspace_bytes(T: int, d: int, f: int, p: RouteParams, ep=None, shared=None) -> int:
    """``ep``: an EpLayout or None; ``shared``: a SharedExperts or None."""
    return int(lib().xshare_moe_workspace_bytes(int(T), int(d), int(f), ctypes.byref(p),
                                                None if ep is None else ctypes.byref(ep),
                                                None if shared is None else ctypes.byref(shared)))


def layer_workspace_bytes(T: int, d: int, f: int, p: RouteParams, ep=None, shared=None) -> int:
    return int(lib().xshare_layer_workspace_bytes(int(T), int(d), int(f), ctypes.byref(p),
                                                  None if ep is None else ctypes.byref(ep),
                                                  None if shared is None else ctypes.byref(shared)))


def _shared(shared, d, f, dev):
    """SharedExperts from a (w1 [N_s,f,d], w3 [N_s,f,d], w2 [N_s,d,f]) tuple of bf16 tensors."""
    if shared is None:
        return None
    w1, w3, w2 = shared
    ns = w1.shape[0]
    _dev(w1, torch.bfloat16, (ns, f, d), "shared w1")
    _dev(w3, torch.bfloat16, (ns, f, d), "shared w3")
    _dev(w2, torch.bfloat16, (ns, d, f), "shared w2")
    return SharedExperts(int(ns), w1.data_ptr(), w3.data_ptr(), w2.data_ptr())


def router_logits(x: torch.Tensor, w_gate: torch.Tensor, *, out=None, workspace=None,
                  stream=None) -> torch.Tensor:
    """h = W_g x on the GPU (fp32 [T, N])."""
    T, d = x.shape
    N = w_gate.shape[0]
    _dev(x, torch.bfloat16, (T, d), "x")
    _dev(w_gate, torch.bfloat16, (N, d), "w_gate")
    out = torch.empty((T, N), dtype=torch.float32, device=x.device) if out is None else out
    _dev(out, torch.float32, (T, N), "logits")
    need = int(lib().xshare_router_workspace_bytes(T, d, N))
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=x.device)
    st = lib().xshare_router_logits(_ptr(x), _ptr(w_gate), T, d, N, _ptr(out), _ptr(workspace),
                                    workspace.numel(), _stream(stream))
    _check(st, "xshare_router_logits")
    return out


class GroupMap:
    """GPU groups of the experts for expert parallelism: ``groups`` None (equal contiguous
    blocks of N / G) or a per-expert sequence / device int32 tensor of group ids."""

    def __init__(self, n_groups: int, groups=None, local_group: int = -1, device="cuda"):
        self.host = None
        self.dev = None
        if groups is not None:
            if isinstance(groups, torch.Tensor) and groups.is_cuda:
                self.dev = _dev(groups, torch.int32, (groups.numel(),), "expert_group")
            else:
                self.host = torch.as_tensor([int(v) for v in groups], dtype=torch.int32)
                self.dev = self.host.to(device)
        self.layout = EpLayout(int(n_groups), int(local_group),
                               None if self.dev is None else self.dev.data_ptr(),
                               None if self.host is None else self.host.data_ptr())

    def with_local(self, local_group: int) -> "GroupMap":
        g = GroupMap.__new__(GroupMap)
        g.host, g.dev = self.host, self.dev
        g.layout = EpLayout(self.layout.n_groups, int(local_group), self.layout.expert_group,
                            self.layout.host_expert_group)
        return g


# ----------------------------------------------------------------------------- helpers

def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t, dtype, shape, name):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check(status, what):
    if status != OK:
        raise XShareError(status, what)


def stats_dict(stats: torch.Tensor) -> dict:
    v = stats.to("cpu").tolist()
    return dict(zip(STATS_FIELDS, v))


def _offsets(req_offsets, device):
    """(device int32 tensor, host int32 array pointer holder) from a list/array/tensor."""
    if isinstance(req_offsets, torch.Tensor) and req_offsets.is_cuda:
        dev = _dev(req_offsets, torch.int32, (req_offsets.numel(),), "req_offsets")
        return dev, None
    host = torch.as_tensor(list(int(v) for v in req_offsets), dtype=torch.int32)
    return host.to(device), host


# ----------------------------------------------------------------------------- entry points

def _route_impl(logits, p, req_offsets, out, workspace, stream):
    T, N = logits.shape
    k = p.top_k
    dev = logits.device
    _dev(logits, torch.float32, (T, N), "logits")
    if N != p.n_experts:
        raise ValueError("logits width must equal n_experts")
    out = dict(out or {})
    sel = out.get("sel_mask") if out.get("sel_mask") is not None else torch.empty(N, dtype=torch.uint8, device=dev)
    ids = out.get("ids") if out.get("ids") is not None else torch.empty((T, k), dtype=torch.int32, device=dev)
    w = out.get("w") if out.get("w") is not None else torch.empty((T, k), dtype=torch.float32, device=dev)
    stats = out.get("stats") if out.get("stats") is not None else torch.empty(8, dtype=torch.int32, device=dev)
    _dev(sel, torch.uint8, (N,), "sel_mask")
    _dev(ids, torch.int32, (T, k), "ids")
    _dev(w, torch.float32, (T, k), "w")
    _dev(stats, torch.int32, (8,), "stats")
    need = route_workspace_bytes(T, p)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    if req_offsets is None:
        st = lib().xshare_route(_ptr(logits), T, ctypes.byref(p), _ptr(sel), _ptr(ids), _ptr(w),
                                _ptr(stats), _ptr(workspace), workspace.numel(), _stream(stream))
        _check(st, "xshare_route")
    else:
        d_off, h_off = _offsets(req_offsets, dev)
        R = d_off.numel() - 1
        hp = None if h_off is None else ctypes.c_void_p(h_off.data_ptr())
        st = lib().xshare_select_hier(_ptr(logits), T, _ptr(d_off), hp, R, ctypes.byref(p),
                                      _ptr(sel), _ptr(ids), _ptr(w), _ptr(stats), _ptr(workspace),
                                      workspace.numel(), _stream(stream))
        _check(st, "xshare_select_hier")
    return dict(sel_mask=sel, ids=ids, w=w, stats=stats)


def select_ep(logits: torch.Tensor, groups: GroupMap, top_k: int, warmup_k0: int,
              per_group_budget: int, score_mode="topk", *, ledger=None, out=None,
              workspace=None, stream=None) -> dict:
    """Algorithms 5-6 on the GPU: dict(sel_mask, ids, w, stats, group_load)."""
    T, N = logits.shape
    dev = logits.device
    _dev(logits, torch.float32, (T, N), "logits")
    p = params(N, top_k, warmup_k0, per_group_budget, "per_group", score_mode, ledger=ledger)
    G = groups.layout.n_groups
    out = dict(out or {})
    sel = out.get("sel_mask") if out.get("sel_mask") is not None else torch.empty(N, dtype=torch.uint8, device=dev)
    ids = out.get("ids") if out.get("ids") is not None else torch.empty((T, top_k), dtype=torch.int32, device=dev)
    w = out.get("w") if out.get("w") is not None else torch.empty((T, top_k), dtype=torch.float32, device=dev)
    stats = out.get("stats") if out.get("stats") is not None else torch.empty(8, dtype=torch.int32, device=dev)
    load = out.get("group_load") if out.get("group_load") is not None else torch.empty(max(G, 1), dtype=torch.int32, device=dev)
    _dev(sel, torch.uint8, (N,), "sel_mask")
    _dev(ids, torch.int32, (T, top_k), "ids")
    _dev(w, torch.float32, (T, top_k), "w")
    _dev(stats, torch.int32, (8,), "stats")
    need = route_workspace_bytes(T, p)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    st = lib().xshare_select_ep(_ptr(logits), T, ctypes.byref(p), ctypes.byref(groups.layout),
                                _ptr(sel), _ptr(ids), _ptr(w), _ptr(load), _ptr(stats),
                                _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "xshare_select_ep")
    return dict(sel_mask=sel, ids=ids, w=w, stats=stats, group_load=load)


def route(logits: torch.Tensor, top_k: int, warmup_k0: int, budget: int, budget_mode="total",
          score_mode="topk", *, tau: float = 0.0, ledger=None, out=None, workspace=None,
          stream=None) -> dict:
    """Algorithm 2 on the GPU: returns dict(sel_mask, ids, w, stats) device tensors."""
    p = params(logits.shape[1], top_k, warmup_k0, budget, budget_mode, score_mode, 0, tau,
               ledger)
    return _route_impl(logits, p, None, out, workspace, stream)


def select_hier(logits: torch.Tensor, req_offsets, top_k: int, warmup_k0: int,
                per_request_budget: int, budget: int, budget_mode="total", score_mode="topk", *,
                tau: float = 0.0, ledger=None, out=None, workspace=None, stream=None) -> dict:
    """Algorithms 3-4 on the GPU; req_offsets as a host sequence (validated) or device tensor."""
    p = params(logits.shape[1], top_k, warmup_k0, budget, budget_mode, score_mode,
               per_request_budget, tau, ledger)
    return _route_impl(logits, p, req_offsets, out, workspace, stream)


def moe_forward(x: torch.Tensor, logits: torch.Tensor, w1: torch.Tensor, w3: torch.Tensor,
                w2: torch.Tensor, top_k: int, warmup_k0: int, budget: int, budget_mode="total",
                score_mode="topk", *, req_offsets=None, per_request_budget: int = 0,
                groups: GroupMap | None = None, tau: float = 0.0, shared=None, ledger=None,
                y=None, routing_out=True, workspace=None, stage_events=None,
                stream=None) -> dict:
    """The MoE layer: returns dict(y [T,d] bf16, and sel_mask/ids/w/stats if routing_out).

    With ``groups`` the selection is Algorithms 5-6 (``budget`` is m_g, budget_mode is
    ignored) and, if groups has a local group, y is that group's share of the layer."""
    T, d = x.shape
    N = logits.shape[1]
    f = w1.shape[1]
    dev = x.device
    _dev(x, torch.bfloat16, (T, d), "x")
    _dev(logits, torch.float32, (T, N), "logits")
    _dev(w1, torch.bfloat16, (N, f, d), "w1")
    _dev(w3, torch.bfloat16, (N, f, d), "w3")
    _dev(w2, torch.bfloat16, (N, d, f), "w2")
    if groups is not None:
        budget_mode = "per_group"
    p = params(N, top_k, warmup_k0, budget, budget_mode, score_mode, per_request_budget, tau,
               ledger)
    ep = None if groups is None else groups.layout
    sh = _shared(shared, d, f, dev)
    if y is None:
        y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    _dev(y, torch.bfloat16, (T, d), "y")
    res = {"y": y}
    if routing_out:
        res.update(sel_mask=torch.empty(N, dtype=torch.uint8, device=dev),
                   ids=torch.empty((T, top_k), dtype=torch.int32, device=dev),
                   w=torch.empty((T, top_k), dtype=torch.float32, device=dev),
                   stats=torch.empty(8, dtype=torch.int32, device=dev))
    need = moe_workspace_bytes(T, d, f, p, ep, sh)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    d_off = h_off = None
    R = 0
    if req_offsets is not None:
        d_off, h_off = _offsets(req_offsets, dev)
        R = d_off.numel() - 1
    ev = None
    if stage_events is not None:
        if len(stage_events) != N_STAGE_EVENTS:
            raise ValueError(f"stage_events needs {N_STAGE_EVENTS} events")
        ev = (ctypes.c_void_p * N_STAGE_EVENTS)(*[e.handle for e in stage_events])
    st = lib().xshare_moe_forward(
        _ptr(x), _ptr(logits), T, d, f, _ptr(w1), _ptr(w3), _ptr(w2), ctypes.byref(p),
        _ptr(d_off), None if h_off is None else ctypes.c_void_p(h_off.data_ptr()), R,
        None if ep is None else ctypes.byref(ep), None if sh is None else ctypes.byref(sh),
        _ptr(y),
        _ptr(res.get("sel_mask")), _ptr(res.get("ids")), _ptr(res.get("w")),
        _ptr(res.get("stats")), _ptr(workspace), workspace.numel(), ev, _stream(stream))
    _check(st, "xshare_moe_forward")
    return res


def moe_forward_noalloc(x: torch.Tensor, logits: torch.Tensor, w1: torch.Tensor,
                        w3: torch.Tensor, w2: torch.Tensor, top_k: int, warmup_k0: int,
                        budget: int, budget_mode="total", score_mode="topk", *, y=None,
                        out=None, stage_events=None, stream=None) -> dict:
    """xshare_moe_forward_noalloc: the layer with the library's own fixed scratch array (no
    workspace).  ``y`` and ``out`` (a dict of sel_mask / ids / w / stats tensors) are
    preallocated outputs; with them the call allocates nothing here either.  Flat selection
    (Algorithm 2) only in this binding."""
    T, d = x.shape
    N = logits.shape[1]
    f = w1.shape[1]
    dev = x.device
    _dev(x, torch.bfloat16, (T, d), "x")
    _dev(logits, torch.float32, (T, N), "logits")
    _dev(w1, torch.bfloat16, (N, f, d), "w1")
    _dev(w3, torch.bfloat16, (N, f, d), "w3")
    _dev(w2, torch.bfloat16, (N, d, f), "w2")
    p = params(N, top_k, warmup_k0, budget, budget_mode, score_mode)
    if y is None:
        y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    _dev(y, torch.bfloat16, (T, d), "y")
    res = {"y": y}
    if out is not None:
        res.update(out)
        _dev(res["sel_mask"], torch.uint8, (N,), "sel_mask")
        _dev(res["ids"], torch.int32, (T, top_k), "ids")
        _dev(res["w"], torch.float32, (T, top_k), "w")
        _dev(res["stats"], torch.int32, (8,), "stats")
    ev = None
    if stage_events is not None:
        if len(stage_events) != N_STAGE_EVENTS:
            raise ValueError(f"stage_events needs {N_STAGE_EVENTS} events")
        ev = (ctypes.c_void_p * N_STAGE_EVENTS)(*[e.handle for e in stage_events])
    st = lib().xshare_moe_forward_noalloc(
        _ptr(x), _ptr(logits), T, d, f, _ptr(w1), _ptr(w3), _ptr(w2), ctypes.byref(p), None,
        None, 0, None, None, _ptr(y), _ptr(res.get("sel_mask")), _ptr(res.get("ids")),
        _ptr(res.get("w")), _ptr(res.get("stats")), ev, _stream(stream))
    _check(st, "xshare_moe_forward_noalloc")
    return res


def moe_forward_fp8(x: torch.Tensor, logits: torch.Tensor, q1: torch.Tensor, q3: torch.Tensor,
                    q2: torch.Tensor, s1: torch.Tensor, s3: torch.Tensor, s2: torch.Tensor,
                    top_k: int, warmup_k0: int, budget: int, budget_mode="total",
                    score_mode="topk", *, req_offsets=None, per_request_budget: int = 0,
                    groups: GroupMap | None = None, tau: float = 0.0, ledger=None, y=None,
                    routing_out=True, workspace=None, stage_events=None, stream=None) -> dict:
    """The MoE layer with FP8 E4M3FN expert weights (uint8 codes) and per-row fp32 scales."""
    T, d = x.shape
    N = logits.shape[1]
    f = q1.shape[1]
    dev = x.device
    _dev(x, torch.bfloat16, (T, d), "x")
    _dev(logits, torch.float32, (T, N), "logits")
    _dev(q1, torch.uint8, (N, f, d), "w1 codes")
    _dev(q3, torch.uint8, (N, f, d), "w3 codes")
    _dev(q2, torch.uint8, (N, d, f), "w2 codes")
    _dev(s1, torch.float32, (N, f), "w1 scales")
    _dev(s3, torch.float32, (N, f), "w3 scales")
    _dev(s2, torch.float32, (N, d), "w2 scales")
    if groups is not None:
        budget_mode = "per_group"
    p = params(N, top_k, warmup_k0, budget, budget_mode, score_mode, per_request_budget, tau,
               ledger)
    ep = None if groups is None else groups.layout
    if y is None:
        y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    _dev(y, torch.bfloat16, (T, d), "y")
    res = {"y": y}
    if routing_out:
        res.update(sel_mask=torch.empty(N, dtype=torch.uint8, device=dev),
                   ids=torch.empty((T, top_k), dtype=torch.int32, device=dev),
                   w=torch.empty((T, top_k), dtype=torch.float32, device=dev),
                   stats=torch.empty(8, dtype=torch.int32, device=dev))
    need = moe_workspace_bytes(T, d, f, p, ep)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    d_off = h_off = None
    R = 0
    if req_offsets is not None:
        d_off, h_off = _offsets(req_offsets, dev)
        R = d_off.numel() - 1
    ev = None
    if stage_events is not None:
        if len(stage_events) != N_STAGE_EVENTS:
            raise ValueError(f"stage_events needs {N_STAGE_EVENTS} events")
        ev = (ctypes.c_void_p * N_STAGE_EVENTS)(*[e.handle for e in stage_events])
    st = lib().xshare_moe_forward_fp8(
        _ptr(x), _ptr(logits), T, d, f, _ptr(q1), _ptr(q3), _ptr(q2), _ptr(s1), _ptr(s3),
        _ptr(s2), ctypes.byref(p), _ptr(d_off),
        None if h_off is None else ctypes.c_void_p(h_off.data_ptr()), R,
        None if ep is None else ctypes.byref(ep), _ptr(y), _ptr(res.get("sel_mask")),
        _ptr(res.get("ids")), _ptr(res.get("w")), _ptr(res.get("stats")), _ptr(workspace),
        workspace.numel(), ev, _stream(stream))
    _check(st, "xshare_moe_forward_fp8")
    return res


def mx_granules(k: int) -> int:
    """Granules of 8 scale blocks (256 inputs) per row in the tiled MXFP4 scale layout."""
    return (k + 255) // 256


def tile_mx_scales(scales: torch.Tensor, stream=None) -> torch.Tensor:
    """xshare_mx_scales_tile: E8M0 scales [n, rows, k/32] (row-major) -> the tiled layout
    the MXFP4 GEMMs read, [n, rows/16, ceil(k/256), 16, 8] uint8 (a new tensor)."""
    n, rows, nb = scales.shape
    k = 32 * nb
    if scales.dtype != torch.uint8 or not scales.is_cuda:
        raise ValueError("scales: a uint8 device tensor [n, rows, k/32]")
    src = scales.contiguous()
    out = torch.empty((n, rows // 16, mx_granules(k), 16, 8), dtype=torch.uint8,
                      device=scales.device)
    assert out.numel() == lib().xshare_mx_scales_tiled_bytes(n, rows, k)
    _check(lib().xshare_mx_scales_tile(_ptr(src), _ptr(out), n, rows, k, _stream(stream)),
           "xshare_mx_scales_tile")
    return out


def mx_tiled(weights):
    """(q1, q3, q2, e1, e3, e2) with row-major scales -> the same with tiled scales."""
    q1, q3, q2, e1, e3, e2 = weights
    return q1, q3, q2, tile_mx_scales(e1), tile_mx_scales(e3), tile_mx_scales(e2)


def moe_forward_mxfp4(x: torch.Tensor, logits: torch.Tensor, q1: torch.Tensor, q3: torch.Tensor,
                      q2: torch.Tensor, e1: torch.Tensor, e3: torch.Tensor, e2: torch.Tensor,
                      top_k: int, warmup_k0: int, budget: int, budget_mode="total",
                      score_mode="topk", *, req_offsets=None, per_request_budget: int = 0,
                      groups: GroupMap | None = None, tau: float = 0.0, ledger=None, y=None,
                      routing_out=True, workspace=None, stage_events=None, stream=None) -> dict:
    """The MoE layer with MXFP4 expert weights: packed E2M1 codes (uint8, two per byte) and
    one E8M0 scale byte per 32 inputs of a row, in the tiled layout (tile_mx_scales)."""
    T, d = x.shape
    N = logits.shape[1]
    f = q1.shape[1]
    dev = x.device
    _dev(x, torch.bfloat16, (T, d), "x")
    _dev(logits, torch.float32, (T, N), "logits")
    _dev(q1, torch.uint8, (N, f, d // 2), "w1 codes")
    _dev(q3, torch.uint8, (N, f, d // 2), "w3 codes")
    _dev(q2, torch.uint8, (N, d, f // 2), "w2 codes")
    _dev(e1, torch.uint8, (N, f // 16, mx_granules(d), 16, 8), "w1 tiled scales")
    _dev(e3, torch.uint8, (N, f // 16, mx_granules(d), 16, 8), "w3 tiled scales")
    _dev(e2, torch.uint8, (N, d // 16, mx_granules(f), 16, 8), "w2 tiled scales")
    if groups is not None:
        budget_mode = "per_group"
    p = params(N, top_k, warmup_k0, budget, budget_mode, score_mode, per_request_budget, tau,
               ledger)
    ep = None if groups is None else groups.layout
    if y is None:
        y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    _dev(y, torch.bfloat16, (T, d), "y")
    res = {"y": y}
    if routing_out:
        res.update(sel_mask=torch.empty(N, dtype=torch.uint8, device=dev),
                   ids=torch.empty((T, top_k), dtype=torch.int32, device=dev),
                   w=torch.empty((T, top_k), dtype=torch.float32, device=dev),
                   stats=torch.empty(8, dtype=torch.int32, device=dev))
    need = moe_workspace_bytes(T, d, f, p, ep)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    d_off = h_off = None
    R = 0
    if req_offsets is not None:
        d_off, h_off = _offsets(req_offsets, dev)
        R = d_off.numel() - 1
    ev = None
    if stage_events is not None:
        if len(stage_events) != N_STAGE_EVENTS:
            raise ValueError(f"stage_events needs {N_STAGE_EVENTS} events")
        ev = (ctypes.c_void_p * N_STAGE_EVENTS)(*[e.handle for e in stage_events])
    st = lib().xshare_moe_forward_mxfp4(
        _ptr(x), _ptr(logits), T, d, f, _ptr(q1), _ptr(q3), _ptr(q2), _ptr(e1), _ptr(e3),
        _ptr(e2), ctypes.byref(p), _ptr(d_off),
        None if h_off is None else ctypes.c_void_p(h_off.data_ptr()), R,
        None if ep is None else ctypes.byref(ep), _ptr(y), _ptr(res.get("sel_mask")),
        _ptr(res.get("ids")), _ptr(res.get("w")), _ptr(res.get("stats")), _ptr(workspace),
        workspace.numel(), ev, _stream(stream))
    _check(st, "xshare_moe_forward_mxfp4")
    return res


def moe_layer(x: torch.Tensor, w_gate: torch.Tensor, w1: torch.Tensor, w3: torch.Tensor,
              w2: torch.Tensor, top_k: int, warmup_k0: int, budget: int, budget_mode="total",
              score_mode="topk", *, shared=None, req_offsets=None, per_request_budget: int = 0,
              groups: GroupMap | None = None, tau: float = 0.0, ledger=None, y=None,
              routing_out=True, logits_out=True, workspace=None, stage_events=None,
              stream=None) -> dict:
    """The whole layer from hidden states: router GEMM, selection, routed and shared experts.
    Returns dict(y, and logits/sel_mask/ids/w/stats as requested)."""
    T, d = x.shape
    N = w_gate.shape[0]
    f = w1.shape[1]
    dev = x.device
    _dev(x, torch.bfloat16, (T, d), "x")
    _dev(w_gate, torch.bfloat16, (N, d), "w_gate")
    _dev(w1, torch.bfloat16, (N, f, d), "w1")
    _dev(w3, torch.bfloat16, (N, f, d), "w3")
    _dev(w2, torch.bfloat16, (N, d, f), "w2")
    if groups is not None:
        budget_mode = "per_group"
    p = params(N, top_k, warmup_k0, budget, budget_mode, score_mode, per_request_budget, tau,
               ledger)
    ep = None if groups is None else groups.layout
    sh = _shared(shared, d, f, dev)
    if y is None:
        y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    _dev(y, torch.bfloat16, (T, d), "y")
    res = {"y": y}
    if logits_out:
        res["logits"] = torch.empty((T, N), dtype=torch.float32, device=dev)
    if routing_out:
        res.update(sel_mask=torch.empty(N, dtype=torch.uint8, device=dev),
                   ids=torch.empty((T, top_k), dtype=torch.int32, device=dev),
                   w=torch.empty((T, top_k), dtype=torch.float32, device=dev),
                   stats=torch.empty(8, dtype=torch.int32, device=dev))
    need = layer_workspace_bytes(T, d, f, p, ep, sh)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    d_off = h_off = None
    R = 0
    if req_offsets is not None:
        d_off, h_off = _offsets(req_offsets, dev)
        R = d_off.numel() - 1
    ev = None
    if stage_events is not None:
        if len(stage_events) != N_STAGE_EVENTS:
            raise ValueError(f"stage_events needs {N_STAGE_EVENTS} events")
        ev = (ctypes.c_void_p * N_STAGE_EVENTS)(*[e.handle for e in stage_events])
    st = lib().xshare_moe_layer(
        _ptr(x), _ptr(w_gate), T, d, f, _ptr(w1), _ptr(w3), _ptr(w2),
        None if sh is None else ctypes.byref(sh), ctypes.byref(p), _ptr(d_off),
        None if h_off is None else ctypes.c_void_p(h_off.data_ptr()), R,
        None if ep is None else ctypes.byref(ep), _ptr(y), _ptr(res.get("logits")),
        _ptr(res.get("sel_mask")), _ptr(res.get("ids")), _ptr(res.get("w")),
        _ptr(res.get("stats")), _ptr(workspace), workspace.numel(), ev, _stream(stream))
    _check(st, "xshare_moe_layer")
    return res


# ----------------------------------------------------------------------------- HIP events

class HipEvent:
    """A raw hipEvent_t (for the stage_events argument and kernel timing on any stream)."""
    _hip = None

    @classmethod
    def _rt(cls):
        if cls._hip is None:
            h = ctypes.CDLL("libamdhip64.so")
            h.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
            h.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            h.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            h.hipEventSynchronize.argtypes = [ctypes.c_void_p]
            h.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                              ctypes.c_void_p]
            h.hipEventDestroy.argtypes = [ctypes.c_void_p]
            cls._hip = h
        return cls._hip

    def __init__(self, timing: bool = True):
        self.handle = ctypes.c_void_p()
        rt = self._rt()
        flags = 0 if timing else 2                 # hipEventDisableTiming
        if rt.hipEventCreateWithFlags(ctypes.byref(self.handle), flags) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")
        self.handle = self.handle.value

    def record(self, stream=None):
        s = torch.cuda.current_stream() if stream is None else stream
        if self._rt().hipEventRecord(self.handle, ctypes.c_void_p(s.cuda_stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def synchronize(self):
        self._rt().hipEventSynchronize(self.handle)

    def elapsed_ms(self, later: "HipEvent") -> float:
        out = ctypes.c_float()
        if self._rt().hipEventElapsedTime(ctypes.byref(out), self.handle, later.handle) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(out.value)

    def __del__(self):
        try:
            if self.handle and self._hip is not None:
                self._hip.hipEventDestroy(self.handle)
        except Exception:
            pass


def moe_forward_v2(x: torch.Tensor, top_k: int, warmup_k0: int, budget: int,
                   budget_mode="total", score_mode="topk", *, logits=None, w_gate=None,
                   weights=(), scales=(None, None, None), weight_format="bf16",
                   req_offsets=None, per_request_budget: int = 0,
                   groups: GroupMap | None = None, tau: float = 0.0, shared=None, ledger=None,
                   y=None, routing_out=True, logits_out=False, workspace=None,
                   stage_events=None, stream=None) -> dict:
    """xshare_moe_forward_v2: the layer from one argument struct.  ``logits`` (fp32 [T, N]) or
    ``w_gate`` (bf16 [N, d], logits computed on the device); ``weights`` = (w1, w3, w2) in
    ``weight_format`` with ``scales`` for FP8 / MXFP4.  Shapes are checked by the library;
    this only marshals pointers."""
    T, d = x.shape
    w1, w3, w2 = weights
    N = (logits if logits is not None else w_gate).shape[0 if logits is None else 1]
    f = w1.shape[1]
    dev = x.device
    if groups is not None:
        budget_mode = "per_group"
    p = params(N, top_k, warmup_k0, budget, budget_mode, score_mode, per_request_budget, tau,
               ledger)
    ep = None if groups is None else groups.layout
    sh = _shared(shared, d, f, dev)
    if y is None:
        y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    res = {"y": y}
    if logits_out:
        res["logits"] = torch.empty((T, N), dtype=torch.float32, device=dev)
    if routing_out:
        res.update(sel_mask=torch.empty(N, dtype=torch.uint8, device=dev),
                   ids=torch.empty((T, top_k), dtype=torch.int32, device=dev),
                   w=torch.empty((T, top_k), dtype=torch.float32, device=dev),
                   stats=torch.empty(8, dtype=torch.int32, device=dev))
    d_off = h_off = None
    R = 0
    if req_offsets is not None:
        d_off, h_off = _offsets(req_offsets, dev)
        R = d_off.numel() - 1
    ev = None
    if stage_events is not None:
        if len(stage_events) != N_STAGE_EVENTS:
            raise ValueError(f"stage_events needs {N_STAGE_EVENTS} events")
        ev = (ctypes.c_void_p * N_STAGE_EVENTS)(*[e.handle for e in stage_events])
    s1, s3, s2 = scales
    a = LayerArgs()
    a.struct_size = ctypes.sizeof(LayerArgs)
    a.T, a.d, a.f = T, d, f
    a.x = x.data_ptr()
    a.logits = None if logits is None else logits.data_ptr()
    a.w_gate = None if w_gate is None else w_gate.data_ptr()
    a.weight_format = WEIGHTS[weight_format]
    a.w1, a.w3, a.w2 = w1.data_ptr(), w3.data_ptr(), w2.data_ptr()
    a.w1_scale = None if s1 is None else s1.data_ptr()
    a.w3_scale = None if s3 is None else s3.data_ptr()
    a.w2_scale = None if s2 is None else s2.data_ptr()
    a.params = ctypes.pointer(p)
    a.req_offsets = None if d_off is None else d_off.data_ptr()
    a.host_offsets = None if h_off is None else h_off.data_ptr()
    a.R = R
    a.ep = None if ep is None else ctypes.pointer(ep)
    a.shared = None if sh is None else ctypes.pointer(sh)
    a.y = y.data_ptr()
    for field, key in (("logits_out", "logits"), ("sel_mask", "sel_mask"), ("topk_ids", "ids"),
                       ("topk_w", "w"), ("stats", "stats")):
        setattr(a, field, None if res.get(key) is None else res[key].data_ptr())
    a.stage_events = None if ev is None else ctypes.cast(ev, ctypes.c_void_p)
    a.stream = _stream(stream).value
    need = int(lib().xshare_moe_forward_v2_workspace_bytes(ctypes.byref(a)))
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=dev)
    a.ws, a.ws_bytes = workspace.data_ptr(), workspace.numel()
    _check(lib().xshare_moe_forward_v2(ctypes.byref(a)), "xshare_moe_forward_v2")
    return res


def probe_stream_read(buf: torch.Tensor, blocks: int = 2048, mode: int = 0, sink=None,
                      stream=None):
    """Enqueues one streaming read of ``buf`` (a contiguous GPU tensor, 16-byte aligned,
    size a multiple of 16 bytes; ``mode`` as xshare_probe_stream_read); time it with
    HipEvents on the same stream."""
    if not buf.is_cuda or not buf.is_contiguous():
        raise ValueError("buf must be a contiguous GPU tensor")
    if sink is None:
        sink = torch.zeros(1, dtype=torch.int32, device=buf.device)
    _check(lib().xshare_probe_stream_read(_ptr(buf), buf.numel() * buf.element_size(),
                                          int(blocks), int(mode), _ptr(sink),
                                          _stream(stream)),
           "xshare_probe_stream_read")
    return sink


def use_timeline_library() -> None:
    """Makes this process load the profiling build (libxshare_timeline.so) instead of the
    product library; call before the first call into the library."""
    global LIB_PATH
    if _lib is not None:
        raise RuntimeError("the library is already loaded")
    LIB_PATH = TIMELINE_LIB_PATH


def block_times(clear: bool = True, stream=None) -> dict:
    """The block timeline of the last expert-GEMM launches (xshare_block_times; the profiling
    build only): uint64 arrays of 100 MHz clock stamps, "gate_up" and "down" [blocks, 2]
    (start, end) and "down_units" [blocks, 33] (start, then unit ends); 0 = not stamped.
    ``clear`` zeroes the stamps afterwards, so the next read holds only later launches."""
    dev = torch.device("cuda", torch.cuda.current_device())
    gu = torch.zeros(2 * TIME_BLOCKS, dtype=torch.int64, device=dev)
    dn = torch.zeros(2 * TIME_BLOCKS, dtype=torch.int64, device=dev)
    units = torch.zeros(TIME_SEQ_BLOCKS * TIME_SEQ_STRIDE, dtype=torch.int64, device=dev)
    _check(lib().xshare_block_times(_ptr(gu), _ptr(dn), _ptr(units), int(bool(clear)),
                                    _stream(stream)),
           "xshare_block_times")
    (stream or torch.cuda.current_stream()).synchronize()
    return {"gate_up": gu.cpu().numpy().view("uint64").reshape(-1, 2),
            "down": dn.cpu().numpy().view("uint64").reshape(-1, 2),
            "down_units": units.cpu().numpy().view("uint64").reshape(-1, TIME_SEQ_STRIDE)}
