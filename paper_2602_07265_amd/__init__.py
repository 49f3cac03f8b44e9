"""XShare batch-level MoE layer (arXiv 2602.07265) for AMD Instinct MI355X (gfx950).

The computation lives in hand-written HIP kernels behind the C ABI of include/xshare.h
(libxshare.so, built in-tree by ``paper_2602_07265_amd.build``); ``xshare`` is the Python
binding with the same entry points.
"""
from .xshare import (GroupMap, HipEvent, XShareError, layer_budgets,  # noqa: F401
                     layer_workspace_bytes, ledger_dict, lib, moe_forward, moe_forward_fp8,
                     moe_forward_mxfp4, moe_layer, moe_workspace_bytes, new_ledger, params,
                     route, route_workspace_bytes, router_logits, select_ep, select_hier,
                     stats_dict, status_string, version)
