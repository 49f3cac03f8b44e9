#!/usr/bin/env python3
"""Benchmark of the XShare MoE layer on one MI355X.

One step = the whole layer for one decode batch: router scoring, batch selection,
refinement, permutation, the SwiGLU expert GEMMs of the selected experts and the combine
(one call of xshare_moe_forward).  Workload: DeepSeek-R1-shaped routed-expert layer,
N=256 experts, k=8, d_model=7168, d_ffn=2048, T=32 tokens, total budget M=48, warm-up
k0=1; logits from 8 domain centroids (seeded), x ~ N(0,1), weights ~ N(0,0.02), bf16.
All inputs are resident in HBM before timing; steps rotate over several batches so each
step selects its own experts.  Prints one JSON line.

    python bench.py [--gpus 1] [--steps 50] [--warmup 5]

Expert parallelism (Section 5, Algorithms 5-6): ``--ep-groups G --per-group-budget m_g``
spreads the experts over G GPU groups (equal contiguous blocks) and times, batch by
batch, every group's share of the layer on this GPU (its experts only, partial y); the
layer time of a batch is the slowest share (the combining collective is not included).
Prints group loads (MaxLoad) against plain top-k routing and against the flat selection
with the same total budget m_g * G.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-layer µs/batch + HBM GB/s (N=256,k=8,B=32); experts activated/batch"
WORKLOAD_NAMES = {
    "ds_t32": "deepseek_r1_routed_moe_T{T}_N{N}_k{k}_d{d}_f{f}_M{M}_k0{k0}",
    "ds_t8": "deepseek_r1_routed_moe_T{T}_N{N}_k{k}_d{d}_f{f}_M{M}_k0{k0}",
    "ds_t16": "deepseek_r1_routed_moe_T{T}_N{N}_k{k}_d{d}_f{f}_M{M}_k0{k0}",
    "ds_iid_t8": "deepseek_r1_iid_routing_T{T}_N{N}_k{k}_d{d}_f{f}_M{M}_k0{k0}",
    "ds_iid_t32": "deepseek_r1_iid_routing_T{T}_N{N}_k{k}_d{d}_f{f}_M{M}_k0{k0}",
    "qwen": "qwen_moe_T{T}_N{N}_k{k}_d{d}_f{f}_M{M}_k0{k0}",
    "mixtral": "mixtral_T{T}_N{N}_k{k}_d{d}_f{f}_M{M}_k0{k0}",
    "tiny": "tiny_T{T}_N{N}_k{k}_d{d}_f{f}_M{M}_k0{k0}",
    "spec": "deepseek_r1_speculative_16x4_N{N}_k{k}_d{d}_f{f}_hier_M{M}_k0{k0}_mr{m_r}",
}
LOGITS_RECIPE = {
    "domains": "{Q} domain centroids N(0,1.5) + N(0,0.5)",
    "iid": "iid N(0,1)",
    "spec": "{Q} domains round-robin over requests, request offset N(0,1), token noise N(0,0.3)",
}
HBM_PEAK_GBS = 8000.0
PROFILE_COUNTERS = os.path.join(ROOT, "profiles", "gate_up_ds_t32_m48_counters.json")
FFN_SOURCE = os.path.join(ROOT, "paper_2602_07265_amd", "csrc", "ffn.hip")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--batches", type=int, default=8, help="distinct seeded batches rotated over")
    ap.add_argument("--workload", default="ds_t32",
                    help="ds_t32 (default; the headline), ds_t8, qwen, mixtral, spec")
    ap.add_argument("--budget", type=int, default=None, help="total budget M (default: workload's)")
    ap.add_argument("--tau", type=float, default=None,
                    help="Algorithm 1's threshold rule instead of a budget: |S| adapts per batch")
    ap.add_argument("--replicas", type=int, default=None,
                    help="weight copies rotated over (default: enough for >= 4 GB of weights)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-vanilla", action="store_true")
    ap.add_argument("--ep-groups", type=int, default=0,
                    help="G > 0: expert-parallel selection and per-group shares")
    ap.add_argument("--per-group-budget", type=int, default=5, help="m_g (with --ep-groups)")
    ap.add_argument("--weights", choices=("bf16", "fp8", "mxfp4"), default="bf16",
                    help="routed-expert weight format (fp8: OCP E4M3FN codes, one fp32 scale "
                         "per output row; mxfp4: E2M1 codes, one E8M0 scale per 32 inputs)")
    ap.add_argument("--full-layer", action="store_true",
                    help="the whole layer from hidden states: router GEMM, selection, routed "
                         "and shared experts (xshare_moe_layer)")
    ap.add_argument("--shared", type=int, default=None,
                    help="shared experts with --full-layer (default: 1 for DeepSeek shapes, else 0)")
    ap.add_argument("--stream-probe", action="store_true",
                    help="only the streaming-read probe: a plain coalesced read of 4 GiB, "
                         "over several grid sizes")
    ap.add_argument("--layers", type=int, default=0,
                    help="L > 0: a pass over L MoE layers sharing the global budget K")
    ap.add_argument("--global-budget", type=int, default=None,
                    help="K (with --layers; default: the workload's M times L)")
    return ap.parse_args()


def _scale_bytes(n_active, d, f, wb, gate_up_only=False):
    """Scale bytes read with the weights: FP8 (wb 1) one fp32 per output row, MXFP4
    (wb 0.5) one byte per 32 weights, bf16 none."""
    if wb == 1:
        return n_active * (2 * f + (0 if gate_up_only else d)) * 4
    if wb == 0.5:
        return n_active * (2 if gate_up_only else 3) * f * d // 32
    return 0


def gate_up_bytes(n_active, T, k, d, f, wb=2):
    """Algorithmic HBM bytes of one gate/up launch: W1, W3 of every active expert (wb bytes
    per weight, plus the format's scales), x, and H written as two bf16 arrays (hi, lo)."""
    return (n_active * 2 * f * d * wb + _scale_bytes(n_active, d, f, wb, True) + T * d * 2
            + T * k * f * 2 * 2)


def layer_bytes(n_active, T, N, d, f, wb=2):
    """Algorithmic HBM bytes of one layer call: active experts' weights (and scales), x,
    logits, y."""
    return (n_active * 3 * f * d * wb + _scale_bytes(n_active, d, f, wb) + T * d * 2
            + T * N * 4 + T * d * 2)


PROBE_BYTES = 4 << 30       # well beyond the 256 MB Infinity Cache


PROBE_MODES = {0: "grid stride, 4 loads", 1: "grid stride, 8 loads",
               2: "chunk per block, 4 loads", 3: "chunk per block, 8 loads"}


def stream_rates(X, torch, runs, blocks, mode, buf):
    """GB/s of ``runs`` timed streaming reads of ``buf`` (xshare_probe_stream_read) after two
    untimed ones, HIP events on the launch stream."""
    sink = torch.zeros(1, dtype=torch.int32, device=buf.device)
    stream = torch.cuda.current_stream()
    for _ in range(2):
        X.probe_stream_read(buf, blocks, mode, sink)
    rates = []
    for _ in range(runs):
        e0, e1 = X.HipEvent(), X.HipEvent()
        e0.record(stream)
        X.probe_stream_read(buf, blocks, mode, sink)
        e1.record(stream)
        torch.cuda.synchronize()
        rates.append(buf.numel() / (e0.elapsed_ms(e1) * 1e-3) / 1e9)
    return rates


# the probe configurations the default bench run measures (the best of a sweep on MI355X)
PROBE_CONFIGS = ((256, 1), (512, 0), (4096, 3), (8192, 2))


def stream_peak(X, np, torch, configs=PROBE_CONFIGS, runs=6):
    """The streaming-read ceiling: the best median over a few probe configurations of a
    4 GiB read.  Returns (median GB/s, best single read GB/s, (blocks, mode))."""
    buf = torch.empty(PROBE_BYTES, dtype=torch.uint8, device="cuda:0")
    best = None
    for blocks, mode in configs:
        r = stream_rates(X, torch, runs, blocks, mode, buf)
        m = float(np.median(r))
        if best is None or m > best[0]:
            best = (m, float(np.max(r)), (blocks, mode))
    del buf
    return best


def run_stream_probe(X, np, torch):
    """The probe alone: GB/s over grid sizes and access patterns (median and best of 10)."""
    buf = torch.empty(PROBE_BYTES, dtype=torch.uint8, device="cuda:0")
    out = {}
    for mode in PROBE_MODES:
        for blocks in (256, 512, 1024, 2048, 4096, 8192):
            r = stream_rates(X, torch, 10, blocks, mode, buf)
            out[f"{blocks} blocks, {PROBE_MODES[mode]}"] = {
                "median_GBs": round(float(np.median(r)), 1), "max_GBs": round(float(np.max(r)), 1)}
            print(f"[probe] mode {mode} ({PROBE_MODES[mode]}), {blocks} blocks: median "
                  f"{np.median(r):.1f} GB/s, best {np.max(r):.1f}", file=sys.stderr, flush=True)
    print(json.dumps({"metric": "streaming read of 4 GiB (HBM read ceiling)", "unit": "GB/s",
                      "bytes": PROBE_BYTES, "runs": out, "peak_GBs": HBM_PEAK_GBS}), flush=True)


def counters_traffic():
    """HBM bytes per gate/up launch from committed rocprofv3 counters, if still current."""
    try:
        prof = json.load(open(PROFILE_COUNTERS))
    except (OSError, ValueError):
        return None
    src = hashlib.sha256(open(FFN_SOURCE, "rb").read()).hexdigest()
    if prof.get("ffn_source_sha256") != src:
        return None
    return prof.get("traffic_bytes_per_launch")


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (single-GPU XShare layer); got --gpus {args.gpus}",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import workloads as W
    from paper_2602_07265_amd import xshare as X

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    X.lib()
    if args.stream_probe:
        return run_stream_probe(X, np, torch)
    if args.ep_groups > 0:
        return run_ep(args, W, X, np, torch)
    if args.full_layer:
        return run_full(args, W, X, np, torch)
    if args.layers > 0:
        return run_pass(args, W, X, np, torch)
    dev = "cuda:0"
    cfg = dict(W.CONFIGS[args.workload])
    T, N, k, d, f = cfg["T"], cfg["N"], cfg["k"], cfg["d"], cfg["f"]
    M = cfg["M"] if args.budget is None else args.budget
    k0, m_r = cfg["k0"], cfg.get("m_r", 0)
    hier = cfg["logits"] == "spec"
    nb = args.batches
    # small layers would sit in the 256 MB Infinity Cache between steps: rotate weight copies

    fp8 = args.weights == "fp8"
    mx4 = args.weights == "mxfp4"
    wb = 1 if fp8 else (0.5 if mx4 else 2)
    layer_gb = N * 3 * d * f * wb / 1e9
    reps = args.replicas or max(1, min(8, int(np.ceil(4.0 / layer_gb))))
    print(f"[bench] {args.workload}: generating layer weights ({layer_gb:.2f} GB x {reps})",
          file=sys.stderr, flush=True)
    if fp8:
        base = W.expert_weights_fp8(N, d, f, 0, dev)
    elif mx4:
        base = W.expert_weights_mxfp4(N, d, f, 0, dev)
    else:
        base = W.expert_weights(N, d, f, 0, dev)
    # the layer's own copies: MXFP4 scales in the GEMMs' tiled layout (once, at load time);
    # the CPU baseline reads the format's row-major scales
    gpu_base = X.mx_tiled(base) if mx4 else base
    wsets = [gpu_base] + [tuple(t.clone() for t in gpu_base) for _ in range(reps - 1)]
    forward = X.moe_forward_fp8 if fp8 else (X.moe_forward_mxfp4 if mx4 else X.moe_forward)
    made = [W.make_logits(cfg, s) for s in range(nb)]
    logits = [torch.from_numpy(h).to(dev) for h, _ in made]
    offs = [None if o is None else [int(v) for v in o] for _, o in made]
    xs = [W.activations(T, d, s, dev) for s in range(nb)]
    bmode = "total" if args.tau is None else "threshold"
    tau = 0.0 if args.tau is None else args.tau
    p = X.params(N, k, k0, M, bmode, threshold=tau)
    ws = torch.empty(X.moe_workspace_bytes(T, d, f, p), dtype=torch.uint8, device=dev)
    y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()

    def call(s, mode, **kw):
        b = s % nb
        wset = wsets[s % reps]
        if mode == "xshare":
            return forward(xs[b], logits[b], *wset, k, k0, M, bmode, y=y, workspace=ws,
                           req_offsets=offs[b] if hier else None, per_request_budget=m_r,
                           tau=tau, **kw)
        return forward(xs[b], logits[b], *wset, k, 0, N, "extra", y=y, workspace=ws, **kw)

    # per-batch routing statistics (deterministic per batch)
    stats = []
    for b in range(nb):
        stats.append((X.stats_dict(call(b, "xshare")["stats"]),
                      X.stats_dict(call(b, "vanilla")["stats"])))
    act = [s[0]["n_active"] for s in stats]
    act_v = [s[1]["n_active"] for s in stats]

    stream = torch.cuda.current_stream()
    nev = X.N_STAGE_EVENTS

    def run(steps, mode, timed):
        evs = [[X.HipEvent() for _ in range(nev)] for _ in range(steps)] if timed else None
        for s in range(steps):
            call(s, mode, routing_out=False, stage_events=evs[s] if timed else None)
        return evs

    print(f"[bench] warmup {args.warmup} + {args.steps} timed steps", file=sys.stderr, flush=True)
    run(args.warmup, "xshare", False)
    torch.cuda.synchronize()
    # timed region 1: the layer alone, events only around the whole region
    t0, t1 = X.HipEvent(), X.HipEvent()
    wall0 = time.perf_counter()
    t0.record(stream)
    run(args.steps, "xshare", False)
    t1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = t0.elapsed_ms(t1) / args.steps
    # timed region 2: the same steps with events at the kernel boundaries (launch stream);
    # an event pair adds a few microseconds, so region 1 gives the headline time
    evs = run(args.steps, "xshare", True)
    torch.cuda.synchronize()
    stage_ms = {name: float(np.mean([e[i].elapsed_ms(e[i + 1]) for e in evs]))
                for i, name in enumerate(X.STAGES)}
    gu_ms = np.array([e[1].elapsed_ms(e[2]) for e in evs])
    step_us = np.array([e[0].elapsed_ms(e[-1]) for e in evs]) * 1e3
    gu_bytes = np.array([gate_up_bytes(act[s % nb], T, k, d, f, wb) for s in range(args.steps)])
    lay_bytes = np.array([layer_bytes(act[s % nb], T, N, d, f, wb) for s in range(args.steps)])

    vanilla = None
    if not args.no_vanilla:
        run(args.warmup, "vanilla", False)
        torch.cuda.synchronize()
        v0, v1 = X.HipEvent(), X.HipEvent()
        v0.record(stream)
        run(args.steps, "vanilla", False)
        v1.record(stream)
        torch.cuda.synchronize()
        vanilla = v0.elapsed_ms(v1) / args.steps

    gbs = float(lay_bytes.mean()) / (ms_step * 1e-3) / 1e9
    gu_achieved = float(gu_bytes.mean()) / (float(gu_ms.mean()) * 1e-3) / 1e9
    # the HBM read ceiling on this GPU, measured in the same run (4 GiB streaming read)
    stream_gbs, stream_best, probe_cfg = stream_peak(X, np, torch)
    # the committed counter record covers the headline workload only
    traffic = counters_traffic() if (args.workload, M, T, args.tau, args.weights) == \
        ("ds_t32", 48, 32, None, "bf16") else None

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(W, xs, logits, offs if hier else None, m_r, base, args.weights, T,
                           N, k, k0, M, d, f, bmode, args.tau)

    out = {
        "metric": METRIC,
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": ("fp8-e4m3 weights, bf16 activations" if fp8 else
                  "mxfp4 (e2m1 + e8m0 per 32) weights, bf16 activations" if mx4 else "bf16"),
        "data": "synthetic",
        "config": {"workload": WORKLOAD_NAMES[args.workload].format(T=T, N=N, k=k, d=d, f=f, M=M,
                                                                     k0=k0, m_r=m_r)
                   + ("" if args.tau is None else f"_tau{args.tau:g}")
                   + ("" if args.weights == "bf16" else "_" + args.weights),
                   "weights": args.weights,
                   "tokens": T, "n_experts": N, "top_k": k, "d_model": d, "d_ffn": f,
                   "budget": None if args.tau is not None else M, "budget_mode": bmode,
                   "threshold": args.tau, "warmup_k0": k0,
                   "per_request_budget": m_r if hier else None,
                   "logits": LOGITS_RECIPE[cfg["logits"]].format(Q=cfg.get("Q")),
                   "batches_rotated": nb, "weight_replicas": reps},
        "us_per_batch": round(ms_step * 1e3, 2),
        "tokens_per_s": round(T / (ms_step * 1e-3), 1),
        "experts_activated": round(float(np.mean(act)), 2),
        "experts_selected_range": [int(min(s[0]["n_selected"] for s in stats)),
                                   int(max(s[0]["n_selected"] for s in stats))],
        "experts_vanilla": round(float(np.mean(act_v)), 2),
        "vanilla_us_per_batch": None if vanilla is None else round(vanilla * 1e3, 2),
        "speedup_vs_vanilla": None if vanilla is None else round(vanilla / ms_step, 3),
        "layer_frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
        "stages_us": {kk: round(v * 1e3, 2) for kk, v in stage_ms.items()},
        "step_us_percentiles": {f"p{q}": round(float(np.percentile(step_us, q)), 2)
                                for q in (10, 50, 90)},
        "roofline": {"kernel": "gate_up_kernel", "bound": "hbm", "achieved": round(gu_achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gu_achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "algorithmic_bytes": round(float(gu_bytes.mean())),
                     "avg_launch_us": round(float(gu_ms.mean()) * 1e3, 2),
                     "frac_of_stream": round(gu_achieved / stream_gbs, 4)},
        "stream_peak_GBs": round(stream_gbs, 1),
        "stream_peak_best_GBs": round(stream_best, 1),
        "stream_probe": f"4 GiB read, {probe_cfg[0]} blocks of 256 threads, "
                        f"{PROBE_MODES[probe_cfg[1]]}; median of 6 reads, best of "
                        f"{len(PROBE_CONFIGS)} configurations",
        "layer_frac_of_stream": round(gbs / stream_gbs, 4),
        "cpu_baseline": cpu,
        "wall_s_timed": round(wall, 3),
    }
    print(json.dumps(out), flush=True)


def run_full(args, W, X, np, torch):
    """The whole layer from hidden states (xshare_moe_layer), against plain top-k routing on
    the same path; the oracle's layer (router, selection, routed and shared experts) as the
    CPU baseline."""
    dev = "cuda:0"
    cfg = dict(W.CONFIGS[args.workload])
    if cfg["logits"] == "spec":
        raise SystemExit("--full-layer takes a flat workload")
    T, N, k, d, f, k0 = cfg["T"], cfg["N"], cfg["k"], cfg["d"], cfg["f"], cfg["k0"]
    M = cfg["M"] if args.budget is None else args.budget
    ns = args.shared if args.shared is not None else (1 if N == 256 else 0)
    Q, nb = cfg.get("Q", 8), args.batches
    print(f"[bench] {args.workload}: whole layer, {ns} shared expert(s)", file=sys.stderr,
          flush=True)
    w1, w3, w2 = W.expert_weights(N, d, f, 0, dev)
    wg = W.router_weights(N, d, 0, dev)
    sh = W.shared_weights(ns, d, f, 0, dev) if ns else None
    xs = [W.activations_domains(T, d, Q, s, dev) for s in range(nb)]
    y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    p = X.params(N, k, k0, M, "total")
    ws = torch.empty(max(X.layer_workspace_bytes(T, d, f, p, None, X._shared(sh, d, f, dev)),
                         X.layer_workspace_bytes(T, d, f, X.params(N, k, 0, N, "extra"), None,
                                                 X._shared(sh, d, f, dev))),
                     dtype=torch.uint8, device=dev)

    def call(s, vanilla=False, **kw):
        b = s % nb
        if vanilla:
            return X.moe_layer(xs[b], wg, w1, w3, w2, k, 0, N, "extra", shared=sh, y=y,
                               workspace=ws, **kw)
        return X.moe_layer(xs[b], wg, w1, w3, w2, k, k0, M, "total", shared=sh, y=y,
                           workspace=ws, **kw)

    act = [X.stats_dict(call(b)["stats"])["n_active"] for b in range(nb)]
    act_v = [X.stats_dict(call(b, True)["stats"])["n_active"] for b in range(nb)]
    stream = torch.cuda.current_stream()

    def timed(vanilla):
        for s in range(args.warmup):
            call(s, vanilla, routing_out=False, logits_out=False)
        torch.cuda.synchronize()
        e0, e1 = X.HipEvent(), X.HipEvent()
        e0.record(stream)
        for s in range(args.steps):
            call(s, vanilla, routing_out=False, logits_out=False)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_ms(e1) / args.steps

    ms = timed(False)
    evs = [[X.HipEvent() for _ in range(X.N_STAGE_EVENTS)] for _ in range(args.steps)]
    for s in range(args.steps):
        call(s, routing_out=False, logits_out=False, stage_events=evs[s])
    torch.cuda.synchronize()
    stage_ms = {name: float(np.mean([e[i].elapsed_ms(e[i + 1]) for e in evs]))
                for i, name in enumerate(("router+route", "gate_up", "down", "combine"))}
    ms_v = None if args.no_vanilla else timed(True)

    def layer_b(n_active):
        return ((n_active + ns) * 3 * f * d * 2 + N * d * 2 + T * d * 2 * 2)
    gbs = float(np.mean([layer_b(a) for a in act])) / (ms * 1e-3) / 1e9

    cpu = None
    if not args.no_cpu_baseline:
        from oracle import ffn as OF
        from oracle import route as OR
        wgb = W.bf16_bits(wg)
        shb = [] if sh is None else [tuple(W.bf16_bits(m[s]) for m in sh) for s in range(ns)]
        spent, done = 0.0, 0
        for b in range(nb):
            xb = W.bf16_bits(xs[b])
            t0 = time.perf_counter()
            h = OF.router_logits(xb, wgb).astype(np.float32)
            r = OR.route(h, k, k0, M)
            t1 = time.perf_counter()
            used = sorted(set(int(e) for e in r.ids.reshape(-1)))
            cache = {e: tuple(W.bf16_bits(m[e]) for m in (w1, w3, w2)) for e in used}
            t2 = time.perf_counter()
            OF.moe_forward(xb, r.ids, r.w, lambda e: cache[e], shared=shb)
            spent += (t1 - t0) + (time.perf_counter() - t2)
            done += 1
            if spent >= 10.0:
                break
        cpu = {"value": round(float(np.mean([layer_b(a) for a in act])) / (spent / done) / 1e9, 3),
               "unit": "GB/s", "us_per_batch": round(spent / done * 1e6, 1),
               "cores": len(os.sched_getaffinity(0)), "kind": "oracle",
               "sample": f"full oracle layer (float64 router, numpy selection, float64 SwiGLU "
                         f"of routed and shared experts) on {done} batches, {spent:.1f} s"}
    out = {
        "metric": "whole MoE layer (router + selection + routed + shared experts): us/batch "
                  "+ HBM GB/s; experts activated/batch",
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}_full_layer_shared{ns}_M{M}_k0{k0}", "tokens": T,
                   "n_experts": N, "top_k": k, "d_model": d, "d_ffn": f, "shared_experts": ns,
                   "budget": M, "budget_mode": "total", "warmup_k0": k0,
                   "activations": f"{Q} domain centroids N(0,1) + 0.5 N(0,1), bf16",
                   "router": "W_g ~ N(0, 1.5/sqrt(d)) bf16", "batches_rotated": nb},
        "us_per_batch": round(ms * 1e3, 2),
        "tokens_per_s": round(T / (ms * 1e-3), 1),
        "experts_activated": round(float(np.mean(act)), 2),
        "experts_vanilla": round(float(np.mean(act_v)), 2),
        "vanilla_us_per_batch": None if ms_v is None else round(ms_v * 1e3, 2),
        "speedup_vs_vanilla": None if ms_v is None else round(ms_v / ms, 3),
        "layer_frac_of_hbm_peak": round(gbs / HBM_PEAK_GBS, 4),
        "stages_us": {kk: round(v * 1e3, 2) for kk, v in stage_ms.items()},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def run_pass(args, W, X, np, torch):
    """The MoE layers of one forward pass sharing a global budget K (Section 3.2): L layers,
    each with its own seeded logits and the uniform budget m_l = K / L, and a device ledger
    that totals sum_l |S_l|.  One step is the whole pass; two weight sets alternate between
    layers (a layer's 48 experts already far exceed the Infinity Cache)."""
    dev = "cuda:0"
    cfg = dict(W.CONFIGS[args.workload])
    if cfg["logits"] == "spec":
        raise SystemExit("--layers takes a flat workload")
    T, N, k, d, f, k0 = cfg["T"], cfg["N"], cfg["k"], cfg["d"], cfg["f"], cfg["k0"]
    L, nb = args.layers, args.batches
    K = args.global_budget if args.global_budget is not None else cfg["M"] * L
    m = X.layer_budgets(K, L)
    print(f"[bench] {args.workload}: pass of {L} layers, K={K} (m_l {min(m)}..{max(m)})",
          file=sys.stderr, flush=True)
    wsets = [W.expert_weights(N, d, f, 0, dev)]
    wsets.append(tuple(t.clone() for t in wsets[0]))
    logits = [[torch.from_numpy(W.make_logits(cfg, 1000 * l + b)[0]).to(dev) for b in range(nb)]
              for l in range(L)]
    xs = [W.activations(T, d, b, dev) for b in range(nb)]
    y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    p = X.params(N, k, k0, max(m), "total")
    ws = torch.empty(max(X.moe_workspace_bytes(T, d, f, p),
                         X.moe_workspace_bytes(T, d, f, X.params(N, k, 0, N, "extra"))),
                     dtype=torch.uint8, device=dev)
    led = X.new_ledger(dev)

    def one_pass(b, vanilla=False, ledger=None, **kw):
        for l in range(L):
            wset = wsets[l % 2]
            if vanilla:
                X.moe_forward(xs[b], logits[l][b], *wset, k, 0, N, "extra", y=y, workspace=ws,
                              ledger=ledger, **kw)
            else:
                X.moe_forward(xs[b], logits[l][b], *wset, k, k0, max(m[l], k), "total", y=y,
                              workspace=ws, ledger=ledger, **kw)

    totals, totals_v = [], []
    for b in range(nb):
        led.zero_()
        one_pass(b, ledger=led, routing_out=False)
        totals.append(X.ledger_dict(led))
        led.zero_()
        one_pass(b, vanilla=True, ledger=led, routing_out=False)
        totals_v.append(X.ledger_dict(led))
    stream = torch.cuda.current_stream()

    def timed(vanilla):
        for s in range(args.warmup):
            one_pass(s % nb, vanilla, routing_out=False)
        torch.cuda.synchronize()
        e0, e1 = X.HipEvent(), X.HipEvent()
        e0.record(stream)
        for s in range(args.steps):
            one_pass(s % nb, vanilla, ledger=None if vanilla else led, routing_out=False)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_ms(e1) / args.steps

    ms = timed(False)
    ms_v = None if args.no_vanilla else timed(True)
    act = float(np.mean([t["active"] for t in totals]))
    gbs = (act * 3 * f * d * 2 + L * (T * d * 4 + T * N * 4)) / (ms * 1e-3) / 1e9
    out = {
        "metric": "MoE layers of a forward pass under a global expert budget K: us per pass "
                  "+ HBM GB/s; sum of |S_l| against K",
        "value": round(ms * 1e3, 1),
        "unit": "us",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}_pass_L{L}_K{K}_k0{k0}", "layers": L,
                   "global_budget": K, "layer_budgets": [min(m), max(m)], "tokens": T,
                   "n_experts": N, "top_k": k, "d_model": d, "d_ffn": f, "warmup_k0": k0,
                   "logits": "per layer: " + LOGITS_RECIPE[cfg["logits"]].format(Q=cfg.get("Q")),
                   "batches_rotated": nb, "weight_sets": 2},
        "us_per_layer": round(ms * 1e3 / L, 2),
        "hbm_gbs": round(gbs, 1),
        "selected_per_pass": round(float(np.mean([t["selected"] for t in totals])), 2),
        "selected_per_pass_max": int(max(t["selected"] for t in totals)),
        "active_per_pass": round(act, 2),
        "vanilla_active_per_pass": round(float(np.mean([t["active"] for t in totals_v])), 2),
        "vanilla_us_per_pass": None if ms_v is None else round(ms_v * 1e3, 1),
        "speedup_vs_vanilla": None if ms_v is None else round(ms_v / ms, 3),
        "ledger_layers": int(totals[0]["layers"]),
        "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


def run_ep(args, W, X, np, torch):
    """Expert-parallel layer: selection with GPU groups, then each group's share timed."""
    dev = "cuda:0"
    cfg = dict(W.CONFIGS[args.workload])
    if cfg["logits"] == "spec":
        raise SystemExit("--ep-groups takes a flat workload")
    T, N, k, d, f, k0 = cfg["T"], cfg["N"], cfg["k"], cfg["d"], cfg["f"], cfg["k0"]
    G, m_g, nb = args.ep_groups, args.per_group_budget, args.batches
    print(f"[bench] {args.workload}: expert parallel G={G} m_g={m_g}", file=sys.stderr, flush=True)
    w1, w3, w2 = W.expert_weights(N, d, f, 0, dev)
    logits = [torch.from_numpy(W.make_logits(cfg, s)[0]).to(dev) for s in range(nb)]
    xs = [W.activations(T, d, s, dev) for s in range(nb)]
    groups = X.GroupMap(G, None, device=dev)
    gid = torch.arange(N, device=dev) // (N // G)
    shares = [groups.with_local(g) for g in range(G)]
    y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    p_ep = X.params(N, k, k0, m_g, "per_group")
    p_van = X.params(N, k, 0, N, "per_group")
    ws = torch.empty(max(X.moe_workspace_bytes(T, d, f, p, s.layout) for p in (p_ep, p_van)
                         for s in shares), dtype=torch.uint8, device=dev)

    def loads(mask):
        return torch.bincount(gid[mask.bool()], minlength=G).cpu().tolist()

    # active experts of every (batch, group) share: algorithmic bytes of the share
    act = np.array([[X.stats_dict(X.moe_forward(xs[b], logits[b], w1, w3, w2, k, k0, m_g,
                                                groups=shares[g], y=y, workspace=ws)["stats"])
                     ["n_active"] for g in range(G)] for b in range(nb)])
    rows = []
    for b in range(nb):
        ep = X.select_ep(logits[b], groups, k, k0, m_g)
        flat = X.route(logits[b], k, k0, max(m_g * G, k), "total")
        van = X.route(logits[b], k, 0, N, "extra")
        rows.append(dict(ep=loads(ep["sel_mask"]), flat=loads(flat["sel_mask"]),
                         van=loads(van["sel_mask"])))
    torch.cuda.synchronize()

    def timed(kk0, mg):
        """[batch][group] microseconds of the share calls, chained events on one stream."""
        stream = torch.cuda.current_stream()
        for s in range(args.warmup):
            X.moe_forward(xs[s % nb], logits[s % nb], w1, w3, w2, k, kk0, mg, groups=shares[s % G],
                          y=y, routing_out=False, workspace=ws)
        reps = max(1, args.steps // nb)
        evs = [X.HipEvent() for _ in range(reps * nb * G + 1)]
        evs[0].record(stream)
        i = 0
        for _ in range(reps):
            for b in range(nb):
                for g in range(G):
                    X.moe_forward(xs[b], logits[b], w1, w3, w2, k, kk0, mg, groups=shares[g], y=y,
                                  routing_out=False, workspace=ws)
                    i += 1
                    evs[i].record(stream)
        torch.cuda.synchronize()
        t = np.array([evs[j].elapsed_ms(evs[j + 1]) for j in range(len(evs) - 1)]) * 1e3
        return t.reshape(reps, nb, G).mean(0)

    t_ep = timed(k0, m_g)
    t_van = None if args.no_vanilla else timed(0, N)
    layer = float(t_ep.max(1).mean())
    slow = t_ep.argmax(1)
    share_bytes = np.array([layer_bytes(act[b, slow[b]], T, N, d, f) for b in range(nb)])
    achieved = float(np.mean(share_bytes / (t_ep[np.arange(nb), slow] * 1e-6))) / 1e9
    mean = lambda key, fn: round(float(np.mean([fn(r[key]) for r in rows])), 2)  # noqa: E731
    out = {
        "metric": f"EP MoE layer: us/batch on the slowest of G={G} GPU groups (its share of "
                  f"the layer; collective excluded) + experts activated and MaxLoad",
        "value": round(layer, 2),
        "unit": "us",
        "n_gpus": 1,
        "steps": max(1, args.steps // nb) * nb,
        "warmup": args.warmup,
        "ms_per_step": round(layer / 1e3, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{args.workload}_ep_G{G}_mg{m_g}_k0{k0}", "tokens": T,
                   "n_experts": N, "top_k": k, "d_model": d, "d_ffn": f, "groups": G,
                   "per_group_budget": m_g, "warmup_k0": k0, "placement": "contiguous blocks",
                   "logits": LOGITS_RECIPE[cfg["logits"]].format(Q=cfg.get("Q")),
                   "batches_rotated": nb},
        "experts_activated": mean("ep", sum),
        "max_group_load": mean("ep", max),
        "vanilla_experts": mean("van", sum),
        "vanilla_max_group_load": mean("van", max),
        "flat_xshare_same_total_max_group_load": mean("flat", max),
        "flat_xshare_same_total_experts": mean("flat", sum),
        "share_us_mean": round(float(t_ep.mean()), 2),
        "slowest_share_active_experts": round(float(np.mean(act[np.arange(nb), slow])), 2),
        "roofline": {"kernel": "slowest group's layer share", "bound": "hbm",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": None,
                     "algorithmic_bytes": round(float(share_bytes.mean()))},
        "vanilla_ep_us_per_batch": None if t_van is None else round(float(t_van.max(1).mean()), 2),
        "speedup_vs_vanilla_ep": None if t_van is None else
        round(float(t_van.max(1).mean()) / layer, 3),
    }
    print(json.dumps(out), flush=True)


def cpu_baseline(W, xs, logits, offs, m_r, weights, fmt, T, N, k, k0, M, d, f, mode="total",
                 tau=None, budget_s=10.0):
    """The oracle on the host cores: routing plus the float64 SwiGLU layer of whole batches,
    over as many of the rotated batches as fit in about budget_s seconds (at least one)."""
    import numpy as np

    from oracle import ffn as OF
    from oracle import route as OR
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    print("[bench] cpu baseline: full oracle on rotated batches", file=sys.stderr, flush=True)
    spent, spent_route, done, active = 0.0, 0.0, 0, []
    wall0 = time.perf_counter()
    for b in range(len(xs)):
        if done and time.perf_counter() - wall0 > 100.0:     # weight decoding is slow
            break
        h = logits[b].cpu().numpy()
        xb = W.bf16_bits(xs[b])
        t0 = time.perf_counter()
        r = OR.route(h, k, k0, M, mode, tau=tau) if offs is None else \
            OR.select_hier(h, offs[b], k, k0, m_r, M, mode, tau=tau)
        t_route = time.perf_counter() - t0
        used = sorted(set(int(e) for e in r.ids.reshape(-1)))
        if fmt != "bf16":                                                   # not timed
            q1, q3, q2, s1, s3, s2 = weights
            dec = OF.dequant_rows if fmt == "fp8" else OF.dequant_mx
            cache = {}
            for n_done, e in enumerate(used):
                cache[e] = tuple(dec(q[e].cpu().numpy(), sc[e].cpu().numpy())
                                 for q, sc in ((q1, s1), (q3, s3), (q2, s2)))
                if n_done % 8 == 7:
                    print(f"[bench] cpu baseline: batch {b}, {n_done + 1}/{len(used)} experts "
                          "decoded", file=sys.stderr, flush=True)
        else:
            cache = {e: tuple(W.bf16_bits(m[e]) for m in weights) for e in used}
        t0 = time.perf_counter()
        OF.moe_forward(xb, r.ids, r.w, lambda e: cache[e])
        spent += t_route + time.perf_counter() - t0
        spent_route += t_route
        done += 1
        print(f"[bench] cpu baseline: batch {b} done, {spent:.1f} s timed so far", file=sys.stderr,
              flush=True)
        active.append(r.n_active)
        del cache
        if spent >= budget_s:
            break
    t_batch = spent / done
    wb = {"bf16": 2, "fp8": 1, "mxfp4": 0.5}[fmt]
    bytes_batch = float(np.mean([layer_bytes(a, T, N, d, f, wb) for a in active]))
    return {"value": round(bytes_batch / t_batch / 1e9, 3), "unit": "GB/s",
            "us_per_batch": round(t_batch * 1e6, 1), "cores": int(cores), "kind": "oracle",
            "route_us_per_batch": round(spent_route / done * 1e6, 1),
            "sample": f"full oracle (numpy routing, float64 SwiGLU of all {T} tokens over their "
                      f"{np.mean(active):.0f} active experts) on {done} of the rotated batches, "
                      f"{spent:.1f} s total; BLAS threads = cores, weight conversion "
                      f"{'' if fmt == 'bf16' else '(' + fmt + ' decode) '}single-threaded and "
                      "not timed"}


if __name__ == "__main__":
    main()
