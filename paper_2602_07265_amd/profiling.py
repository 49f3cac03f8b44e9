"""Workload driver for hardware-counter profiling of the expert GEMMs.

    rocprofv3 --pmc FETCH_SIZE -d OUT -o fetch --output-format csv -- \
        python -m paper_2602_07265_amd.profiling
    rocprofv3 --pmc WRITE_SIZE -d OUT -o write --output-format csv -- \
        python -m paper_2602_07265_amd.profiling

Runs the DeepSeek-R1-shaped layer (N=256, k=8, d=7168, f=2048, T=32 tokens, total budget
48, warm-up 1; seeded domain-centroid logits; --weights bf16, fp8 or mxfp4; --workload and
--budget for another flat workload of workloads.CONFIGS) for --calls calls over rotating
batches, then
a plain device-to-device copy of --copy-mib MiB (torch's copy kernel) --copies times.  The
copy reads and writes a known number of bytes, so it calibrates what the counters report
per byte.  Prints, per batch, the active experts and the algorithmic bytes of one gate/up
launch (weights and scales of the active experts, x, H as bf16 hi and lo) to compare with
the counters.

    python -m paper_2602_07265_amd.profiling --summarize OUT

summarises the counter CSVs that rocprofv3 wrote under OUT: per kernel of this library
(and the calibration copy) and counter, the dispatches and their mean value, as one JSON
line.

    python -m paper_2602_07265_amd.profiling --counters-json OUT_F OUT_W DRIVER_LOG

    python -m paper_2602_07265_amd.profiling --timeline [--workload W --budget M --weights F]

loads the profiling build (libxshare_timeline.so), runs the layer on --seeds batches (after
--warm calls each) and prints the expert GEMMs' block timeline of one call per batch: per
launch the blocks, their span and durations, how many run at once over time, the gap
between the launches, the persistent down blocks' unit durations and their end times per
XCD (workgroup id mod 8), as markdown and as one JSON line.

writes the traffic record of the expert GEMMs (profiles/gate_up_ds_t32_m48_counters.json,
read by bench.py) from a FETCH_SIZE run (OUT_F), a WRITE_SIZE run (OUT_W) and the
driver's own printed line (DRIVER_LOG).
"""
from __future__ import annotations

import argparse
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def summarize(out_dir: str) -> dict:
    """{kernel: {counter: {"dispatches": n, "mean": m}}} over rocprofv3's counter CSVs."""
    import csv
    import glob

    acc: dict = {}
    for path in glob.glob(os.path.join(out_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as fh:
            for row in csv.DictReader(fh):
                name = row["Kernel_Name"]
                if "xs::" not in name and "copy" not in name:
                    continue
                ours = "xs::" in name
                short = name.replace("void ", "").replace("xs::(anonymous namespace)::", "")
                short = short.split("(")[0] if ours else "copy: " + short[:80]
                per = acc.setdefault(short, {}).setdefault(row["Counter_Name"], [])
                per.append(float(row["Counter_Value"]))
    out = {}
    for k, cs in acc.items():
        out[k] = {}
        for c, v in cs.items():
            out[k][c] = {"dispatches": len(v), "mean": sum(v) / len(v)}
            if k.startswith("copy: "):
                # copies: the calibration copies are the largest dispatches of the run
                out[k][c]["largest"] = sorted(v)[-4:]
    return out


def counters_json(fetch: dict, write: dict, driver: dict) -> dict:
    """The traffic record bench.py reads: per launch of the expert GEMMs, FETCH_SIZE and
    WRITE_SIZE (KiB per dispatch, summaries of two counter runs of this driver) scaled by
    what the same counters read for the driver's device copy of known size, against the
    algorithmic bytes the driver printed; stamped with the sha256 of ffn.hip (bench.py
    ignores the record once that file changes)."""
    import hashlib

    nbytes = driver["copy_bytes"]
    copies = [k for k in fetch if k.startswith("copy: ")]
    fk = max((fetch[k]["FETCH_SIZE"]["largest"] for k in copies), key=lambda v: v[-1])
    wk = max((write[k]["WRITE_SIZE"]["largest"] for k in copies if k in write
              and "WRITE_SIZE" in write[k]), key=lambda v: v[-1])
    ff = round(nbytes / 1024 / (sum(fk) / len(fk)), 4)        # bytes read per FETCH KiB
    wf = round(nbytes / 1024 / (sum(wk) / len(wk)), 4)
    ffn = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc", "ffn.hip")

    def pick(prefixes):
        names = [k for k in fetch if any(k.startswith(p) for p in prefixes) and "true" not in k]
        return max(names, key=lambda k: fetch[k]["FETCH_SIZE"]["dispatches"])

    def rec(name, alg_key):
        fkib = fetch[name]["FETCH_SIZE"]["mean"]
        wkib = write[name]["WRITE_SIZE"]["mean"]
        alg = sum(c[alg_key] for c in driver["calls"]) / len(driver["calls"])
        return {"fetch_kib_per_dispatch": fkib, "write_kib_per_dispatch": wkib,
                "traffic_bytes_per_launch": round(fkib * 1024 * ff + wkib * 1024 * wf),
                "algorithmic_bytes_per_launch": round(alg)}

    gu = pick(("gate_up_kernel<",))
    dn = pick(("down_kernel<", "down_seq_kernel<"))
    out = {"kernel": gu, "workload": driver["workload"],
           "commands": [
               "rocprofv3 --pmc FETCH_SIZE -d OUT_F -o fetch --output-format csv -- "
               "python -u paper_2602_07265_amd/profiling.py",
               "rocprofv3 --pmc WRITE_SIZE -d OUT_W -o write --output-format csv -- "
               "python -u paper_2602_07265_amd/profiling.py",
               "python -m paper_2602_07265_amd.profiling --counters-json OUT_F OUT_W DRIVER"],
           "ffn_source_sha256": hashlib.sha256(open(ffn, "rb").read()).hexdigest(),
           "copy_calibration": {"bytes_copied": nbytes, "fetch_kib": fk, "write_kib": wk,
                                "fetch_factor": ff, "write_factor": wf}}
    out.update(rec(gu, "gate_up_bytes"))
    out["down_kernel"] = dict(name=dn, **rec(dn, "down_bytes"))
    return out


def _launch_stats(st, en, t0):
    """Span, block durations and the running-block profile of one launch (µs from t0)."""
    import numpy as np

    s, e = (st - t0) / 100.0, (en - t0) / 100.0
    dur = e - s
    edges = np.arange(s.min(), e.max() + 10.0, 10.0)
    running = [int(np.sum((s <= b + 5.0) & (e > b + 5.0))) for b in edges[:-1]]
    return {"blocks": int(len(s)), "first_start": round(float(s.min()), 1),
            "last_start": round(float(s.max()), 1), "last_end": round(float(e.max()), 1),
            "span": round(float(e.max() - s.min()), 1),
            "block_us": [round(float(v), 1) for v in (dur.mean(), dur.std(), dur.min(), dur.max())],
            "end_p50_p90": [round(float(np.percentile(e, q)), 1) for q in (50, 90)],
            "running_per_10us": running}


def timeline_of(bt):
    """Summary of one call's block stamps (xshare.block_times)."""
    import numpy as np

    gu = bt["gate_up"].astype(np.int64)
    gid = np.nonzero(gu[:, 0])[0]
    t0 = int(gu[gid, 0].min())
    out = {"gate_up": _launch_stats(gu[gid, 0], gu[gid, 1], t0)}
    dn = bt["down"].astype(np.int64)
    did = np.nonzero(dn[:, 0])[0]
    un = bt["down_units"].astype(np.int64)
    sid = np.nonzero(un[:, 0])[0]
    if len(did):
        out["down"] = _launch_stats(dn[did, 0], dn[did, 1], t0)
        down_start = int(dn[did, 0].min())
    if len(sid):
        starts = un[sid, 0]
        ends = [row[1:][row[1:] > 0] for row in un[sid]]
        last = np.array([r[-1] for r in ends])
        out["down_persistent"] = _launch_stats(starts, last, t0)
        per_unit = {}
        for st0, r in zip(starts, ends):
            prev = st0
            for j, t in enumerate(r):
                per_unit.setdefault(j, []).append((t - prev) / 100.0)
                prev = t
        out["down_persistent"]["unit_us"] = {
            j: [round(float(np.mean(v)), 1), round(float(np.std(v)), 2)] for j, v in per_unit.items()}
        xcd = sid % 8
        out["down_persistent"]["end_by_xcd"] = [
            round(float((last[xcd == x].mean() - t0) / 100.0), 1) for x in range(8) if np.any(xcd == x)]
        down_start = int(starts.min())
    if len(did) or len(sid):
        out["gap_us"] = round((down_start - int(gu[gid, 1].max())) / 100.0, 1)
    return out


def timeline(args):
    import math

    import torch

    import workloads as W
    from paper_2602_07265_amd import xshare as X

    X.use_timeline_library()
    dev = "cuda:0"
    c = W.CONFIGS[args.workload]
    T, N, k, d, f, k0, M = c["T"], c["N"], c["k"], c["d"], c["f"], c["k0"], args.budget
    if args.weights == "fp8":
        base, wb = W.expert_weights_fp8(N, d, f, 0, dev), 1.0
    elif args.weights == "mxfp4":
        base, wb = X.mx_tiled(W.expert_weights_mxfp4(N, d, f, 0, dev)), 0.5
    else:
        base, wb = W.expert_weights(N, d, f, 0, dev), 2.0
    # weight copies rotated as in bench.py, so that no call finds its experts in the
    # 256 MB Infinity Cache
    reps = max(1, min(8, math.ceil(4.0e9 / (N * 3 * d * f * wb))))
    wsets = [base] + [tuple(t.clone() for t in base) for _ in range(reps - 1)]
    p = X.params(N, k, k0, M)
    ws = torch.empty(X.moe_workspace_bytes(T, d, f, p), dtype=torch.uint8, device=dev)
    y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)

    def call(seed, r):
        h = torch.from_numpy(W.make_logits(c, seed)[0]).to(dev)
        x = W.activations(T, d, seed, dev)
        w = wsets[r % reps]
        X.moe_forward_v2(x, k, k0, M, logits=h, weights=w[:3],
                         scales=tuple(w[3:6]) if len(w) > 3 else (None,) * 3,
                         weight_format=args.weights, y=y, workspace=ws)

    runs = []
    n = 0
    for seed in range(args.seeds):
        for _ in range(args.warm):
            call(seed, n)
            n += 1
        X.block_times(clear=True)
        call(seed, n)
        n += 1
        torch.cuda.synchronize()
        runs.append(dict(seed=seed, **timeline_of(X.block_times(clear=True))))
        print(f"# {args.workload} M={M} {args.weights} seed {seed}: gate/up span "
              f"{runs[-1]['gate_up']['span']} us", file=sys.stderr, flush=True)
    print(timeline_markdown(args, runs))
    print(json.dumps({"workload": f"{args.workload} M={M} {args.weights}", "runs": runs}))


def timeline_markdown(args, runs) -> str:
    lines = [f"Block timeline, {args.workload} M={args.budget} {args.weights} "
             f"(µs from the first gate/up block's start; one call per batch)", "",
             "| seed | launch | blocks | starts | last end | span | block µs mean / sd / min / max | "
             "end p50 / p90 |", "|---|---|---|---|---|---|---|---|"]
    for r in runs:
        for name in ("gate_up", "down", "down_persistent"):
            if name not in r:
                continue
            v = r[name]
            b = v["block_us"]
            lines.append(f"| {r['seed']} | {name} | {v['blocks']} | {v['first_start']}-{v['last_start']} "
                         f"| {v['last_end']} | {v['span']} | {b[0]} / {b[1]} / {b[2]} / {b[3]} | "
                         f"{v['end_p50_p90'][0]} / {v['end_p50_p90'][1]} |")
    lines.append("")
    for r in runs:
        lines.append(f"seed {r['seed']}: gap from the last gate/up block's end to the first down "
                     f"block's start {r.get('gap_us')} µs")
        for name in ("gate_up", "down", "down_persistent"):
            if name in r:
                lines.append(f"- {name}, blocks running per 10 µs: "
                             + " ".join(str(v) for v in r[name]["running_per_10us"]))
        if "down_persistent" in r:
            u = r["down_persistent"]["unit_us"]
            lines.append("- persistent down units, µs mean (sd) by position in the block: "
                         + ", ".join(f"{j}: {v[0]} ({v[1]})" for j, v in u.items()))
            lines.append("- persistent down blocks' mean end by XCD (workgroup id mod 8): "
                         + ", ".join(str(v) for v in r["down_persistent"]["end_by_xcd"]))
    return "\n".join(lines)


def main():
    if len(sys.argv) == 3 and sys.argv[1] == "--summarize":
        print(json.dumps(summarize(sys.argv[2])))
        return
    if len(sys.argv) == 5 and sys.argv[1] == "--counters-json":
        # OUT_F, OUT_W: the two counter runs' directories; DRIVER: this driver's printed line
        drv = None
        for line in open(sys.argv[4]):
            if line.startswith("{"):
                drv = json.loads(line)
        print(json.dumps(counters_json(summarize(sys.argv[2]), summarize(sys.argv[3]), drv),
                         indent=1))
        return
    ap = argparse.ArgumentParser()
    ap.add_argument("--calls", type=int, default=8)
    ap.add_argument("--batches", type=int, default=8)
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--copies", type=int, default=4)
    ap.add_argument("--budget", type=int, default=48)
    ap.add_argument("--weights", choices=("bf16", "fp8", "mxfp4"), default="bf16")
    ap.add_argument("--workload", default="ds_t32", help="a flat workload of workloads.CONFIGS")
    ap.add_argument("--timeline", action="store_true",
                    help="the GEMMs' block timeline from the profiling build")
    ap.add_argument("--seeds", type=int, default=4, help="--timeline: batches")
    ap.add_argument("--warm", type=int, default=3, help="--timeline: calls before each")
    args = ap.parse_args()
    if args.timeline:
        timeline(args)
        return

    import torch

    import workloads as W
    from paper_2602_07265_amd import xshare as X

    dev = "cuda:0"
    c = W.CONFIGS[args.workload]
    T, N, k, d, f, k0, M = c["T"], c["N"], c["k"], c["d"], c["f"], c["k0"], args.budget
    if args.weights == "fp8":
        wset = W.expert_weights_fp8(N, d, f, 0, dev)
        wb, sb = 1.0, None              # one byte per weight, one fp32 scale per row
    elif args.weights == "mxfp4":
        wset = X.mx_tiled(W.expert_weights_mxfp4(N, d, f, 0, dev))
        wb, sb = 0.5, 1.0 / 32          # half a byte per weight, one scale byte per 32
    else:
        wset = W.expert_weights(N, d, f, 0, dev)
        wb, sb = 2.0, 0.0
    logits = [torch.from_numpy(W.make_logits(c, s)[0]).to(dev) for s in range(args.batches)]
    xs = [W.activations(T, d, s, dev) for s in range(args.batches)]
    p = X.params(N, k, k0, M)
    ws = torch.empty(X.moe_workspace_bytes(T, d, f, p), dtype=torch.uint8, device=dev)
    y = torch.empty((T, d), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()
    per_call = []
    for s in range(args.calls):
        b = s % args.batches
        r = X.moe_forward_v2(xs[b], k, k0, M, logits=logits[b], weights=wset[:3],
                             scales=tuple(wset[3:6]) if len(wset) > 3 else (None,) * 3,
                             weight_format=args.weights, y=y, workspace=ws)
        st = X.stats_dict(r["stats"])
        n = st["n_active"]
        # one matrix of each active expert: W1 or W3 ([f, d]: f rows), W2 ([d, f]: d rows)
        gu_w = n * (f * d * wb + (f * 4 if sb is None else f * d * sb))
        dn_w = n * (f * d * wb + (d * 4 if sb is None else f * d * sb))
        rows = T * k   # routed rows: x read once, H written (hi and lo) and read, Y written
        per_call.append({"call": s, "n_active": n,
                         "gate_up_bytes": round(2 * gu_w + T * d * 2 + rows * f * 4),
                         "down_bytes": round(dn_w + rows * f * 4 + rows * d * 4)})
    nbytes = args.copy_mib << 20
    src = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(args.copies):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"workload": f"{args.workload} M={M} {args.weights}", "copy_bytes": nbytes,
                      "calls": per_call}))


if __name__ == "__main__":
    main()
