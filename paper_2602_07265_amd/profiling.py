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


def main():
    if len(sys.argv) == 3 and sys.argv[1] == "--summarize":
        print(json.dumps(summarize(sys.argv[2])))
        return
    ap = argparse.ArgumentParser()
    ap.add_argument("--calls", type=int, default=8)
    ap.add_argument("--batches", type=int, default=8)
    ap.add_argument("--copy-mib", type=int, default=1024)
    ap.add_argument("--copies", type=int, default=4)
    ap.add_argument("--budget", type=int, default=48)
    ap.add_argument("--weights", choices=("bf16", "fp8", "mxfp4"), default="bf16")
    ap.add_argument("--workload", default="ds_t32", help="a flat workload of workloads.CONFIGS")
    args = ap.parse_args()

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
