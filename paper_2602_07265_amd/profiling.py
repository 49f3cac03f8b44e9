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
