"""Builds libxshare.so (gfx950) in-tree with hipcc.

    python -m paper_2602_07265_amd.build      # or build() from Python

Translation units:
* route.hip -- expert selection; -ffp-contract=off and correctly rounded fp32 division, so
               the gate arithmetic is exactly the documented sequence of fp32 operations;
* ffn.hip   -- expert GEMMs (bf16 MFMA) and the combine;
* abi.hip   -- the extern "C" entry points declared in include/xshare.h;
* probe.hip -- the streaming-read probe (measurement of the HBM read ceiling).
Every HIP compile disables packed-fp32 instruction selection.  The same sources built with
XS_BLOCK_TIMES=1 give libxshare_timeline.so, the profiling build whose expert GEMMs stamp
every block's start and end (xshare_block_times); nothing but the profiling driver loads it.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libxshare.so")
# the profiling build: the same sources with the GEMMs' block timeline (XS_BLOCK_TIMES=1)
TIMELINE_LIB = os.path.join(PKG, "libxshare_timeline.so")
ARCH = "gfx950"

COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-fPIC", "-std=c++17", "-Wall",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]
UNITS = {
    "route.hip": ["-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
                  "-fno-fast-math"],
    "ffn.hip": [],
    "abi.hip": [],
    "probe.hip": [],
}


def hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: install ROCm or put hipcc on PATH")


def build(verbose: bool = False, timeline: bool = True) -> str:
    """Compiles every translation unit and links libxshare.so (and, with `timeline`, the
    profiling build libxshare_timeline.so); returns the product library's path.  The
    compiles run in parallel."""
    jobs = [(LIB, "_build", [])]
    if timeline:
        jobs.append((TIMELINE_LIB, "_build_timeline", ["-DXS_BLOCK_TIMES=1"]))
    cc = hipcc()
    compiles, links = [], []
    for lib, objname, defines in jobs:
        objdir = os.path.join(PKG, objname)
        os.makedirs(objdir, exist_ok=True)
        objs = []
        for unit, flags in UNITS.items():
            obj = os.path.join(objdir, unit.replace(".hip", ".o"))
            compiles.append([cc, *COMMON, *flags, *defines, "-c", os.path.join(CSRC, unit),
                             "-o", obj])
            objs.append(obj)
        links.append((lib, objs))
    _run_all(compiles, verbose)
    for lib, objs in links:
        tmp = lib + ".tmp"
        _run([cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs], verbose)
        os.replace(tmp, lib)
    return LIB


def _run_all(cmds, verbose, parallel: int = min(8, os.cpu_count() or 1)):
    """Runs the commands, `parallel` at a time; raises on the first failure."""
    pending = list(cmds)
    running = []
    while pending or running:
        while pending and len(running) < parallel:
            cmd = pending.pop(0)
            if verbose:
                print(" ".join(cmd), flush=True)
            running.append((cmd, subprocess.Popen(cmd, stdout=subprocess.PIPE,
                                                  stderr=subprocess.STDOUT, text=True)))
        cmd, proc = running.pop(0)
        out, _ = proc.communicate()
        if proc.returncode != 0:
            for _, p in running:
                p.wait()
            sys.stderr.write(out)
            raise RuntimeError(f"build step failed ({proc.returncode}): {' '.join(cmd)}")
        _report(out, verbose)


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"build step failed ({res.returncode}): {' '.join(cmd)}")
    _report(res.stdout + res.stderr, verbose)


def _report(out, verbose):
    # the host pass does not know the packed-fp32 target feature; that warning is expected
    noise = [ln for ln in out.splitlines()
             if ln.strip() and "packed-fp32-ops" not in ln and "not a recognized feature" not in ln]
    if verbose and noise:
        sys.stderr.write("\n".join(noise) + "\n")


if __name__ == "__main__":
    print(build(verbose=True))
