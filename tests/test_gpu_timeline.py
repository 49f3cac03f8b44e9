"""The profiling build's block timeline on the GPU.

The profiling driver loads libxshare_timeline.so (the same sources with XS_BLOCK_TIMES=1),
so it runs in a child process of its own: this process has loaded the product library.
Every block of the gate/up and down launches must be stamped, and start before it ends;
the persistent down grid of the DeepSeek T=32 layer must stamp every unit.
"""
import json
import os
import subprocess
import sys

import pytest

from helpers import say

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _timeline(*args):
    cmd = [sys.executable, "-u", "-m", "paper_2602_07265_amd.profiling", "--timeline",
           "--seeds", "1", "--warm", "1", *args]
    say("timeline:", " ".join(args))
    r = subprocess.run(cmd, cwd=ROOT, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    return json.loads([ln for ln in r.stdout.splitlines() if ln.startswith("{")][-1])["runs"][0]


def _sane(stats):
    mean, sd, lo, hi = stats["block_us"]
    assert stats["blocks"] > 0 and 0 < lo <= mean <= hi and stats["span"] >= hi
    assert stats["first_start"] >= 0 and stats["last_end"] > stats["first_start"]


def test_block_timeline_grid_launches():
    """Qwen-MoE shape, total budget 32: 12 one-tile gate/up blocks and 16 down blocks of
    128 rows per active expert."""
    run = _timeline("--workload", "qwen", "--budget", "32")
    _sane(run["gate_up"])
    _sane(run["down"])
    assert run["gate_up"]["blocks"] == 12 * 32 and run["down"]["blocks"] == 16 * 32
    assert run["gap_us"] > 0


def test_block_timeline_persistent_down():
    """DeepSeek T=32, total budget 48: 768 two-tile gate/up blocks, then the persistent down
    grid of 256 blocks with three units each."""
    run = _timeline("--workload", "ds_t32", "--budget", "48")
    _sane(run["gate_up"])
    _sane(run["down_persistent"])
    assert run["gate_up"]["blocks"] == 768
    assert run["down_persistent"]["blocks"] == 256
    assert sorted(run["down_persistent"]["unit_us"]) == ["0", "1", "2"]
