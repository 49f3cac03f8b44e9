"""Selection parity on the GPU: the HIP path must equal the oracle bit for bit.

Compared on every case: the selected-set mask, each token's routed experts (rank order),
their fp32 gates (bitwise), and the statistics |S|, |active|, |U|, |S_0|, budget_eff.
"""
import numpy as np
import pytest

import workloads as W
from helpers import assert_route_equal, gpu_route, oracle_route, say, score_order_case

pytestmark = pytest.mark.gpu

F32 = np.float32


def _case(h, k, k0, M, mode="total", score="topk", offsets=None, m_r=0, label=""):
    say(f"route case {label} T={h.shape[0]} N={h.shape[1]} k={k} k0={k0} M={M} {mode} {score}"
        f"{'' if offsets is None else f' hier R={len(offsets) - 1} m_r={m_r}'}")
    got = gpu_route(h, k, k0, M, mode, score, offsets, m_r)
    ref = oracle_route(h, k, k0, M, mode, score, offsets, m_r)
    assert_route_equal(got, ref, label)
    return got


@pytest.mark.parametrize("cfg", ["tiny", "mixtral", "qwen", "ds_t8", "ds_t32", "ds_iid_t32"])
def test_route_parity_workloads(cfg):
    c = W.CONFIGS[cfg]
    for seed in range(8):
        h, _ = W.make_logits(c, seed)
        for k0 in sorted({0, 1, min(2, c["k"])}):
            for M in c["M_sweep"]:
                _case(h, c["k"], k0, M, "total", "topk", label=f"{cfg}/s{seed}")
            for m in (0, 8):
                _case(h, c["k"], k0, m, "extra", "topk", label=f"{cfg}/s{seed}")


@pytest.mark.parametrize("cfg", ["tiny", "qwen", "ds_t32"])
def test_route_parity_dense_scores(cfg):
    c = W.CONFIGS[cfg]
    for seed in range(3):
        h, _ = W.make_logits(c, seed)
        for k0 in (0, 1):
            _case(h, c["k"], k0, c["M"], "total", "dense", label=f"{cfg}/dense/s{seed}")
            _case(h, c["k"], k0, 4, "extra", "dense", label=f"{cfg}/dense/s{seed}")


def test_route_vanilla_mode_equals_plain_topk():
    c = W.CONFIGS["ds_t32"]
    h, _ = W.make_logits(c, 0)
    got = _case(h, 8, 0, 256, "extra", label="vanilla")
    assert got["stats"][0] == got["stats"][2]        # |S| == |U|


def test_route_adversarial_ties_and_signed_zero():
    rng = np.random.default_rng(0)
    for it in range(12):
        T, N = int(rng.integers(1, 70)), int(rng.choice([8, 16, 33, 64, 100, 256]))
        k = int(rng.integers(1, min(N, 9) + 1))
        h = (np.round(rng.standard_normal((T, N)) * 3) / 4).astype(F32)
        h[rng.random(h.shape) < 0.15] = F32(-0.0)
        h[rng.random(h.shape) < 0.15] = F32(0.0)
        M = int(rng.integers(k, N + 1))
        _case(h, k, int(rng.integers(0, k + 1)), M, "total", label=f"ties{it}")
        _case(h, k, int(rng.integers(0, k + 1)), int(rng.integers(0, 6)), "extra",
              label=f"ties{it}")
    h = np.zeros((16, 64), F32)                       # every logit equal
    _case(h, 4, 1, 8, label="all-equal")
    h = np.full((16, 64), -1.0e4, F32)                # gaps far beyond the exp underflow
    h[np.arange(16), np.arange(16) * 3] = 0.0
    h[np.arange(16), np.arange(16) * 3 + 1] = -50.0
    _case(h, 4, 1, 20, label="underflow")
    _case(h, 4, 0, 6, "extra", label="underflow")


def test_route_ties_four_tokens_per_wave():
    """Batches of 33-128 tokens over at most 128 experts rank four tokens per wave (one per
    16-lane row), with up to 16 ranks a row: quarter-step ties, signed zeros, rows with fewer
    keys than k, a batch just past the register cache (129 tokens), bit-exact parity."""
    rng = np.random.default_rng(7)
    shapes = [(33, 16, 4), (40, 64, 8), (64, 128, 8), (100, 50, 16), (128, 128, 12),
              (64, 8, 8), (48, 100, 9), (129, 128, 8), (96, 12, 16)]
    for it, (T, N, k) in enumerate(shapes):
        h = (np.round(rng.standard_normal((T, N)) * 3) / 4).astype(F32)
        h[rng.random(h.shape) < 0.15] = F32(-0.0)
        h[rng.random(h.shape) < 0.15] = F32(0.0)
        k = min(k, N)
        M = int(rng.integers(k, N + 1))
        _case(h, k, int(rng.integers(0, k + 1)), M, "total", label=f"rows{it}")
        _case(h, k, int(rng.integers(0, k + 1)), int(rng.integers(0, 6)), "extra",
              label=f"rows{it}")
    c = W.CONFIGS["qwen"]
    for seed in range(4):
        h, _ = W.make_logits(c, seed)
        for M in (8, 32, 64):
            _case(h, c["k"], 1, M, "total", label=f"qwen/s{seed}")


def test_route_score_sum_order_decides_the_set():
    """The case where the ascending token order of the score sums decides which of two
    experts takes the last slot (the oracle's pin derives it by hand): bit-exact parity."""
    h, k, M, A, B = score_order_case()
    _case(h, k, 0, M, label="score order")
    got = gpu_route(h, k, 0, M)
    assert got["sel_mask"][A] == 1 and got["sel_mask"][B] == 0


def test_route_shapes_edges():
    rng = np.random.default_rng(1)
    for T, N, k, M in [(0, 16, 2, 8), (1, 256, 8, 8), (37, 200, 6, 30), (5, 1024, 32, 100),
                       (64, 8, 2, 5), (3, 1, 1, 1), (1024, 256, 8, 96), (2048, 64, 4, 16),
                       (4096, 16, 2, 8)]:
        h = rng.standard_normal((T, N)).astype(F32)
        _case(h, k, min(1, k), M, "total", label=f"edge T{T} N{N}")
        _case(h, k, min(2, k), 3, "extra", label=f"edge T{T} N{N}")


def test_hier_parity_spec_workload():
    c = W.CONFIGS["spec"]
    for seed in range(6):
        h, off = W.make_logits(c, seed)
        for k0 in (0, 1, 2):
            for m_r in (0, 4, 5):
                _case(h, 8, k0, 64, "total", offsets=off, m_r=m_r, label=f"spec/s{seed}")
                _case(h, 8, k0, 40, "total", offsets=off, m_r=m_r, label=f"spec/s{seed}")
                _case(h, 8, k0, 0, "extra", offsets=off, m_r=m_r, label=f"spec/s{seed}")
        _case(h, 8, 1, 64, "total", "dense", offsets=off, m_r=4, label=f"spec/dense/s{seed}")


def test_hier_parity_ragged_groupings():
    rng = np.random.default_rng(2)
    for it in range(16):
        T = int(rng.integers(1, 80))
        R = int(rng.integers(1, T + 1))
        cuts = np.sort(rng.choice(np.arange(1, T), R - 1, replace=False)) if R > 1 else []
        off = [0, *[int(c) for c in cuts], T]
        N = int(rng.choice([16, 64, 128, 256]))
        k = int(rng.integers(1, 9))
        h = rng.standard_normal((T, N)).astype(F32)
        if it % 3 == 0:
            h = (np.round(h * 2) / 4).astype(F32)
        _case(h, k, int(rng.integers(0, k + 1)), max(k, int(rng.integers(1, N + 1))), "total",
              offsets=off, m_r=int(rng.integers(0, 6)), label=f"ragged{it}")
        _case(h, k, int(rng.integers(0, k + 1)), int(rng.integers(0, 5)), "extra",
              offsets=off, m_r=int(rng.integers(0, 6)), label=f"ragged{it}")


def test_hier_invalid_device_offsets_yield_empty_selection():
    h = W.logits_iid(8, 16, 0)
    say("route case invalid device offsets")
    got = gpu_route(h, 2, 1, 8, offsets=[0, 5, 3, 8], m_r=2, device_offsets_only=True)
    assert got["stats"][0] == -1 and got["sel_mask"].sum() == 0
    assert np.all(got["ids"] == -1)


def _threshold_case(h, k, k0, tau, score="topk", offsets=None, m_r=0, label=""):
    t = float(np.float32(tau))
    say(f"route case {label} T={h.shape[0]} N={h.shape[1]} k={k} k0={k0} tau={t} {score}"
        f"{'' if offsets is None else f' hier m_r={m_r}'}")
    got = gpu_route(h, k, k0, 0, "threshold", score, offsets, m_r, tau=t)
    ref = oracle_route(h, k, k0, 0, "threshold", score, offsets, m_r, tau=t)
    assert_route_equal(got, ref, label)


def test_route_threshold_rule():
    """Algorithm 1's threshold: the stopping size depends on fp32 sums in the stated order;
    tau = 1 makes rank-order and index-order sums meet in their last bits."""
    for cfg in ("tiny", "qwen", "ds_t8", "ds_t32", "ds_iid_t32", "mixtral"):
        c = W.CONFIGS[cfg]
        for seed in range(4):
            h, _ = W.make_logits(c, seed)
            for k0 in (0, 1, 2):
                for tau in (0.0, 0.3, 0.6, 0.9, 0.99, 1.0, 1.5):
                    _threshold_case(h, c["k"], k0, tau, label=f"{cfg}/s{seed}")
            _threshold_case(h, c["k"], 1, 0.7, "dense", label=f"{cfg}/dense/s{seed}")
            _threshold_case(h, c["k"], 1, 1.0, "dense", label=f"{cfg}/dense/s{seed}")
    rng = np.random.default_rng(5)
    for it in range(10):                               # ties and tiny gates
        T, N = int(rng.integers(1, 70)), int(rng.choice([16, 64, 256, 1024]))
        h = (np.round(rng.standard_normal((T, N)) * 3) / 4).astype(F32)
        h[rng.random(h.shape) < 0.1] = F32(-40.0)
        _threshold_case(h, int(rng.integers(1, 9)), 1, float(rng.uniform(0.5, 1.0)),
                        label=f"ties{it}")
    c = W.CONFIGS["spec"]
    for seed in range(3):
        h, off = W.make_logits(c, seed)
        for tau in (0.5, 0.9, 1.0):
            _threshold_case(h, 8, 1, tau, offsets=off, m_r=4, label=f"spec/s{seed}")


def test_route_is_deterministic():
    c = W.CONFIGS["spec"]
    h, off = W.make_logits(c, 9)
    say("route determinism")
    a = gpu_route(h, 8, 1, 64, offsets=off, m_r=4)
    for _ in range(3):
        b = gpu_route(h, 8, 1, 64, offsets=off, m_r=4)
        for key in a:
            assert np.array_equal(a[key], b[key])
