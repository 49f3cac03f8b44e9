"""Expert-parallel selection and per-group layer shares on the GPU (Section 5,
Algorithms 5-6), against the oracle: selection bit-exact (set, ids, weights, group loads,
statistics); each group's share of y within 2e-2 * RMS of the float64 oracle share."""
import numpy as np
import pytest
import torch

import workloads as W
from helpers import (DEV, OracleOutputs, assert_ffn_close, assert_route_equal, bf16_weights_of,
                     make_layer, say)
from oracle import ffn as OF
from oracle import route as OR

pytestmark = pytest.mark.gpu



def _groups(N, G, kind, seed):
    if kind == "contiguous":
        return None, OR.contiguous_groups(N, G)
    rng = np.random.default_rng(seed)
    gr = [int(v) for v in rng.integers(0, G, N)]
    return gr, gr


def _check_ep(h, k, k0, m_g, G, kind="contiguous", score="topk", seed=0, device_map_only=False,
              label=""):
    from paper_2602_07265_amd import xshare as X
    T, N = h.shape
    given, gr = _groups(N, G, kind, seed)
    if given is not None and device_map_only:
        given = torch.tensor(given, dtype=torch.int32, device=DEV)
    say(f"ep case {label} T={T} N={N} k={k} k0={k0} m_g={m_g} G={G} {kind} {score}")
    gm = X.GroupMap(G, given, device=DEV)
    res = X.select_ep(torch.from_numpy(np.ascontiguousarray(h)).to(DEV), gm, k, k0, m_g, score)
    torch.cuda.synchronize()
    got = {key: v.cpu().numpy() for key, v in res.items()}
    ref = OR.select_ep(h, k, k0, m_g, gr, G, score)
    assert_route_equal(got, ref, label)
    assert list(got["group_load"][:G]) == ref.extra["loads"], label
    assert got["stats"][6] == ref.extra["max_load"], label
    assert got["stats"][4] == ref.n_warmup, label
    return ref


def test_ep_tiny_sweep():
    for seed in range(6):
        h, _ = W.make_logits(W.CONFIGS["tiny"], seed)
        for G in (1, 2, 4, 8, 16):
            for k0, m_g in [(1, 2), (0, 1), (2, 3), (1, 0), (0, 0)]:
                _check_ep(h, 2, k0, m_g, G, seed=seed, label=f"tiny/s{seed}")


def test_ep_scattered_groups_and_dense_scores():
    for seed in range(4):
        h = W.logits_domains(24, 64, 4, seed)
        for G, m_g in [(3, 2), (5, 4), (8, 1)]:
            _check_ep(h, 4, 1, m_g, G, "scattered", seed=seed, label=f"scattered/s{seed}")
            _check_ep(h, 4, 1, m_g, G, "scattered", seed=seed, device_map_only=True,
                      label=f"device-map/s{seed}")
        _check_ep(h, 4, 1, 2, 4, score="dense", label=f"dense/s{seed}")


def test_ep_deepseek_shapes():
    # Table 2's setting: DeepSeek-R1 experts over 8 GPUs, (k0, m_g) = (1, 5); batches of 8
    # and 16 tokens, plus the 32-token batch and the 64-token speculative batch.
    for T in (8, 16, 32, 64):
        for seed in range(3):
            h = W.logits_domains(T, 256, 8, seed)
            for m_g in (3, 5, 8):
                _check_ep(h, 8, 1, m_g, 8, seed=seed, label=f"ds T{T} s{seed}")
    h = W.logits_domains(100, 256, 8, 0)                    # beyond the bitmask path
    _check_ep(h, 8, 1, 5, 8, label="ds T100")
    _check_ep(W.logits_domains(64, 128, 8, 1), 8, 1, 4, 16, label="qwen G16")


def test_ep_degenerate_cases():
    h = W.logits_domains(12, 32, 3, 5)
    ref = _check_ep(h, 4, 0, 1, 32, label="one expert per group")      # plain top-k
    assert np.array_equal(ref.ids, ref.vanilla_ids)
    _check_ep(h, 4, 0, 0, 4, label="m_g 0: top-up to k")
    _check_ep(h, 4, 4, 1, 4, label="k0 = k")
    _check_ep(h[:1], 4, 1, 2, 4, label="one token")
    _check_ep(h, 4, 1, 1000, 4, label="budget above N")


def test_ep_empty_batch_and_bad_device_map():
    from paper_2602_07265_amd import xshare as X
    say("ep case empty batch")
    gm = X.GroupMap(4, None, device=DEV)
    res = X.select_ep(torch.empty((0, 16), device=DEV), gm, 2, 1, 2)
    torch.cuda.synchronize()
    assert int(res["sel_mask"].sum()) == 0 and int(res["stats"][0]) == 0
    say("ep case group id out of range on the device")
    bad = torch.tensor([0, 1, 2, 3] * 3 + [0, 1, 2, 7], dtype=torch.int32, device=DEV)
    gm = X.GroupMap(4, bad, device=DEV)
    h = torch.from_numpy(W.logits_domains(8, 16, 2, 0)).to(DEV)
    res = X.select_ep(h, gm, 2, 1, 2)
    torch.cuda.synchronize()
    assert int(res["stats"][0]) == -1
    assert int(res["sel_mask"].sum()) == 0
    assert bool((res["ids"] == -1).all()) and bool((res["w"] == 0).all())
    assert int(res["group_load"].sum()) == 0


def _share(cfg, seed, G, m_g, local, kind="contiguous", rows=None, layer=None, label=""):
    from paper_2602_07265_amd import xshare as X
    h, _, x, w1, w3, w2 = layer if layer is not None else make_layer(cfg, seed)
    N, k = cfg["N"], cfg["k"]
    given, gr = _groups(N, G, kind, seed)
    say(f"ep share {label} T={cfg['T']} N={N} d={cfg['d']} f={cfg['f']} G={G} m_g={m_g} "
        f"local={local} {kind}")
    gm = X.GroupMap(G, given, local_group=local, device=DEV)
    res = X.moe_forward(x, torch.from_numpy(h).to(DEV), w1, w3, w2, k, 1, m_g, groups=gm)
    torch.cuda.synchronize()
    got = {key: v.cpu().numpy() for key, v in res.items() if key != "y"}
    ref = OR.select_ep(h, k, 1, m_g, gr, G)
    mine = None if local < 0 else {e for e in range(N) if gr[e] == local}
    assert np.array_equal(got["sel_mask"], ref.sel_mask), label
    assert np.array_equal(got["ids"], ref.ids), label
    listed = ref.n_active if mine is None else len(set(ref.ids.reshape(-1).tolist()) & mine)
    assert got["stats"][1] == listed, label
    rows = list(range(cfg["T"])) if rows is None else rows
    y_ref = OracleOutputs(x, bf16_weights_of(w1, w3, w2)).y(ref.ids, ref.w, rows, local=mine)
    y_gpu = OF.bf16_to_f64(W.bf16_bits(res["y"]))[rows]
    assert np.all(np.isfinite(y_gpu))
    # rows of tokens with no expert on the group are exactly zero; the error is measured
    # over the others (the RMS of a share over all rows shrinks with the rows it misses)
    hit = np.array([mine is None or bool(set(ref.ids[i].tolist()) & mine) for i in rows])
    assert not np.any(y_gpu[~hit]), f"{label}: rows without a term on the group must be 0"
    if not np.any(hit):
        return res["y"], 0.0
    err = assert_ffn_close(y_gpu[hit], y_ref[hit], label, f" listed={listed}")
    return res["y"], err


def test_ep_layer_shares_sum_to_the_layer():
    c = dict(N=32, k=4, d=128, f=256, T=24, logits="domains", Q=3)
    layer = make_layer(c, 3)
    full, _ = _share(c, 3, 4, 3, -1, layer=layer, label="whole layer")
    shares = [_share(c, 3, 4, 3, g, layer=layer, label=f"group {g}")[0].float() for g in range(4)]
    # y and every share are rounded to bf16 once (relative error <= 2^-9 each)
    diff = (sum(shares) - full.float()).abs().max().item()
    bound = 2 ** -9 * (full.float().abs().max().item() + sum(t.abs().max().item() for t in shares))
    assert diff <= 1.01 * bound + 1e-6


def test_ep_layer_shares_scattered_and_split():
    # few wide experts per group: the down GEMM of a share splits its reduction
    c = dict(N=16, k=2, d=128, f=1024, T=16, logits="domains", Q=2)
    layer = make_layer(c, 1)
    for g in range(4):
        _share(c, 1, 4, 1, g, kind="scattered", layer=layer, label=f"scattered group {g}")


def test_ep_layer_share_deepseek():
    c = W.CONFIGS["ds_t32"]
    layer = make_layer(c, 0)
    for local in (0, 5):
        _share(c, 0, 8, 5, local, layer=layer, label=f"ds_t32 group {local}")
    del layer
    torch.cuda.empty_cache()
