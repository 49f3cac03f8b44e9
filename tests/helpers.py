"""Shared test helpers: running the HIP path and the oracle on the same seeded inputs."""
import sys

import numpy as np
import torch

import workloads as W
from oracle import ffn as OF
from oracle import route as OR

DEV = "cuda:0"


def say(*a):
    """Progress line naming the case, flushed before the GPU step it precedes."""
    print(*a, flush=True)
    sys.stdout.flush()


def gpu_route(h, k, k0, M, budget_mode="total", score_mode="topk", offsets=None, m_r=0,
              device_offsets_only=False, tau=0.0):
    from paper_2602_07265_amd import xshare as X
    hd = torch.from_numpy(np.ascontiguousarray(h)).to(DEV)
    if offsets is None:
        res = X.route(hd, k, k0, M, budget_mode, score_mode, tau=tau)
    else:
        off = torch.tensor(np.asarray(offsets, np.int32), device=DEV) if device_offsets_only \
            else list(int(v) for v in offsets)
        res = X.select_hier(hd, off, k, k0, m_r, M, budget_mode, score_mode, tau=tau)
    torch.cuda.synchronize()
    return {key: v.cpu().numpy() for key, v in res.items()}


def oracle_route(h, k, k0, M, budget_mode="total", score_mode="topk", offsets=None, m_r=0,
                 tau=None):
    if offsets is None:
        return OR.route(h, k, k0, M, budget_mode, score_mode, tau)
    return OR.select_hier(h, offsets, k, k0, m_r, M, budget_mode, score_mode, tau)


def assert_route_equal(got, ref, label=""):
    T, k = ref.ids.shape
    assert np.array_equal(got["sel_mask"], ref.sel_mask), f"{label}: selected set differs"
    assert np.array_equal(got["ids"].reshape(T, k), ref.ids), f"{label}: routing ids differ"
    assert np.array_equal(got["w"].reshape(T, k).view(np.uint32), ref.w.view(np.uint32)), \
        f"{label}: routing weights differ"
    st = got["stats"]
    exp = [ref.n_selected, ref.n_active, ref.n_vanilla_union, ref.n_warmup]
    assert list(st[:4]) == exp, f"{label}: stats {list(st[:4])} != {exp}"
    assert st[5] == ref.budget_eff, f"{label}: budget_eff {st[5]} != {ref.budget_eff}"


def make_layer(cfg, seed, device=DEV):
    """x [T,d], logits [T,N] (numpy fp32), offsets, and all expert weights on the device."""
    h, off = W.make_logits(cfg, seed)
    x = W.activations(cfg["T"], cfg["d"], seed, device)
    w1, w3, w2 = W.expert_weights(cfg["N"], cfg["d"], cfg["f"], seed, device)
    return h, off, x, w1, w3, w2


def expert_fetcher(w1, w3, w2):
    cache = {}

    def get(e):
        if e not in cache:
            cache[e] = tuple(W.bf16_bits(m[e]) for m in (w1, w3, w2))
        return cache[e]
    return get


def ffn_error(y_gpu, y_ref):
    """max |y_gpu - y_ref| / RMS(y_ref) over the compared rows."""
    yg = y_gpu.astype(np.float64)
    rms = float(np.sqrt(np.mean(y_ref ** 2)))
    return float(np.max(np.abs(yg - y_ref))) / rms, rms


def bf16_to_f64(t):
    return OF.bf16_to_f64(W.bf16_bits(t))


def last_listed_rows(ids, rows, n=2, per=2, heavy=8):
    """rows plus up to `per` tokens of each of the last n experts of the GEMMs' active list
    (experts with more than `heavy` rows first, then the others, each class in expert
    order), from the oracle's routing: the slots that a launch's last round holds."""
    e, c = np.unique(ids[ids >= 0], return_counts=True)
    order = [int(j) for j in e[c > heavy]] + [int(j) for j in e[c <= heavy]]
    out = list(rows)
    for j in order[-n:]:
        out += [int(i) for i in np.nonzero((ids == j).any(axis=1))[0][:per]]
    return sorted(set(out))
