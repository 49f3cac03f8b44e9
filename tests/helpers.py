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


def score_order_case():
    """Logits whose selection depends on the order of the score sums (s_j = sum_i g_ij).

    k = 6.  A token's gates are 1/m for the m experts tied at the top of its logits (exp(0)
    = 1 each, so the softmax gives 1/m, correctly rounded) and 0 for the rest of its top-k,
    which sit more than 80 below (exp underflows to 0).  Expert A = 2 takes gates fp32(1/3),
    1/4, fp32(1/6) from tokens 0, 1, 2; expert B = 1 takes 1/2 and 1/4 from tokens 3, 4 (an
    exact 0.75); experts 3-7 are alone at the top of tokens 5-9 (gate 1, score 1).  With a
    total budget of 6 the last slot goes to A or B.  Returns (h fp32 [10, 64], k, M, A, B).
    """
    N, k = 64, 6
    A, B = 2, 1
    h = np.full((10, N), -200.0, dtype=np.float32)
    zeros = list(range(50, 55))                   # the rest of each token's top-k, gate 0
    filler = iter(range(10, 40))
    tops = {0: [A] + [next(filler) for _ in range(2)],
            1: [A] + [next(filler) for _ in range(3)],
            2: [A] + [next(filler) for _ in range(5)],
            3: [B] + [next(filler) for _ in range(1)],
            4: [B] + [next(filler) for _ in range(3)]}
    for i in range(5, 10):
        tops[i] = [i - 2]
    for i, top in tops.items():
        h[i, top] = 10.0
        h[i, zeros[:k - len(top)]] = -100.0
    return h, k, 6, A, B


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


class OracleOutputs:
    """The oracle's expert outputs E_e(x_i) on every token of one batch, computed once per
    expert and shared by the routings of several budgets; y then follows from the oracle's
    rank-ordered routed sum (plus the shared experts' outputs, weight 1).

    ``weights_of(e)`` returns expert e's (w1, w3, w2) as bf16 bit arrays or float64 values; it
    is called once per expert and its arrays are dropped after use."""

    def __init__(self, x, weights_of, shared=()):
        self.X = OF.bf16_to_f64(W.bf16_bits(x))
        self.weights_of = weights_of
        self.out = {}
        self.shared = [OF.expert_ffn(self.X, *s) for s in shared]

    def y(self, ids, w, rows=None, local=None):
        T, d = self.X.shape
        rows = list(range(T)) if rows is None else [int(i) for i in rows]
        need = {int(e) for e in np.unique(np.asarray(ids)[rows]) if e >= 0}
        if local is not None:
            need &= set(local)
        for e in sorted(need - set(self.out)):
            self.out[e] = OF.expert_ffn(self.X, *self.weights_of(e))
        y = OF.combine(self.out, ids, w, d, rows, local)
        for s in self.shared:
            y += s[rows]
        return y


def bf16_weights_of(w1, w3, w2):
    return lambda e: tuple(W.bf16_bits(m[e]) for m in (w1, w3, w2))


def ffn_error(y_gpu, y_ref):
    """max |y_gpu - y_ref| / RMS(y_ref) over the compared rows."""
    yg = y_gpu.astype(np.float64)
    rms = float(np.sqrt(np.mean(y_ref ** 2)))
    return float(np.max(np.abs(yg - y_ref))) / rms, rms


TOL = 2e-2   # the layer output's tolerance, in units of RMS(y_ref)


def half_ulp_bf16(y):
    """Half a bf16 unit in the last place at |y| (8 significant bits): the most that rounding
    the exact value to bf16 can move it."""
    a = np.abs(np.asarray(y, dtype=np.float64))
    _, e = np.frexp(a)                       # a = m 2^e, 0.5 <= m < 1
    return np.where(a > 0, np.ldexp(1.0, e - 9), 0.0)


def rounding_excess(y_gpu, y_ref):
    """max(|y_gpu - y_ref| - half_ulp_bf16(y_ref)) / RMS(y_ref): the error beyond the bf16
    rounding that the output format forces on any result, the exact value's included."""
    rms = float(np.sqrt(np.mean(y_ref ** 2)))
    d = np.abs(y_gpu.astype(np.float64) - y_ref) - half_ulp_bf16(y_ref)
    return float(np.max(d)) / rms


def assert_ffn_close(y_gpu, y_ref, label="", note=""):
    """y within TOL * RMS(y_ref) of the oracle beyond the rounding of y to bf16.  The plain
    max |y_gpu - y_ref| / RMS is printed too; where the largest outputs sit just under a power
    of two (5.6 RMS on the speculative batch, 8.5 RMS on a group share) the exact value
    rounded to bf16 alone already misses TOL, so the bar is on the error beyond that."""
    assert np.all(np.isfinite(y_gpu)), f"{label}: non-finite output"
    err, rms = ffn_error(y_gpu, y_ref)
    exc = rounding_excess(y_gpu, y_ref)
    say(f"  max err / RMS = {err:.3e}, beyond bf16 rounding {exc:.3e} (RMS {rms:.3e}){note}")
    assert exc <= TOL, f"{label}: error beyond bf16 rounding {exc:.3e} x RMS exceeds {TOL}"
    return err


def bf16_to_f64(t):
    return OF.bf16_to_f64(W.bf16_bits(t))
