"""Seeded synthetic inputs for the XShare batch-level MoE layer.

This module is shared by the CPU oracle's tests, the HIP path's tests and the
benchmark.  It draws router logits, activations and expert weights and holds
none of the method's arithmetic (no gating, no selection, no FFN).

Workload recipe (the paper's own decode batches come from real models and
datasets that are not available; these stand in for them):

* router logits h[T,N] (fp32):
  - ``iid``: h ~ N(0,1) iid, the control case behind the closed form for the
    expected number of activated experts (Section 1);
  - ``domains``: Q domain centroids c_q ~ N(0, 1.5) per expert, each token picks
    a domain uniformly and adds noise N(0, 0.5);
  - ``spec``: R requests x L tokens (Section 4: a speculative verify batch of
    b requests with 1 + L_s tokens each); request r belongs to domain r mod Q
    (batches mix domains as in the paper's heterogeneous-request experiment,
    Section 6.3), carries its own offset N(0, 1) per expert, and each token adds
    noise N(0, 0.3), so tokens of one request are correlated (Assumption 4.1).
  Logits are drawn in float64 from numpy's PCG64 and rounded to fp32.
* activations x[T,d] and expert weights (bf16): an approximately normal value
  (Irwin-Hall sum of four 16-bit uniforms, rescaled to the requested standard
  deviation) from a counter-based integer hash of the element index, rounded to
  bf16 with round-to-nearest-even in integer arithmetic.  Every operation is an
  integer op or one IEEE fp32 multiply, so torch produces identical bits on the
  CPU and on the GPU, and any single expert matrix can be regenerated on its own.
  x ~ N(0,1), weights ~ N(0, 0.02) (standard deviation, not variance).
* the whole layer (router GEMM h = W_g x and shared experts, Section 2.1): the
  router sees x, so x carries the domain structure instead of the logits:
  x_i = c_q(i) + 0.5 eps_i with Q centroids c_q ~ N(0,1) per feature and
  eps ~ N(0,1) (both bf16 draws as above, summed in fp32, rounded to bf16 in
  integer RNE); W_g ~ N(0, 1.5 / sqrt(d)) in bf16, so a logit has a domain part
  of standard deviation about 1.5 and a token part of about 0.75.  Shared
  experts have the routed experts' shape and N(0, 0.02) weights.
"""
from __future__ import annotations

import math

import numpy as np

SEED_ROOT = 260207265

# stream ids
_S_LOGITS = 0
_S_X = 1
_S_W = 2
_MATRIX_ID = {"w1": 0, "w3": 1, "w2": 2, "s1": 3, "s3": 4, "s2": 5}
_S_ROUTER = 3


def _rng(*ids: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([SEED_ROOT, *ids])))


# ----------------------------------------------------------------------------- logits

def logits_iid(T: int, N: int, seed: int) -> np.ndarray:
    """fp32 [T,N], iid N(0,1)."""
    g = _rng(_S_LOGITS, 1, T, N, seed)
    return g.standard_normal((T, N)).astype(np.float32)


def logits_domains(T: int, N: int, n_domains: int, seed: int,
                   centroid_std: float = 1.5, noise_std: float = 0.5) -> np.ndarray:
    """fp32 [T,N] = centroid[domain(token)] + noise."""
    g = _rng(_S_LOGITS, 2, T, N, n_domains, seed)
    cent = g.normal(0.0, centroid_std, (n_domains, N))
    dom = g.integers(0, n_domains, T)
    noise = g.normal(0.0, noise_std, (T, N))
    return (cent[dom] + noise).astype(np.float32)


def logits_spec(n_req: int, tokens_per_req: int, N: int, n_domains: int, seed: int,
                centroid_std: float = 1.5, offset_std: float = 1.0,
                noise_std: float = 0.3) -> tuple[np.ndarray, np.ndarray]:
    """Speculative verify batch: (fp32 [R*L, N], int32 request offsets [R+1]).

    Request r owns tokens [r*L, (r+1)*L), belongs to domain r mod Q and has its
    own per-expert offset; tokens add independent noise.
    """
    g = _rng(_S_LOGITS, 3, n_req, tokens_per_req, N, n_domains, seed)
    cent = g.normal(0.0, centroid_std, (n_domains, N))
    off = g.normal(0.0, offset_std, (n_req, N))
    noise = g.normal(0.0, noise_std, (n_req, tokens_per_req, N))
    dom = np.arange(n_req) % n_domains
    h = cent[dom][:, None, :] + off[:, None, :] + noise
    offsets = (np.arange(n_req + 1) * tokens_per_req).astype(np.int32)
    return h.reshape(n_req * tokens_per_req, N).astype(np.float32), offsets


def logits_spec_domains(n_req: int, n_domains: int) -> np.ndarray:
    """Domain index of each request in ``logits_spec``."""
    return np.arange(n_req) % n_domains


# ----------------------------------------------------------------------------- bf16 tensors

def _mul32(x, m: int):
    """(x * m) mod 2^32 for int64 tensors holding values in [0, 2^32), without overflow."""
    lo = x & 0xFFFF
    hi = x >> 16
    return (lo * m + ((hi * m) & 0xFFFF) * 65536) & 0xFFFFFFFF


def _mix32(x):
    """32-bit integer hash: xorshift-multiply rounds with the published "lowbias32"
    constants 0x7feb352d / 0x846ca68b (Chris Wellons' hash-prospector search)."""
    x = x ^ (x >> 16)
    x = _mul32(x, 0x7FEB352D)
    x = x ^ (x >> 15)
    x = _mul32(x, 0x846CA68B)
    x = x ^ (x >> 16)
    return x


_IH_SD = 65536.0 / math.sqrt(3.0)   # std of a sum of four uniforms on [0, 65536)
_IH_MEAN = 2 * 65535                # its mean (integer part of 4 * 65535 / 2)


def _keys(key: tuple[int, ...]) -> tuple[int, int]:
    st = np.random.SeedSequence([SEED_ROOT, *key]).generate_state(2, dtype=np.uint32)
    return int(st[0]), int(st[1])


def bf16_normal(shape, std: float, key: tuple[int, ...], device="cpu", chunk: int = 1 << 24):
    """bf16 tensor of ``shape`` with approximately N(0, std) entries.

    Element n (row-major index) is a function of (key, n) only.
    """
    import torch

    numel = int(np.prod(shape)) if len(shape) else 1
    if numel >= 1 << 32:
        raise ValueError("bf16_normal: a single tensor must have < 2^32 elements")
    k1, k2 = _keys(key)
    scale = torch.tensor(std / _IH_SD, dtype=torch.float32, device=device)
    out = torch.empty(numel, dtype=torch.int16, device=device)
    for s in range(0, numel, chunk):
        e = min(numel, s + chunk)
        n = torch.arange(s, e, dtype=torch.int64, device=device)
        h1 = _mix32(n ^ k1)
        h2 = _mix32(h1 ^ k2)
        u = (h1 & 0xFFFF) + (h1 >> 16) + (h2 & 0xFFFF) + (h2 >> 16) - _IH_MEAN
        v = u.to(torch.int32).to(torch.float32) * scale          # exact convert, one fp32 multiply
        b = v.view(torch.int32).to(torch.int64) & 0xFFFFFFFF
        b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16                  # round to nearest even
        out[s:e] = (b - ((b & 0x8000) << 1)).to(torch.int16)     # as signed 16-bit pattern
        del n, h1, h2, u, v, b
    return out.view(torch.bfloat16).reshape(shape)


def activations(T: int, d: int, seed: int, device="cpu"):
    """x [T,d] bf16, ~N(0,1)."""
    return bf16_normal((T, d), 1.0, (_S_X, T, d, seed), device)


def _round_bf16(v):
    """fp32 tensor -> bf16 with round-to-nearest-even done in integer arithmetic."""
    import torch

    b = v.contiguous().view(torch.int32).to(torch.int64) & 0xFFFFFFFF
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    return (b - ((b & 0x8000) << 1)).to(torch.int16).view(torch.bfloat16)


def activations_domains(T: int, d: int, n_domains: int, seed: int, device="cpu"):
    """x [T,d] bf16 = c[domain(token)] + 0.5 eps: hidden states with domain structure."""
    import torch

    dom = _rng(_S_X, 2, T, d, n_domains, seed).integers(0, n_domains, T)
    c = bf16_normal((n_domains, d), 1.0, (_S_X, 3, d, n_domains, seed), device).float()
    eps = bf16_normal((T, d), 1.0, (_S_X, 4, T, d, seed), device).float()
    v = c[torch.as_tensor(dom, device=device)] + eps * 0.5      # fp32: one multiply, one add
    return _round_bf16(v).reshape(T, d)


def router_weights(N: int, d: int, seed: int, device="cpu"):
    """W_g [N,d] bf16 ~ N(0, 1.5 / sqrt(d)) (nn.Linear [out,in] layout)."""
    return bf16_normal((N, d), 1.5 / math.sqrt(d), (_S_ROUTER, N, d, seed), device)


def shared_weights(n_shared: int, d: int, f: int, seed: int, device="cpu", std: float = 0.02):
    """(w1 [N_s,f,d], w3 [N_s,f,d], w2 [N_s,d,f]) bf16 of the always-on shared experts."""
    import torch

    w1 = torch.empty((n_shared, f, d), dtype=torch.bfloat16, device=device)
    w3 = torch.empty((n_shared, f, d), dtype=torch.bfloat16, device=device)
    w2 = torch.empty((n_shared, d, f), dtype=torch.bfloat16, device=device)
    for e in range(n_shared):
        w1[e] = expert_matrix(e, "s1", d, f, seed, device, std)
        w3[e] = expert_matrix(e, "s3", d, f, seed, device, std)
        w2[e] = expert_matrix(e, "s2", d, f, seed, device, std)
    return w1, w3, w2


def quantize_rows_e4m3(w):
    """bf16 matrix [rows, cols] -> (OCP FP8 E4M3FN codes uint8 [rows, cols], fp32 scale
    [rows]) with scale = max|row| / 448 (1 for an all-zero row) and codes = w / scale
    rounded to nearest even by torch's float8_e4m3fn conversion."""
    import torch

    v = w.float()
    amax = v.abs().amax(dim=1)
    scale = torch.where(amax > 0, amax / 448.0, torch.ones_like(amax))
    q = (v / scale[:, None]).clamp(-448.0, 448.0).to(torch.float8_e4m3fn)
    return q.view(torch.uint8), scale


def expert_weights_fp8(N: int, d: int, f: int, seed: int, device="cpu", std: float = 0.02):
    """FP8 versions of expert_weights, quantized per output row:
    (q1 [N,f,d], q3 [N,f,d], q2 [N,d,f] uint8 codes; s1 [N,f], s3 [N,f], s2 [N,d] fp32)."""
    import torch

    q = [torch.empty((N, f, d), dtype=torch.uint8, device=device),
         torch.empty((N, f, d), dtype=torch.uint8, device=device),
         torch.empty((N, d, f), dtype=torch.uint8, device=device)]
    sc = [torch.empty((N, f), dtype=torch.float32, device=device),
          torch.empty((N, f), dtype=torch.float32, device=device),
          torch.empty((N, d), dtype=torch.float32, device=device)]
    for e in range(N):
        for i, which in enumerate(("w1", "w3", "w2")):
            q[i][e], sc[i][e] = quantize_rows_e4m3(expert_matrix(e, which, d, f, seed, device, std))
    return (*q, *sc)


def quantize_mx_e2m1(w):
    """Matrix [rows, cols] (cols a multiple of 32) -> MXFP4: (packed E2M1 codes uint8
    [rows, cols / 2], element 2c in the low nibble; E8M0 scales uint8 [rows, cols / 32]).

    Per block of 32 elements of a row, as the OCP MX conversion does: the shared exponent
    X = floor(log2(max |v|)) - 2 (2 = the exponent of E2M1's largest value, 6 = 1.5 * 2^2;
    X = -127 for an all-zero block, clamped to [-127, 127]); each v / 2^X rounded to the
    nearest E2M1 value, ties to even mantissa, saturating at +-6."""
    import torch

    v = w.float()
    rows, cols = v.shape
    blk = v.reshape(rows, cols // 32, 32)
    amax = blk.abs().amax(dim=2)
    _, ex = torch.frexp(amax)                       # amax = m * 2^ex, m in [0.5, 1)
    X = torch.where(amax > 0, ex - 1 - 2, torch.full_like(ex, -127)).clamp(-127, 127)
    a = (blk.abs() / torch.exp2(X.float())[:, :, None]).clamp(max=6.0)
    # the grid spacing is 0.5 below 2, 1 in [2, 4), 2 from 4; an even multiple of the
    # spacing has an even mantissa, so round-half-even of a / step is the format's rounding
    step = torch.where(a < 2.0, 0.5, torch.where(a < 4.0, 1.0, 2.0))
    q = torch.round(a / step) * step
    idx = torch.where(q < 2.0, q * 2.0, torch.where(q < 4.0, q + 2.0, q / 2.0 + 4.0))
    code = idx.to(torch.uint8) | (torch.signbit(blk).to(torch.uint8) << 3)
    code = code.reshape(rows, cols)
    packed = code[:, 0::2] | (code[:, 1::2] << 4)
    return packed.contiguous(), (X + 127).to(torch.uint8)


def expert_weights_mxfp4(N: int, d: int, f: int, seed: int, device="cpu", std: float = 0.02):
    """MXFP4 versions of expert_weights: (q1 [N,f,d/2], q3 [N,f,d/2], q2 [N,d,f/2] packed
    E2M1 codes; e1 [N,f,d/32], e3 [N,f,d/32], e2 [N,d,f/32] E8M0 scales), uint8."""
    import torch

    q = [torch.empty((N, f, d // 2), dtype=torch.uint8, device=device),
         torch.empty((N, f, d // 2), dtype=torch.uint8, device=device),
         torch.empty((N, d, f // 2), dtype=torch.uint8, device=device)]
    sc = [torch.empty((N, f, d // 32), dtype=torch.uint8, device=device),
          torch.empty((N, f, d // 32), dtype=torch.uint8, device=device),
          torch.empty((N, d, f // 32), dtype=torch.uint8, device=device)]
    for e in range(N):
        for i, which in enumerate(("w1", "w3", "w2")):
            q[i][e], sc[i][e] = quantize_mx_e2m1(expert_matrix(e, which, d, f, seed, device, std))
    return (*q, *sc)


def expert_matrix(e: int, which: str, d: int, f: int, seed: int, device="cpu", std: float = 0.02):
    """One expert matrix in nn.Linear [out,in] layout: w1/w3 (s1/s3 for shared experts) are
    [f,d], w2 (s2) is [d,f]."""
    shape = (d, f) if which in ("w2", "s2") else (f, d)
    return bf16_normal(shape, std, (_S_W, _MATRIX_ID[which], e, d, f, seed), device)


def expert_weights(N: int, d: int, f: int, seed: int, device="cpu", std: float = 0.02):
    """(w1 [N,f,d], w3 [N,f,d], w2 [N,d,f]) bf16; expert e's slice equals expert_matrix(e, ...)."""
    import torch

    w1 = torch.empty((N, f, d), dtype=torch.bfloat16, device=device)
    w3 = torch.empty((N, f, d), dtype=torch.bfloat16, device=device)
    w2 = torch.empty((N, d, f), dtype=torch.bfloat16, device=device)
    for e in range(N):
        w1[e] = expert_matrix(e, "w1", d, f, seed, device, std)
        w3[e] = expert_matrix(e, "w3", d, f, seed, device, std)
        w2[e] = expert_matrix(e, "w2", d, f, seed, device, std)
    return w1, w3, w2


def bf16_bits(t) -> np.ndarray:
    """uint16 numpy array of a bf16 tensor's bit patterns (host copy)."""
    import torch

    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(np.uint16)


# ----------------------------------------------------------------------------- named workloads

#: Workloads with the shapes of the paper's models (Appendix A, Section 1) and the
#: logits recipe above.  ``M`` is the default budget, ``M_sweep`` the tested ones.
CONFIGS = {
    "tiny": dict(N=16, k=2, d=64, f=128, T=8, M=8, M_sweep=(8,), k0=1, logits="iid"),
    "mixtral": dict(N=8, k=2, d=4096, f=14336, T=16, M=5, M_sweep=(5,), k0=1,
                    logits="domains", Q=4),
    "qwen": dict(N=128, k=8, d=2048, f=768, T=64, M=48, M_sweep=(32, 48, 64), k0=1,
                 logits="domains", Q=8),
    "ds_t8": dict(N=256, k=8, d=7168, f=2048, T=8, M=48, M_sweep=(24, 48, 96), k0=1,
                  logits="domains", Q=8),
    "ds_t16": dict(N=256, k=8, d=7168, f=2048, T=16, M=48, M_sweep=(24, 48, 96), k0=1,
                   logits="domains", Q=8),
    "ds_t32": dict(N=256, k=8, d=7168, f=2048, T=32, M=48, M_sweep=(24, 48, 96), k0=1,
                   logits="domains", Q=8),
    "ds_iid_t8": dict(N=256, k=8, d=7168, f=2048, T=8, M=48, M_sweep=(24, 48, 96), k0=1,
                      logits="iid"),
    "ds_iid_t32": dict(N=256, k=8, d=7168, f=2048, T=32, M=48, M_sweep=(24, 48, 96), k0=1,
                       logits="iid"),
    "spec": dict(N=256, k=8, d=7168, f=2048, T=64, R=16, L=4, M=64, M_sweep=(64,), k0=1,
                 m_r=4, logits="spec", Q=4),
}


def make_logits(cfg: dict, seed: int):
    """(logits fp32 [T,N], request offsets int32 [R+1] or None) for a named config dict."""
    kind = cfg["logits"]
    if kind == "iid":
        return logits_iid(cfg["T"], cfg["N"], seed), None
    if kind == "domains":
        return logits_domains(cfg["T"], cfg["N"], cfg["Q"], seed), None
    if kind == "spec":
        return logits_spec(cfg["R"], cfg["L"], cfg["N"], cfg["Q"], seed)
    raise ValueError(kind)
