"""Seeded input generators: determinism, distributions, and the speculative-batch calibration."""
import numpy as np
import torch

import workloads as W


def test_logits_deterministic_and_seeded():
    for name, c in W.CONFIGS.items():
        a, oa = W.make_logits(c, 3)
        b, ob = W.make_logits(c, 3)
        d, _ = W.make_logits(c, 4)
        assert a.dtype == np.float32 and a.shape == (c["T"], c["N"])
        assert np.array_equal(a, b) and not np.array_equal(a, d)
        if c["logits"] == "spec":
            assert np.array_equal(oa, ob) and oa[0] == 0 and oa[-1] == c["T"]


def test_bf16_generator_distribution_and_rounding():
    t = W.bf16_normal((512, 1024), 0.02, (9, 9))
    v = t.float()
    assert abs(float(v.mean())) < 2e-4
    assert abs(float(v.std()) - 0.02) < 2e-4
    # integer rounding equals torch's own fp32 -> bf16 round-to-nearest-even
    u = W.bf16_normal((64, 64), 1.0, (1,))
    assert torch.equal(u, u.float().to(torch.bfloat16))
    # regenerating one expert matrix alone gives the same slice
    w1, w3, w2 = W.expert_weights(3, 64, 32, 5)
    assert torch.equal(w2[1], W.expert_matrix(1, "w2", 64, 32, 5))
    assert torch.equal(w1[2], W.expert_matrix(2, "w1", 64, 32, 5))
    assert not torch.equal(w1[2], w3[2])


def test_bf16_bits_roundtrip():
    t = W.activations(4, 16, 0)
    bits = W.bf16_bits(t)
    assert bits.dtype == np.uint16 and bits.shape == (4, 16)
    back = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16)
    assert torch.equal(back, t)


def _topk_sets(h, k):
    return [set(np.argsort(-h[i].astype(np.float64), kind="stable")[:k]) for i in range(h.shape[0])]


def test_spec_batch_overlap_calibration():
    """Section 4: top-k overlap of tokens of one request is 2-3x that of same-domain tokens."""
    same_req, same_dom, diff_dom = [], [], []
    R_, L, Q = 16, 4, 4
    for seed in range(20):
        h, off = W.logits_spec(R_, L, 256, Q, seed)
        sets = _topk_sets(h, 8)
        dom = W.logits_spec_domains(R_, Q)
        for a in range(R_ * L):
            for b in range(a + 1, R_ * L):
                ra, rb = a // L, b // L
                ov = len(sets[a] & sets[b])
                if ra == rb:
                    same_req.append(ov)
                elif dom[ra] == dom[rb]:
                    same_dom.append(ov)
                else:
                    diff_dom.append(ov)
    ratio = np.mean(same_req) / np.mean(same_dom)
    assert 2.0 <= ratio <= 3.0, ratio
    assert np.mean(diff_dom) < np.mean(same_dom)


def test_domain_logits_concentrate_routing():
    """Domain-centroid batches activate fewer experts than iid routing (skewed popularity)."""
    iid = np.mean([len(set().union(*_topk_sets(W.logits_iid(32, 256, s), 8))) for s in range(10)])
    dom = np.mean([len(set().union(*_topk_sets(W.logits_domains(32, 256, 8, s), 8))) for s in range(10)])
    assert dom < 0.75 * iid
