"""Pins for the oracle's importance-weighted group aggregation (Appendix A.7,
the "Ipt." rows of Table 5): each query head's window-summed attention is
multiplied by its summarization score, then max- or mean-pooled over the
group; "only" copies the attention of the group's top-scored head.

Pinned against closed forms (identical keys make every row uniform) and
against torch.softmax in fp64 on small random inputs.
"""
import math

import numpy as np
import pytest
import torch

import oracle


def _closed_identical(C, w):
    return sum(1.0 / n for n in range(C - w + 1, C + 1))


def test_identical_keys_closed_form():
    """Identical keys: every head's window attention of a scored key is a = sum 1/n over the row
    lengths, so max gives max(sigma)*a, mean gives mean(sigma)*a and only gives a."""
    rng = np.random.Generator(np.random.PCG64(3))
    B, Hq, Hkv, d, C, w = 2, 6, 2, 8, 90, 12
    q_win = rng.standard_normal((B, Hq, w, d))
    k = np.broadcast_to(rng.standard_normal(d), (B, Hkv, C, d)).copy()
    sig = np.array([0.2, 0.9, 0.5, 0.0, 0.3, 0.3])
    lse = oracle.window_lse(q_win, k)
    a = _closed_identical(C, w)
    G = Hq // Hkv
    for agg, want in ((oracle.GROUP_IPT_MAX, lambda s: s.max() * a), (oracle.GROUP_IPT_MEAN, lambda s: s.mean() * a),
                      (oracle.GROUP_IPT_ONLY, lambda s: a)):
        out = oracle.window_colsum(q_win, k, lse, agg=agg, qhead_scores=sig)
        for h in range(Hkv):
            np.testing.assert_allclose(out[:, h], want(sig[h * G:(h + 1) * G]), rtol=1e-12)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_against_torch_softmax(seed):
    rng = np.random.Generator(np.random.PCG64(200 + seed))
    B, Hq, Hkv, d, C, w = 2, 6, 2, 16, 41, 6
    G = Hq // Hkv
    q_win = rng.standard_normal((B, Hq, w, d))
    k = rng.standard_normal((B, Hkv, C, d)) * 2.0
    sig = rng.random(Hq)
    sig[1] = sig[0]  # a tie inside the first group: "only" must take the lower head
    sig[0] = sig[1] = max(sig[:G]) + 0.1
    lse = oracle.window_lse(q_win, k)
    qt = torch.from_numpy(q_win)
    kt = torch.from_numpy(k).repeat_interleave(G, dim=1)
    logits = qt @ kt.transpose(-1, -2) / math.sqrt(d)
    pos = torch.arange(C - w, C)[:, None]
    logits = logits.masked_fill(~(torch.arange(C)[None, :] <= pos), float("-inf"))
    A = torch.softmax(logits, dim=-1).sum(dim=2)[..., : C - w].reshape(B, Hkv, G, C - w).numpy()
    S = sig.reshape(Hkv, G)[None, :, :, None]
    top = np.argmax(sig.reshape(Hkv, G), axis=1)  # first maximum
    refs = {oracle.GROUP_IPT_MAX: (S * A).max(axis=2), oracle.GROUP_IPT_MEAN: (S * A).mean(axis=2),
            oracle.GROUP_IPT_ONLY: np.stack([A[:, h, top[h]] for h in range(Hkv)], axis=1)}
    for agg, ref in refs.items():
        out = oracle.window_colsum(q_win, k, lse, agg=agg, qhead_scores=sig)
        np.testing.assert_allclose(out, ref, rtol=1e-11, atol=1e-15)
    # unit scores: the importance-weighted mean is the plain group mean
    np.testing.assert_allclose(oracle.window_colsum(q_win, k, lse, agg=oracle.GROUP_IPT_MEAN, qhead_scores=np.ones(Hq)),
                               oracle.window_colsum(q_win, k, lse), rtol=1e-13)


def test_invalid_scores():
    q_win = np.zeros((1, 2, 2, 4))
    k = np.zeros((1, 1, 8, 4))
    lse = oracle.window_lse(q_win, k)
    with pytest.raises(oracle.OracleError):
        oracle.window_colsum(q_win, k, lse, agg=oracle.GROUP_IPT_MAX, qhead_scores=np.array([1.0, -1.0]))
    with pytest.raises(oracle.OracleError):
        oracle.window_colsum(q_win, k, lse, agg=oracle.GROUP_IPT_MAX, qhead_scores=np.array([1.0]))
