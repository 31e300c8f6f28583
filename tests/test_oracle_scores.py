"""Pins for the oracle's observation-window scores and pooling.

Token selection follows SnapKV-style cumulative attention of a final
observation window (Sec. 3.3 last paragraph; Sec. 5, Query-Aware window =
the last prompt tokens). The paper prints no numeric example, so the oracle is
pinned against closed forms computed with exact integer/rational arithmetic
(independent of the oracle's exp/log path), and against torch's softmax in
fp64 on small random inputs.
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden():
    with open(os.path.join(GOLDEN, "scores_closed_forms.json")) as f:
        return json.load(f)


def test_toy_example():
    g = _golden()["toy"]
    q_win = np.array([[[[1.0]]]])                      # B=1, Hq=1, w=1, d=1
    k = np.array([[[[0.0], [math.log(2)], [math.log(3)]]]])  # B=1, Hkv=1, C=3
    lse = oracle.window_lse(q_win, k, scale=1.0)
    assert lse[0, 0, 0] == pytest.approx(g["lse"], rel=1e-15)
    a = oracle.window_colsum(q_win, k, lse, scale=1.0)
    np.testing.assert_allclose(a[0, 0], g["a"], rtol=1e-14)
    pooled = oracle.pool(a, 3)
    np.testing.assert_allclose(pooled[0, 0], g["pooled_k3"], rtol=1e-14)


def test_identical_keys_closed_form():
    """All keys equal: uniform causal softmax, a_j = sum_{n=C-w+1}^{C} 1/n (tiny workload shape)."""
    g = _golden()["identical_keys"]
    C, w, kp = g["C"], g["w"], g["kp"]
    rng = np.random.Generator(np.random.PCG64(5))
    B, Hq, Hkv, d = 1, 4, 2, 64
    q_win = rng.standard_normal((B, Hq, w, d))
    base = rng.standard_normal((B, Hkv, 1, d))
    k = np.repeat(base, C, axis=2)
    lse = oracle.window_lse(q_win, k)
    # lse_i = l + ln(C-w+i+1) with l = <q_i, u_h>/sqrt(d)
    for q in range(Hq):
        for i in range(w):
            l = float(q_win[0, q, i] @ base[0, q // 2, 0]) / math.sqrt(d)
            assert lse[0, q, i] == pytest.approx(l + math.log(C - w + i + 1), rel=1e-12, abs=1e-12)
    a = oracle.window_colsum(q_win, k, lse)
    assert a.shape == (B, Hkv, C - w)
    np.testing.assert_allclose(a, g["a"], rtol=1e-12)
    exact = sum(Fraction(1, n) for n in range(C - w + 1, C + 1))
    assert float(exact) == pytest.approx(g["a"], rel=1e-15)
    pooled = oracle.pool(a, kp)
    np.testing.assert_allclose(pooled[0, :, :3], np.tile(g["pooled_edge"], (Hkv, 1)), rtol=1e-12)
    np.testing.assert_allclose(pooled[0, :, -3:], np.tile(g["pooled_edge"][::-1], (Hkv, 1)), rtol=1e-12)
    np.testing.assert_allclose(pooled[0, :, 3:-3], g["a"], rtol=1e-12)


def _power_sum(c: int, n: int, rev_C: int | None = None) -> int:
    """sum_{t=0}^{n} base(t)^c with base(t) = t+1, or C-t when rev_C is given (exact integers)."""
    if rev_C is None:
        return sum((t + 1) ** c for t in range(n + 1))
    return sum((rev_C - t) ** c for t in range(n + 1))


def test_power_law_closed_form_gqa_batch():
    """Keys ln(j+1) or ln(C-j) make softmax rows exact power laws; pins scale, causality,
    the window-row positions, the query-head -> KV-head map, the group mean and batching."""
    B, Hq, Hkv, d, C, w = 2, 4, 2, 4, 40, 3
    G = Hq // Hkv
    # default scale 1/sqrt(4) = 1/2; query (2c, 0, 0, 0) turns <q,k>/2 into c * k[0]
    cs = np.array([[1, 0, 2, 3], [3, 2, 0, 1]])  # per (b, q head) exponent
    q_win = np.zeros((B, Hq, w, d))
    q_win[:, :, :, 0] = 2.0 * cs[:, :, None]
    rng = np.random.Generator(np.random.PCG64(7))
    k = rng.standard_normal((B, Hkv, C, d))  # other coordinates meet zero query entries
    j = np.arange(C)
    # (b, kv head) families: forward ln(j+1) or reversed ln(C-j)
    rev = np.array([[False, True], [True, False]])
    for b in range(B):
        for h in range(Hkv):
            k[b, h, :, 0] = np.log(C - j) if rev[b, h] else np.log(j + 1)
    lse = oracle.window_lse(q_win, k)
    a = oracle.window_colsum(q_win, k, lse)
    for b in range(B):
        for h in range(Hkv):
            rc = C if rev[b, h] else None
            expect = []
            for jj in range(C - w):
                tot = Fraction(0)
                for g in range(G):
                    c = int(cs[b, h * G + g])
                    for i in range(w):
                        pos = C - w + i
                        num = (C - jj if rev[b, h] else jj + 1) ** c
                        tot += Fraction(num, _power_sum(c, pos, rc))
                expect.append(float(tot / G))
            np.testing.assert_allclose(a[b, h], expect, rtol=1e-12)
            for g in range(G):
                c = int(cs[b, h * G + g])
                for i in range(w):
                    ref = math.log(_power_sum(c, C - w + i, rc))
                    assert lse[b, h * G + g, i] == pytest.approx(ref, rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_against_torch_softmax(seed):
    """Random small inputs: the same quantities through torch.softmax with a causal mask in fp64."""
    rng = np.random.Generator(np.random.PCG64(100 + seed))
    B, Hq, Hkv, d, C, w = 2, 6, 2, 16, 37, 5
    q_win = rng.standard_normal((B, Hq, w, d))
    k = rng.standard_normal((B, Hkv, C, d)) * 2.0
    lse = oracle.window_lse(q_win, k)
    a = oracle.window_colsum(q_win, k, lse)
    qt = torch.from_numpy(q_win)
    kt = torch.from_numpy(k).repeat_interleave(Hq // Hkv, dim=1)  # repeat_kv order
    logits = qt @ kt.transpose(-1, -2) / math.sqrt(d)  # [B, Hq, w, C]
    pos = torch.arange(C - w, C)[:, None]
    mask = torch.arange(C)[None, :] <= pos
    logits = logits.masked_fill(~mask, float("-inf"))
    p = torch.softmax(logits, dim=-1)
    ref_lse = torch.logsumexp(logits, dim=-1).numpy()
    np.testing.assert_allclose(lse, ref_lse, rtol=1e-12, atol=1e-12)
    colsum = p.sum(dim=2)[..., : C - w]  # [B, Hq, C-w]
    ref = colsum.reshape(B, Hkv, Hq // Hkv, C - w).mean(dim=2).numpy()
    np.testing.assert_allclose(a, ref, rtol=1e-11, atol=1e-15)
    # every window row is a distribution over its visible keys
    assert torch.allclose(p.sum(-1), torch.ones(B, Hq, w, dtype=torch.float64))


def test_pool_pins():
    x = np.zeros((2, 11))
    x[0, 5] = 7.0
    x[1, :] = 1.0
    p = oracle.pool(x, 7)
    np.testing.assert_array_equal(p[0], [0, 0, 1, 1, 1, 1, 1, 1, 1, 0, 0])
    np.testing.assert_allclose(p[1], np.array([4, 5, 6, 7, 7, 7, 7, 7, 6, 5, 4]) / 7.0, rtol=1e-15)
    # kernel 1 is the identity
    r = np.random.Generator(np.random.PCG64(1)).random((3, 20))
    np.testing.assert_array_equal(oracle.pool(r, 1), r)
    # scipy's uniform filter with zero padding agrees in the interior and at the edges
    from scipy.ndimage import uniform_filter1d
    np.testing.assert_allclose(oracle.pool(r, 5), uniform_filter1d(r, 5, axis=-1, mode="constant"),
                               rtol=1e-13)
    with pytest.raises(oracle.OracleError):
        oracle.pool(r, 4)
