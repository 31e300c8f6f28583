"""Pins for the oracle's token selection, gather and decode.

Selection keeps, inside each head's budget, the middle tokens with the
largest pooled window score (Sec. 3.3 last paragraph), with sink and recent
window always kept (Sec. 3.3). The cache is per KV head, before repetition
(Appendix A.2). Pins: a rank-count definition of top-k that uses no sort,
closed forms, torch's scaled-dot-product attention in fp64, and the
100 %-budget case that must reproduce full attention.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rank_select(pooled, C, w, s, W, m):
    """Candidate j is kept iff fewer than m candidates beat it (higher score, or equal score
    at a lower position). No sorting involved."""
    cand = list(range(s, C - W))
    kept = []
    for j in cand:
        better = sum(1 for t in cand if pooled[t] > pooled[j] or (pooled[t] == pooled[j] and t < j))
        if better < m:
            kept.append(j)
    return sorted(list(range(s)) + kept + list(range(C - W, C)))


@pytest.mark.parametrize("seed", range(12))
def test_select_matches_rank_definition(seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    C = int(rng.integers(8, 80))
    w = int(rng.integers(1, 6))
    W = int(rng.integers(w, min(C // 2, w + 6) + 1))
    s = int(rng.integers(0, max(1, C - W - 1)))
    M = C - s - W
    # heavy ties: values from a tiny set
    pooled = rng.integers(0, 4, size=C - w).astype(np.float64) / 7.0
    for m in sorted({0, M, int(rng.integers(0, M + 1)), M // 2}):
        got = oracle.select(pooled, C, w, s, W, m)
        assert got.tolist() == _rank_select(pooled, C, w, s, W, m)
        assert len(got) == s + m + W
        assert np.all(np.diff(got) > 0)


def test_select_toy_tie():
    g = json.load(open(os.path.join(GOLDEN, "scores_closed_forms.json")))["toy"]
    got = oracle.select(np.array(g["pooled_k3"]), C=3, w=1, s=0, W=1, m=1)
    assert got.tolist() == g["kept_s0_W1_m1"]


def test_identical_keys_keep_lowest_positions():
    """Equal pooled scores over the interior: ties go to the lower positions, kept = [s, s+m)."""
    C, w, s, W, kp = 2048, 32, 4, 32, 7
    rng = np.random.Generator(np.random.PCG64(3))
    q_win = rng.standard_normal((1, 2, w, 16))
    k = np.repeat(rng.standard_normal((1, 1, 1, 16)), C, axis=2)
    v = rng.standard_normal((1, 1, C, 16))
    for m in (0, 1, 700, 2009):
        res = oracle.compress(q_win, k, v, [s + W + m], w=w, kp=kp, s=s, W=W)
        expect = list(range(s)) + list(range(s, s + m)) + list(range(C - W, C))
        assert res["kept_pos"].tolist() == expect


def test_compress_full_budget_keeps_everything():
    rng = np.random.Generator(np.random.PCG64(11))
    B, Hq, Hkv, d, C, w = 2, 4, 2, 8, 50, 4
    q_win = rng.standard_normal((B, Hq, w, d))
    k = rng.standard_normal((B, Hkv, C, d))
    v = rng.standard_normal((B, Hkv, C, d))
    res = oracle.compress(q_win, k, v, [C, C], w=w, kp=3, s=2, W=6)
    assert res["kept_pos"].tolist() == list(range(C)) * (B * Hkv)
    assert res["offsets"].tolist() == [0, C, 2 * C, 3 * C, 4 * C]
    np.testing.assert_array_equal(res["k_c"], k.reshape(-1, d))
    np.testing.assert_array_equal(res["v_c"], v.reshape(-1, d))


def test_compress_ragged_gather_and_offsets():
    rng = np.random.Generator(np.random.PCG64(12))
    B, Hq, Hkv, d, C, w, s, W = 2, 6, 3, 8, 60, 4, 3, 5
    q_win = rng.standard_normal((B, Hq, w, d))
    k = rng.standard_normal((B, Hkv, C, d))
    v = rng.standard_normal((B, Hkv, C, d))
    budgets = [s + W + 0, s + W + 17, C]
    res = oracle.compress(q_win, k, v, budgets, w=w, kp=7, s=s, W=W)
    T = sum(budgets)
    assert res["offsets"].tolist() == [0, 8, 33, 93, 101, 126, 186]
    assert res["kept_pos"].size == B * T
    off = res["offsets"]
    for b in range(B):
        for h in range(Hkv):
            seg = slice(off[b * Hkv + h], off[b * Hkv + h + 1])
            pos = res["kept_pos"][seg]
            np.testing.assert_array_equal(res["k_c"][seg], k[b, h, pos])
            np.testing.assert_array_equal(res["v_c"][seg], v[b, h, pos])
            assert pos.tolist() == _rank_select(res["pooled"][b, h], C, w, s, W, budgets[h] - s - W)


def _sdpa(q, k, v, G):
    """torch scaled-dot-product attention in fp64 with repeat_kv grouping; q [B,Hq,d]."""
    qt = torch.from_numpy(q)[:, :, None, :]
    kt = torch.from_numpy(k).repeat_interleave(G, dim=1)
    vt = torch.from_numpy(v).repeat_interleave(G, dim=1)
    return F.scaled_dot_product_attention(qt, kt, vt)[:, :, 0, :].numpy()


def test_decode_full_budget_equals_full_attention():
    rng = np.random.Generator(np.random.PCG64(21))
    B, Hq, Hkv, d, C, w = 2, 6, 2, 16, 64, 4
    q_win = rng.standard_normal((B, Hq, w, d))
    k = rng.standard_normal((B, Hkv, C, d)) * 2
    v = rng.standard_normal((B, Hkv, C, d))
    q = rng.standard_normal((B, Hq, d))
    res = oracle.compress(q_win, k, v, [C] * Hkv, w=w, kp=7, s=4, W=8)
    out, lse = oracle.decode(q, res["k_c"], res["v_c"], res["offsets"], Hkv)
    np.testing.assert_allclose(out, _sdpa(q, k, v, Hq // Hkv), rtol=1e-12, atol=1e-13)
    kt = torch.from_numpy(k).repeat_interleave(Hq // Hkv, dim=1)
    ref_lse = torch.logsumexp(torch.einsum("bhd,bhcd->bhc", torch.from_numpy(q), kt) / math.sqrt(d), -1)
    np.testing.assert_allclose(lse, ref_lse.numpy(), rtol=1e-12)


def test_decode_ragged_segments_against_sdpa():
    rng = np.random.Generator(np.random.PCG64(22))
    B, Hq, Hkv, d = 2, 8, 4, 32
    G = Hq // Hkv
    lens = [[5, 1, 17, 40], [3, 64, 2, 9]]
    segs_k, segs_v, offsets = [], [], [0]
    for b in range(B):
        for h in range(Hkv):
            segs_k.append(rng.standard_normal((lens[b][h], d)) * 3)
            segs_v.append(rng.standard_normal((lens[b][h], d)))
            offsets.append(offsets[-1] + lens[b][h])
    kc, vc = np.concatenate(segs_k), np.concatenate(segs_v)
    q = rng.standard_normal((B, Hq, d))
    out, _ = oracle.decode(q, kc, vc, offsets, Hkv)
    for b in range(B):
        for qh in range(Hq):
            i = b * Hkv + qh // G
            ref = _sdpa(q[b:b + 1, qh:qh + 1], segs_k[i][None, None], segs_v[i][None, None], 1)
            np.testing.assert_allclose(out[b, qh], ref[0, 0], rtol=1e-12, atol=1e-13)


def test_decode_closed_forms():
    rng = np.random.Generator(np.random.PCG64(23))
    d = 8
    q = rng.standard_normal((1, 2, d))
    # one KV head: a single-row segment returns that row exactly
    kc = rng.standard_normal((1, d))
    vc = rng.standard_normal((1, d))
    out, lse = oracle.decode(q, kc, vc, [0, 1], 1)
    np.testing.assert_array_equal(out[0, 0], vc[0])
    assert lse[0, 0] == pytest.approx(float(q[0, 0] @ kc[0]) / math.sqrt(d), rel=1e-14)
    # identical keys: the mean of the value rows
    kc = np.repeat(rng.standard_normal((1, d)), 9, axis=0)
    vc = rng.standard_normal((9, d))
    out, _ = oracle.decode(q, kc, vc, [0, 9], 1)
    np.testing.assert_allclose(out[0, 1], vc.mean(axis=0), rtol=1e-13, atol=1e-15)
    # an empty segment gives zeros and -inf
    out, lse = oracle.decode(q, kc, vc, [0, 0, 9], 2)
    assert np.all(out[0, 0] == 0) and lse[0, 0] == -np.inf
