"""Pins for the oracle's observation-window placement (Sec. 5: Query-Aware,
Query-Unaware and Proxy-Query windows). Window row i sits at position
win0 + i and attends to the cached keys 0..min(win0 + i, C - 1); the keys
before the window, [0, win0), are scored.

* A window ending before a question of q_len tokens (win0 = C - q_len - w)
  sees exactly what the default window of the prompt truncated before the
  question sees: the results must be identical, bit for bit.
* A window after the prompt (win0 = C, proxy queries) sees every cached key:
  checked against torch.softmax without a mask in fp64, and against the
  identical-key closed form a_j = w / C.
"""
import math

import numpy as np
import pytest
import torch

import oracle


def _inputs(seed, B=2, Hq=6, Hkv=2, d=16, C=53, w=7):
    rng = np.random.Generator(np.random.PCG64(300 + seed))
    return rng.standard_normal((B, Hq, w, d)), rng.standard_normal((B, Hkv, C, d)) * 2.0


@pytest.mark.parametrize("q_len", [1, 9])
def test_query_unaware_equals_truncated_prompt(q_len):
    q, k = _inputs(q_len)
    C, w = k.shape[2], q.shape[2]
    win0 = C - q_len - w
    lse = oracle.window_lse(q, k, win0=win0)
    ref_lse = oracle.window_lse(q, k[:, :, :C - q_len])
    assert np.array_equal(lse, ref_lse)
    for agg, qs in ((oracle.GROUP_MEAN, None), (oracle.GROUP_IPT_MAX, np.linspace(0.1, 1.0, q.shape[1]))):
        a = oracle.window_colsum(q, k, lse, agg=agg, qhead_scores=qs, win0=win0)
        ref = oracle.window_colsum(q, k[:, :, :C - q_len], ref_lse, agg=agg, qhead_scores=qs)
        assert a.shape == ref.shape == (k.shape[0], k.shape[1], win0)
        assert np.array_equal(a, ref)


def test_proxy_window_sees_every_key():
    q, k = _inputs(5)
    B, Hq, w, d = q.shape
    C, Hkv = k.shape[2], k.shape[1]
    lse = oracle.window_lse(q, k, win0=C)
    a = oracle.window_colsum(q, k, lse, win0=C)
    logits = torch.from_numpy(q) @ torch.from_numpy(k).repeat_interleave(Hq // Hkv, dim=1).transpose(-1, -2)
    logits = logits / math.sqrt(d)
    np.testing.assert_allclose(lse, torch.logsumexp(logits, dim=-1).numpy(), rtol=1e-12, atol=1e-12)
    ref = torch.softmax(logits, dim=-1).sum(dim=2).reshape(B, Hkv, Hq // Hkv, C).mean(dim=2).numpy()
    assert a.shape == (B, Hkv, C)
    np.testing.assert_allclose(a, ref, rtol=1e-11, atol=1e-15)


def test_proxy_identical_keys_closed_form():
    q, k = _inputs(6)
    k[:] = k[:, :, :1]
    C, w = k.shape[2], q.shape[2]
    a = oracle.window_colsum(q, k, oracle.window_lse(q, k, win0=C), win0=C)
    np.testing.assert_allclose(a, w / C, rtol=1e-12)


def test_selection_needs_scores_for_every_candidate():
    pooled = np.arange(40, dtype=np.float64)
    # 40 scored keys of C = 50: candidates [s, C - W) must end by 40
    assert oracle.select(pooled, 50, 10, 2, 10, 5).tolist()[:2] == [0, 1]
    with pytest.raises(oracle.OracleError):
        oracle.select(pooled, 50, 10, 2, 9, 5)  # C - W = 41 > 40
    sel = oracle.select(np.arange(50.0), 50, 0, 2, 4, 3, win0=50)  # proxy: every key scored
    assert sel.tolist() == [0, 1, 43, 44, 45, 46, 47, 48, 49]
    with pytest.raises(oracle.OracleError):
        oracle.window_lse(*_inputs(7), win0=54)
