"""Pins for the oracle's decode during generation: each KV head's compressed
rows plus the rows appended since compression (one per generated token, per
KV head, shared by the group's query heads; Appendix A.2).

* At a 100 % budget the compressed cache is the prompt, so decode over it
  plus the appended rows is full attention over prompt + new tokens: checked
  against torch's scaled_dot_product_attention in fp64.
* A segment with no compressed rows attends to its appended rows alone.
* An appended key far above the rest makes the output its V row.
"""
import math

import numpy as np
import pytest
import torch

import oracle


def _rng(seed):
    return np.random.Generator(np.random.PCG64(400 + seed))


@pytest.mark.parametrize("n_new", [1, 5, 12])
def test_full_budget_plus_new_tokens_is_full_attention(n_new):
    rng = _rng(n_new)
    B, Hq, Hkv, d, C, cap = 2, 6, 2, 16, 40, 12
    G = Hq // Hkv
    k = rng.standard_normal((B, Hkv, C, d))
    v = rng.standard_normal((B, Hkv, C, d))
    kn = rng.standard_normal((B, Hkv, cap, d))
    vn = rng.standard_normal((B, Hkv, cap, d))
    q = rng.standard_normal((B, Hq, d))
    offsets = np.arange(B * Hkv + 1, dtype=np.int64) * C  # every segment holds its whole prompt
    out, lse = oracle.decode_append(q, k.reshape(-1, d), v.reshape(-1, d), offsets, kn, vn, n_new, Hkv)
    kk = torch.from_numpy(np.concatenate([k, kn[:, :, :n_new]], axis=2)).repeat_interleave(G, dim=1)
    vv = torch.from_numpy(np.concatenate([v, vn[:, :, :n_new]], axis=2)).repeat_interleave(G, dim=1)
    qq = torch.from_numpy(q)[:, :, None, :]
    ref = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv)[:, :, 0].numpy()
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-13)
    logits = (qq @ kk.transpose(-1, -2))[:, :, 0] / math.sqrt(d)
    np.testing.assert_allclose(lse, torch.logsumexp(logits, dim=-1).numpy(), rtol=1e-12, atol=1e-12)


def test_empty_segment_and_no_new_rows():
    rng = _rng(20)
    B, Hq, Hkv, d, cap = 1, 4, 2, 8, 6
    kc = rng.standard_normal((7, d))
    vc = rng.standard_normal((7, d))
    kn = rng.standard_normal((B, Hkv, cap, d))
    vn = rng.standard_normal((B, Hkv, cap, d))
    q = rng.standard_normal((B, Hq, d))
    offsets = np.array([0, 0, 7], dtype=np.int64)  # head 0 kept nothing, head 1 seven rows
    out, lse = oracle.decode_append(q, kc, vc, offsets, kn, vn, 3, Hkv)
    # head 0 (query heads 0, 1): attention over its three appended rows only
    lg = q[0, :2] @ kn[0, 0, :3].T / math.sqrt(d)
    p = np.exp(lg - lg.max(axis=1, keepdims=True))
    p /= p.sum(axis=1, keepdims=True)
    np.testing.assert_allclose(out[0, :2], p @ vn[0, 0, :3], rtol=1e-12)
    # nothing appended and nothing kept: zero output, lse = -inf
    out0, lse0 = oracle.decode_append(q, kc, vc, offsets, kn, vn, 0, Hkv)
    assert np.all(out0[0, :2] == 0) and np.all(np.isneginf(lse0[0, :2]))
    ref, ref_lse = oracle.decode(q, kc, vc, offsets, Hkv)
    np.testing.assert_array_equal(out0[0, 2:], ref[0, 2:])


def test_dominant_new_key_returns_its_value():
    rng = _rng(21)
    B, Hq, Hkv, d, cap = 1, 2, 1, 8, 4
    q = rng.standard_normal((B, Hq, d))
    q[0, 1] = q[0, 0]
    kc = rng.standard_normal((30, d)) * 0.1
    vc = rng.standard_normal((30, d))
    kn = rng.standard_normal((B, Hkv, cap, d)) * 0.1
    vn = rng.standard_normal((B, Hkv, cap, d))
    kn[0, 0, 2] = 40.0 * q[0, 0] / np.linalg.norm(q[0, 0])  # logit ~ 40*|q|/sqrt(8), far above the rest
    out, _ = oracle.decode_append(q, kc, vc, np.array([0, 30]), kn, vn, 3, Hkv)
    np.testing.assert_allclose(out[0], np.broadcast_to(vn[0, 0, 2], (2, d)), rtol=1e-9, atol=1e-9)


def test_invalid():
    z = np.zeros((1, 1, 2, 4))
    with pytest.raises(oracle.OracleError):
        oracle.decode_append(np.zeros((1, 1, 4)), np.zeros((1, 4)), np.zeros((1, 4)), np.array([0, 1]), z, z, 3, 1)
