"""Seeded synthetic workloads for the SGD-KV hot path.

This module only draws random inputs and describes the workload shapes; it
holds none of the method's arithmetic, so both the HIP path's tests/bench and
the CPU oracle can use it.

The paper evaluates on MRCR, ETHIC and BABILong prompts with Qwen2.5-7B-1M
(28 layers x 4 KV heads, 28 query heads, head dim 128) and Qwen3-32B
(64 query heads, 8 KV heads). None of those models, prompts or the paper's
measured head scores are available, so seeded synthetic tensors of the same
shapes stand in for them:
  * K, V ~ N(0,1); 1 % of token positions (uniform over [4, C), shared by
    all heads and by K and V) are scaled by 8 ("heavy hitters"), the first 4
    positions by 16 ("attention sinks"); drawn in fp32, rounded to bf16;
  * window queries and decode queries ~ N(0,1);
  * per-KV-head summarization scores ~ Beta(0.5, 2), or a skewed mix where
    20 % of the heads draw from U(0.8, 1) and the rest from U(0, 0.1).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    key: str
    name: str
    layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    seq_len: int
    obs_window: int
    pool_kernel: int
    b_sink: int
    b_window: int
    batch: int
    dtype: str  # "f32" or "bf16"
    seed: int
    scores: str  # "uniform", "beta", "skewed"
    ratios: tuple = field(default=(0.25,))

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads


WORKLOADS = {
    # tiny fp32 case the oracle finishes in seconds
    "tiny": Workload("tiny", "tiny-fp32-2k", 1, 4, 2, 64, 2048, 32, 7, 4, 32, 1, "f32", 0,
                     "uniform", (0.25,)),
    # one Qwen2.5-7B-shaped layer at a 32K prompt
    "qwen25_32k": Workload("qwen25_32k", "qwen2.5-7b-32k-1L-b1", 1, 28, 4, 128, 32768, 64, 7,
                           1024, 1024, 1, "bf16", 1, "beta", (0.25,)),
    # the 28-layer Qwen2.5-7B stack at a 128K prompt, batch 8
    "qwen25_128k": Workload("qwen25_128k", "qwen2.5-7b-128k-28L-b8", 28, 28, 4, 128, 131072, 64,
                            7, 1024, 1024, 8, "bf16", 2, "beta", (0.10, 0.25, 0.50)),
    # one Qwen3-32B-shaped layer at a 256K prompt, batch 16
    "qwen3_256k": Workload("qwen3_256k", "qwen3-32b-256k-1L-b16", 1, 64, 8, 128, 262144, 64, 7,
                           128, 128, 16, "bf16", 3, "beta", (0.25,)),
    # one Qwen2.5-7B-shaped layer at a 1M (2^20) prompt, batch 32, skewed scores
    "qwen25_1m": Workload("qwen25_1m", "qwen2.5-7b-1m-1L-b32", 1, 28, 4, 128, 1 << 20, 64, 7,
                          1024, 1024, 32, "bf16", 4, "skewed", (0.25,)),
}


def head_scores(wl: Workload) -> np.ndarray:
    """Per-KV-head summarization scores, fp64 [layers * num_kv_heads], layer-major."""
    rng = np.random.Generator(np.random.PCG64(wl.seed))
    n = wl.layers * wl.num_kv_heads
    if wl.scores == "uniform":
        return rng.uniform(0.0, 1.0, size=n)
    if wl.scores == "beta":
        return rng.beta(0.5, 2.0, size=n)
    if wl.scores == "skewed":
        hot = max(1, int(round(0.2 * n)))
        perm = rng.permutation(n)
        out = rng.uniform(0.0, 0.1, size=n)
        out[perm[:hot]] = rng.uniform(0.8, 1.0, size=hot)
        return out
    raise ValueError(wl.scores)


def numpy_tensors(wl: Workload, batch: int | None = None, seq_len: int | None = None,
                  seed: int | None = None) -> dict:
    """fp32 N(0,1) tensors from NumPy PCG64 (the tiny fp32 workload)."""
    B = wl.batch if batch is None else batch
    C = wl.seq_len if seq_len is None else seq_len
    rng = np.random.Generator(np.random.PCG64(1000 + (wl.seed if seed is None else seed)))
    Hq, Hkv, d, w = wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.obs_window
    q_win = rng.standard_normal((B, Hq, w, d), dtype=np.float32)
    k = rng.standard_normal((B, Hkv, C, d), dtype=np.float32)
    v = rng.standard_normal((B, Hkv, C, d), dtype=np.float32)
    q = rng.standard_normal((B, Hq, d), dtype=np.float32)
    return dict(q_win=q_win, k=k, v=v, q=q)


def _stream_seed(seed: int, layer: int, b: int) -> int:
    return (seed * 1_000_003 + layer * 10_007 + b * 101 + 17) & 0x7FFFFFFF


def torch_layer_tensors(wl: Workload, layer: int, device, batch: int | None = None,
                        seq_len: int | None = None, dtype=None, out: dict | None = None) -> dict:
    """One layer's inputs drawn on `device` with a seeded torch.Generator.

    Returns q_win [B,Hq,w,d], k and v [B,Hkv,C,d], q [B,Hq,d] in `dtype`
    (bf16 for the Qwen-shaped workloads). Sequence b of layer l uses the
    stream seeded by (wl.seed, l, b). If `out` holds preallocated tensors of
    the right shapes they are filled in place.
    """
    import torch

    B = wl.batch if batch is None else batch
    C = wl.seq_len if seq_len is None else seq_len
    if dtype is None:
        dtype = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    Hq, Hkv, d, w = wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.obs_window
    if out is None:
        out = dict(
            q_win=torch.empty((B, Hq, w, d), dtype=dtype, device=device),
            k=torch.empty((B, Hkv, C, d), dtype=dtype, device=device),
            v=torch.empty((B, Hkv, C, d), dtype=dtype, device=device),
            q=torch.empty((B, Hq, d), dtype=dtype, device=device),
        )
    n_hh = C // 100
    for b in range(B):
        g = torch.Generator(device=device)
        g.manual_seed(_stream_seed(wl.seed, layer, b))
        if C > 4 and n_hh > 0:
            hh = torch.randperm(C - 4, generator=g, device=device)[:n_hh] + 4
        else:
            hh = torch.zeros(0, dtype=torch.long, device=device)
        for name in ("k", "v"):
            x = torch.randn((Hkv, C, d), generator=g, device=device, dtype=torch.float32)
            x[:, hh, :] *= 8.0
            x[:, : min(4, C), :] *= 16.0
            out[name][b].copy_(x.to(dtype))
            del x
        out["q_win"][b].copy_(torch.randn((Hq, w, d), generator=g, device=device,
                                          dtype=torch.float32).to(dtype))
        out["q"][b].copy_(torch.randn((Hq, d), generator=g, device=device,
                                      dtype=torch.float32).to(dtype))
    return out
