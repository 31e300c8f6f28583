"""The decode entry point that allocates nothing (sgdkv_decode_attention_noalloc), on the GPU.

Two calls in a row through the C ABI, the second with a smaller input (fewer sequences, shorter
segments, another dtype and head size), each compared with sgdkv_decode_attention_ex on the same
inputs with a caller workspace: the same kernels with the same split plan, so outputs and LSE are
bitwise equal. The first call also attends to rows appended after compression.
"""
import numpy as np
import pytest
import torch

import paper_2609_03235_amd as sg

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _case(seed, B, Hq, Hkv, d, C, dtype, n_new=0, cap=0):
    rng = np.random.Generator(np.random.PCG64(seed))
    w, s, W = 32, 16, 64
    t = {n: torch.from_numpy(rng.standard_normal(shape).astype(np.float32)).to(dtype).to(DEV)
         for n, shape in dict(q_win=(B, Hq, w, d), k=(B, Hkv, C, d), v=(B, Hkv, C, d), q=(B, Hq, d)).items()}
    budgets = rng.integers(s + W, C + 1, size=Hkv)
    budgets[0] = s + W  # an empty middle
    res = sg.compress_layer(t["q_win"], t["k"], t["v"], budgets, pool_kernel=7, b_sink=s, b_window=W)
    tail = {}
    if cap:
        tail = dict(k_new=torch.from_numpy(rng.standard_normal((B, Hkv, cap, d)).astype(np.float32)).to(dtype).to(DEV),
                    v_new=torch.from_numpy(rng.standard_normal((B, Hkv, cap, d)).astype(np.float32)).to(dtype).to(DEV),
                    n_new=n_new)
    return t, res, tail


def _compare(t, res, tail, Hkv, tag):
    B, Hq, d = t["q"].shape
    ref, ref_lse = sg.decode_attention(t["q"], res["k_c"], res["v_c"], res["offsets"], res["offsets_host"], Hkv,
                                       out_dtype=torch.float32, **tail)
    out = torch.full((B, Hq, d), float("nan"), dtype=torch.float32, device=DEV)
    lse = torch.full((B, Hq), float("nan"), dtype=torch.float32, device=DEV)
    sg.decode_attention(t["q"], res["k_c"], res["v_c"], res["offsets"], res["offsets_host"], Hkv,
                        out_dtype=torch.float32, out=out, lse=lse, no_alloc=True, **tail)
    torch.cuda.synchronize()
    assert torch.isfinite(ref).all()
    assert torch.equal(out, ref), f"{tag}: outputs differ from the workspace entry point"
    assert torch.equal(lse, ref_lse), f"{tag}: lse differs from the workspace entry point"


def test_noalloc_matches_workspace_entry_point_twice():
    print("[gpu case] no-alloc decode: large bf16 call with appended rows", flush=True)
    t, res, tail = _case(3, B=3, Hq=28, Hkv=4, d=128, C=40000, dtype=torch.bfloat16, n_new=37, cap=64)
    _compare(t, res, tail, 4, "first call")
    print("[gpu case] no-alloc decode: smaller fp32 call", flush=True)
    t2, res2, _ = _case(4, B=1, Hq=8, Hkv=2, d=64, C=3000, dtype=torch.float32)
    _compare(t2, res2, {}, 2, "second call")
