"""SGD-KV CPU oracle -- test infrastructure only.

A thin ctypes wrapper over ``sgdkv_oracle.c``: plain fp64 C that computes
what the SGD-KV hot path computes, step by step, straight from the paper's
definitions (Sec. 3.3 with Eq. 2, Appendix A.1 Algorithm 1, Appendix A.2 and
A.7, Sec. 5). Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU
baseline leg of ``bench.py`` may import this package. It shares no code with
the HIP product path and never imports it.

End-to-end outputs are *parity unpinned* against the paper, which prints no
numeric worked example of the hot path; each step is pinned separately by
the ``-m "not gpu"`` tests (closed forms, invariants, brute force, library
routines).
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "sgdkv_oracle.c")
DEFAULT_LIB_PATH = os.path.join(_HERE, "libsgdkv_oracle.so")
# The mutation test points this at deliberately broken builds of the oracle.
LIB_PATH = os.environ.get("SGDKV_ORACLE_LIB", DEFAULT_LIB_PATH)

_lib = None


GCC_FLAGS = ["-O2", "-fopenmp", "-ffp-contract=off", "-fno-fast-math", "-std=c11", "-Wall",
             "-shared", "-fPIC"]


def build(force: bool = True, src: str = SRC, out: str = DEFAULT_LIB_PATH) -> str:
    """Compile the oracle with gcc (fp64, OpenMP, no FP contraction)."""
    if force or not os.path.exists(out):
        tmp = out + ".tmp"
        subprocess.run(["gcc", *GCC_FLAGS, src, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, out)
    return out


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        build(force=False)
    lib = ctypes.CDLL(LIB_PATH)
    i32, i64, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_double
    P = ctypes.c_void_p
    lib.orc_reduce_group_max.argtypes = [P, i32, i32, i32, P]
    lib.orc_total_from_ratio.argtypes = [f64, i32, i32, i64, i64, i64, i32, P]
    lib.orc_allocate_budgets.argtypes = [P, i32, i32, i64, i64, i64, i64, i32, P]
    lib.orc_allocate_variant.argtypes = [P, P, i32, i32, i64, i64, i64, i64, i32, i32, f64, P]
    lib.orc_window_lse.argtypes = [P, P, i32, i32, i32, i32, i64, i32, i64, f64, P]
    lib.orc_window_colsum.argtypes = [P, P, P, i32, i32, i32, i32, i64, i32, i64, f64, P]
    lib.orc_window_colsum_ipt.argtypes = [P, P, P, i32, i32, i32, i32, i64, i32, i64, f64, P, i32, P]
    lib.orc_pool.argtypes = [P, i64, i64, i32, P]
    lib.orc_select.argtypes = [P, i64, i64, i64, i64, i64, P]
    lib.orc_decode.argtypes = [P, P, P, P, i32, i32, i32, i32, f64, P, P]
    lib.orc_decode_append.argtypes = [P, P, P, P, P, P, i64, i64, i32, i32, i32, i32, f64, P, P]
    lib.orc_num_threads.argtypes = []
    for f in ("orc_reduce_group_max", "orc_total_from_ratio", "orc_allocate_budgets", "orc_allocate_variant",
              "orc_window_lse", "orc_window_colsum", "orc_window_colsum_ipt", "orc_pool", "orc_select", "orc_decode", "orc_decode_append",
              "orc_num_threads"):
        getattr(lib, f).restype = i32
    _lib = lib
    return lib


class OracleError(ValueError):
    pass


def _f64(a) -> np.ndarray:
    """Exact fp64 copy of a numpy array or a CPU torch tensor (bf16/fp32 upcast exactly)."""
    if hasattr(a, "detach"):
        a = a.detach().cpu().double().numpy()
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError(f"oracle {what}: invalid arguments")


def num_threads() -> int:
    return int(_load().orc_num_threads())


def set_num_threads(n: int) -> None:
    """OpenMP threads of the oracle's later calls from this thread (its libgomp is the process's)."""
    _load()
    ctypes.CDLL("libgomp.so.1").omp_set_num_threads(int(n))


# --------------------------------------------------------------- allocation
def reduce_group_max(per_q, num_kv_heads: int) -> np.ndarray:
    """[L, Hq] per-query-head scores -> [L, Hkv], max over each group (Appendix A.7)."""
    a = _f64(per_q)
    L, Hq = a.shape
    out = np.zeros((L, num_kv_heads), dtype=np.float64)
    _check(_load().orc_reduce_group_max(_ptr(a), L, Hq, num_kv_heads, _ptr(out)), "reduce_group_max")
    return out


def total_from_ratio(R: float, L: int, H: int, C: int, s: int, W: int, of_middle: int = 0) -> int:
    """Total kept rows for ratio R (of all rows, or of the middle as in Eq. 2)."""
    t = ctypes.c_int64(0)
    _check(_load().orc_total_from_ratio(float(R), L, H, C, s, W, int(of_middle), ctypes.byref(t)),
           "total_from_ratio")
    return int(t.value)


def allocate_budgets(scores, L: int, H: int, C: int, s: int, W: int, total: int,
                     mode: int = 0) -> np.ndarray:
    """Per-KV-head budgets b_h (Eq. 2 + Algorithm 1), int64 [L*H], layer-major."""
    sc = _f64(scores).reshape(-1)
    if sc.size != L * H:
        raise OracleError("scores must hold L*H values")
    out = np.zeros(L * H, dtype=np.int64)
    _check(_load().orc_allocate_budgets(_ptr(sc), L, H, C, s, W, int(total), int(mode), _ptr(out)),
           "allocate_budgets")
    return out


ALLOC_PLAIN, ALLOC_THR, ALLOC_REVERSE, ALLOC_MIX, ALLOC_BINARY, ALLOC_BINARY_REVERSE = range(6)


def allocate_variant(scores, L: int, H: int, C: int, s: int, W: int, total: int, variant: int,
                     mode: int = 0, scores2=None, full_fraction: float = 0.0) -> np.ndarray:
    """Allocation variants of the head-configuration ablation (Appendix A.7, Table 5)."""
    sc = _f64(scores).reshape(-1)
    if sc.size != L * H:
        raise OracleError("scores must hold L*H values")
    s2 = None if scores2 is None else _f64(scores2).reshape(-1)
    if s2 is not None and s2.size != L * H:
        raise OracleError("scores2 must hold L*H values")
    out = np.zeros(L * H, dtype=np.int64)
    _check(_load().orc_allocate_variant(_ptr(sc), _ptr(s2) if s2 is not None else None, L, H, C, s, W,
                                        int(total), int(mode), int(variant), ctypes.c_double(full_fraction),
                                        _ptr(out)), "allocate_variant")
    return out


# ------------------------------------------------------------------ scores
def _scale(d: int, scale):
    return 1.0 / math.sqrt(d) if scale is None or scale == 0 else float(scale)


def _win0(C: int, w: int, win0):
    return C - w if win0 is None else int(win0)


def window_lse(q_win, k, num_kv_heads: int | None = None, scale=None, win0=None) -> np.ndarray:
    """LSE of each observation-window row over its causal keys; [B, Hq, w]. Row i sits at position
    win0 + i (default C - w: the last w prompt tokens)."""
    q = _f64(q_win)
    kk = _f64(k)
    B, Hq, w, d = q.shape
    _, Hkv, C, _ = kk.shape
    out = np.zeros((B, Hq, w), dtype=np.float64)
    _check(_load().orc_window_lse(_ptr(q), _ptr(kk), B, Hq, Hkv, d, C, w, _win0(C, w, win0), _scale(d, scale),
                                  _ptr(out)), "window_lse")
    return out


GROUP_MEAN, GROUP_IPT_MAX, GROUP_IPT_MEAN, GROUP_IPT_ONLY = range(4)


def window_colsum(q_win, k, lse, scale=None, agg: int = GROUP_MEAN, qhead_scores=None, win0=None) -> np.ndarray:
    """Cumulative window attention of each scored key (keys before the window, [0, win0)),
    aggregated over the query group (the plain mean, or an importance-weighted Ipt. variant,
    Appendix A.7); [B, Hkv, win0]."""
    q = _f64(q_win)
    kk = _f64(k)
    ls = _f64(lse)
    B, Hq, w, d = q.shape
    _, Hkv, C, _ = kk.shape
    p0 = _win0(C, w, win0)
    if not 0 <= p0 <= C:
        raise OracleError("win0 outside [0, C]")
    out = np.zeros((B, Hkv, p0), dtype=np.float64)
    if agg == GROUP_MEAN:
        _check(_load().orc_window_colsum(_ptr(q), _ptr(kk), _ptr(ls), B, Hq, Hkv, d, C, w, p0,
                                         _scale(d, scale), _ptr(out)), "window_colsum")
        return out
    qs = _f64(qhead_scores).reshape(-1)
    if qs.size != Hq:
        raise OracleError("qhead_scores must hold Hq values")
    _check(_load().orc_window_colsum_ipt(_ptr(q), _ptr(kk), _ptr(ls), B, Hq, Hkv, d, C, w, p0, _scale(d, scale),
                                         _ptr(qs), int(agg), _ptr(out)), "window_colsum_ipt")
    return out


def pool(a, kp: int) -> np.ndarray:
    """Average pooling along the last axis (odd kernel, stride 1, zero padding)."""
    x = _f64(a)
    n = x.shape[-1]
    rows = int(np.prod(x.shape[:-1])) if x.ndim > 1 else 1
    out = np.zeros_like(x)
    _check(_load().orc_pool(_ptr(x), rows, n, kp, _ptr(out)), "pool")
    return out


def select(pooled_row, C: int, w: int, s: int, W: int, m: int, win0=None) -> np.ndarray:
    """Kept positions of one head, ascending: sink, top-m candidates, window. The row holds the
    scores of keys [0, win0) (default C - w)."""
    p = _f64(pooled_row).reshape(-1)
    n = _win0(C, w, win0)
    if p.size != n:
        raise OracleError("pooled row must hold one score per key before the window")
    out = np.zeros(s + m + W, dtype=np.int32)
    _check(_load().orc_select(_ptr(p), C, n, s, W, m, _ptr(out)), "select")
    return out


# -------------------------------------------------------------- full steps
def compress(q_win, k, v, budgets, *, w: int, kp: int, s: int, W: int, scale=None,
             lse=None, agg: int = GROUP_MEAN, qhead_scores=None, win0=None) -> dict:
    """One layer's compression: scores, pooling, per-head selection and gather.

    budgets: [Hkv] int (the layer's rows per KV head, shared by every sequence).
    win0: position of the first window row (default C - w; see window_lse).
    Returns kept_pos [B*T] int32, offsets [B*Hkv+1] int64, k_c/v_c [B*T, d] fp64
    (exact copies of the input rows), colsum/pooled [B, Hkv, win0], lse [B, Hq, w].
    """
    q = _f64(q_win)
    kk = _f64(k)
    vv = _f64(v)
    B, Hq, w_, d = q.shape
    _, Hkv, C, _ = kk.shape
    assert w_ == w
    budgets = np.asarray(budgets, dtype=np.int64).reshape(-1)
    assert budgets.size == Hkv
    if lse is None:
        lse = window_lse(q, kk, scale=scale, win0=win0)
    colsum = window_colsum(q, kk, lse, scale=scale, agg=agg, qhead_scores=qhead_scores, win0=win0)
    pooled = pool(colsum, kp)
    T = int(budgets.sum())
    kept = np.zeros(B * T, dtype=np.int32)
    offsets = np.zeros(B * Hkv + 1, dtype=np.int64)
    k_c = np.zeros((B * T, d), dtype=np.float64)
    v_c = np.zeros((B * T, d), dtype=np.float64)
    row = 0
    for b in range(B):
        for h in range(Hkv):
            offsets[b * Hkv + h] = row
            m = int(budgets[h]) - s - W
            pos = select(pooled[b, h], C, w, s, W, m, win0=win0)
            n = pos.size
            kept[row:row + n] = pos
            k_c[row:row + n] = kk[b, h, pos]
            v_c[row:row + n] = vv[b, h, pos]
            row += n
    offsets[B * Hkv] = row
    return dict(kept_pos=kept, offsets=offsets, k_c=k_c, v_c=v_c, colsum=colsum, pooled=pooled,
                lse=lse)


def decode_append(q, k_c, v_c, offsets, k_new, v_new, n_new: int, num_kv_heads: int, scale=None):
    """Decode over each segment's compressed rows plus rows 0..n_new-1 of k_new/v_new
    [B, Hkv, capacity, d] (the tokens appended since compression): (out [B,Hq,d], lse [B,Hq])."""
    qq = _f64(q)
    kc = _f64(k_c)
    vc = _f64(v_c)
    kn = _f64(k_new)
    vn = _f64(v_new)
    off = np.ascontiguousarray(np.asarray(offsets, dtype=np.int64))
    B, Hq, d = qq.shape
    cap = kn.shape[2]
    out = np.zeros((B, Hq, d), dtype=np.float64)
    lse = np.zeros((B, Hq), dtype=np.float64)
    _check(_load().orc_decode_append(_ptr(qq), _ptr(kc), _ptr(vc), _ptr(off), _ptr(kn), _ptr(vn), cap, int(n_new),
                                     B, Hq, num_kv_heads, d, _scale(d, scale), _ptr(out), _ptr(lse)),
           "decode_append")
    return out, lse


def decode(q, k_c, v_c, offsets, num_kv_heads: int, scale=None):
    """Decode attention over the ragged per-KV-head cache: (out [B,Hq,d], lse [B,Hq])."""
    qq = _f64(q)
    kc = _f64(k_c)
    vc = _f64(v_c)
    off = np.ascontiguousarray(np.asarray(offsets, dtype=np.int64))
    B, Hq, d = qq.shape
    out = np.zeros((B, Hq, d), dtype=np.float64)
    lse = np.zeros((B, Hq), dtype=np.float64)
    _check(_load().orc_decode(_ptr(qq), _ptr(kc), _ptr(vc), _ptr(off), B, Hq, num_kv_heads, d,
                              _scale(d, scale), _ptr(out), _ptr(lse)), "decode")
    return out, lse
