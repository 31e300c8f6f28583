"""SGD-KV hot path on AMD Instinct MI355X (gfx950).

Thin ctypes binding over ``libsgdkv.so`` (the C ABI declared in
``include/sgdkv.h``): every step of the path runs in the library's HIP
kernels; this module only converts tensors to pointers, allocates the output
tensors with torch, and passes torch's current stream. If the library is not
built, every call raises -- there is no fallback implementation.

Entry points (same names as the C ABI without the ``sgdkv_`` prefix):
  allocate_budgets, total_from_ratio, reduce_query_head_scores   (host)
  compress_workspace_size, compress_layer                        (device)
  decode_workspace_size, decode_attention                        (device)
"""
from __future__ import annotations

import ctypes
import math
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsgdkv.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = 0, 1, 2, 3, 4
DTYPE_F32, DTYPE_BF16 = 0, 1
SYMBOLS = ("sgdkv_last_error", "sgdkv_version", "sgdkv_reduce_query_head_scores", "sgdkv_total_from_ratio",
           "sgdkv_allocate_budgets", "sgdkv_allocate_budgets_variant", "sgdkv_segment_offsets",
           "sgdkv_compress_workspace_size",
           "sgdkv_compress_layer", "sgdkv_compress_layer_ex",
           "sgdkv_decode_workspace_size", "sgdkv_decode_attention", "sgdkv_decode_workspace_size_ex",
           "sgdkv_decode_attention_ex", "sgdkv_decode_attention_noalloc", "sgdkv_append_kv", "sgdkv_profile_enable",
           "sgdkv_profile_reset", "sgdkv_profile_read")


class SgdkvError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"sgdkv status {status}: {message}")
        self.status = status
        self.message = message


class CompressDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("obs_window", ctypes.c_int32), ("pool_kernel", ctypes.c_int32),
                ("seq_len", ctypes.c_int64), ("b_sink", ctypes.c_int64), ("b_window", ctypes.c_int64),
                ("dtype", ctypes.c_int32), ("scale", ctypes.c_float)]


class CompressOpts(ctypes.Structure):
    _fields_ = [("group_agg", ctypes.c_int32), ("reserved", ctypes.c_int32), ("qhead_scores", ctypes.c_void_p),
                ("window_pos", ctypes.c_int64), ("gather_stream", ctypes.c_void_p)]


class DecodeDesc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("kv_dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32),
                ("scale", ctypes.c_float)]


_lib = None


def load_library():
    """Load libsgdkv.so (after torch, so both share torch's HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() or "
                          "python paper_2609_03235_amd/build.py")
    try:
        import torch  # noqa: F401  -- binds the HIP runtime torch ships before ours resolves it
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.sgdkv_last_error.restype = ctypes.c_char_p
    lib.sgdkv_last_error.argtypes = []
    lib.sgdkv_version.restype = i32
    lib.sgdkv_version.argtypes = []
    sigs = {
        "sgdkv_reduce_query_head_scores": [P, i32, i32, i32, P],
        "sgdkv_total_from_ratio": [f64, i32, i32, i64, i64, i64, i32, P],
        "sgdkv_allocate_budgets": [P, i32, i32, i64, i64, i64, i64, i32, P],
        "sgdkv_allocate_budgets_variant": [P, P, i32, i32, i64, i64, i64, i64, i32, i32, f64, P],
        "sgdkv_segment_offsets": [P, i32, i32, P],
        "sgdkv_compress_workspace_size": [P, P],
        "sgdkv_compress_layer": [P, P, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P],
        "sgdkv_compress_layer_ex": [P, P, P, P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P],
        "sgdkv_decode_workspace_size": [P, P, P],
        "sgdkv_decode_attention": [P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P],
        "sgdkv_decode_workspace_size_ex": [P, P, i64, P],
        "sgdkv_decode_attention_ex": [P, P, P, P, P, P, P, P, P, P, ctypes.c_size_t, P],
        "sgdkv_decode_attention_noalloc": [P, P, P, P, P, P, P, P, P, P],
        "sgdkv_append_kv": [P, P, P, P, P, i64, i64, P],
        "sgdkv_profile_enable": [i32],
        "sgdkv_profile_reset": [],
        "sgdkv_profile_read": [i32, P, P, P, P],
    }
    for name, args in sigs.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = i32
    _lib = lib
    return lib


def _check(status: int):
    if status != OK:
        raise SgdkvError(status, load_library().sgdkv_last_error().decode())


def version() -> int:
    return int(load_library().sgdkv_version())


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


# ------------------------------------------------------------------ host
def reduce_query_head_scores(per_qhead, num_kv_heads: int) -> np.ndarray:
    a = np.ascontiguousarray(np.asarray(per_qhead, dtype=np.float64))
    L, Hq = a.shape
    out = np.zeros((L, num_kv_heads), dtype=np.float64)
    _check(load_library().sgdkv_reduce_query_head_scores(_np_ptr(a), L, Hq, num_kv_heads, _np_ptr(out)))
    return out


def total_from_ratio(R: float, L: int, H: int, C: int, b_sink: int, b_window: int, of_middle: int = 0) -> int:
    t = ctypes.c_int64(0)
    _check(load_library().sgdkv_total_from_ratio(float(R), L, H, C, b_sink, b_window, int(of_middle),
                                                 ctypes.byref(t)))
    return int(t.value)


def allocate_budgets(scores, L: int, H: int, C: int, b_sink: int, b_window: int, total: int,
                     mode: int = 0) -> np.ndarray:
    sc = np.ascontiguousarray(np.asarray(scores, dtype=np.float64).reshape(-1))
    if sc.size != L * H:
        raise SgdkvError(ERR_INVALID_ARG, "scores must hold L*H values")
    out = np.zeros(L * H, dtype=np.int64)
    _check(load_library().sgdkv_allocate_budgets(_np_ptr(sc), L, H, C, b_sink, b_window, int(total), int(mode),
                                                 _np_ptr(out)))
    return out


ALLOC_PLAIN, ALLOC_THR, ALLOC_REVERSE, ALLOC_MIX, ALLOC_BINARY, ALLOC_BINARY_REVERSE = range(6)


def allocate_budgets_variant(scores, L: int, H: int, C: int, b_sink: int, b_window: int, total: int,
                             variant: int, mode: int = 0, scores2=None, full_fraction: float = 0.0) -> np.ndarray:
    sc = np.ascontiguousarray(np.asarray(scores, dtype=np.float64).reshape(-1))
    if sc.size != L * H:
        raise SgdkvError(ERR_INVALID_ARG, "scores must hold L*H values")
    s2 = None
    if scores2 is not None:
        s2 = np.ascontiguousarray(np.asarray(scores2, dtype=np.float64).reshape(-1))
        if s2.size != L * H:
            raise SgdkvError(ERR_INVALID_ARG, "scores2 must hold L*H values")
    out = np.zeros(L * H, dtype=np.int64)
    _check(load_library().sgdkv_allocate_budgets_variant(
        _np_ptr(sc), _np_ptr(s2) if s2 is not None else None, L, H, C, b_sink, b_window, int(total), int(mode),
        int(variant), float(full_fraction), _np_ptr(out)))
    return out


def segment_offsets(layer_budgets, batch: int) -> np.ndarray:
    """Host copy of the ragged cache's row offsets [batch * Hkv + 1] for one layer's budgets
    (sgdkv_segment_offsets): the values compress_layer writes to its device offsets."""
    bud = np.ascontiguousarray(np.asarray(layer_budgets, dtype=np.int64).reshape(-1))
    out = np.zeros(int(batch) * bud.size + 1, dtype=np.int64)
    _check(load_library().sgdkv_segment_offsets(_np_ptr(bud), int(batch), bud.size, _np_ptr(out)))
    return out


# ---------------------------------------------------------------- device
def _dtype_code(t) -> int:
    import torch
    if t.dtype == torch.bfloat16:
        return DTYPE_BF16
    if t.dtype == torch.float32:
        return DTYPE_F32
    raise SgdkvError(ERR_INVALID_ARG, f"unsupported dtype {t.dtype}")


def _ptr(t):
    if t is None:
        return None
    if not t.is_contiguous():
        raise SgdkvError(ERR_INVALID_ARG, "tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def compress_desc(q_win, k, *, obs_window=None, pool_kernel: int, b_sink: int, b_window: int,
                  scale: float = 0.0) -> CompressDesc:
    B, Hq, w, d = q_win.shape
    Bk, Hkv, C, dk = k.shape
    if Bk != B or dk != d or (obs_window is not None and obs_window != w):
        raise SgdkvError(ERR_INVALID_ARG, f"shape mismatch q_win {tuple(q_win.shape)} k {tuple(k.shape)}")
    return CompressDesc(B, Hq, Hkv, d, w, pool_kernel, C, b_sink, b_window, _dtype_code(k), float(scale))


def compress_workspace_size(desc: CompressDesc) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().sgdkv_compress_workspace_size(ctypes.byref(desc), ctypes.byref(n)))
    return int(n.value)


def alloc_workspace(nbytes: int, device):
    """Device workspace as a uint8 tensor (torch's allocator returns 256-byte aligned blocks)."""
    import torch
    ws = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)
    assert ws.data_ptr() % 256 == 0
    return ws


GROUP_MEAN, GROUP_IPT_MAX, GROUP_IPT_MEAN, GROUP_IPT_ONLY = range(4)


def compress_layer(q_win, k, v, layer_budgets, *, pool_kernel: int, b_sink: int, b_window: int,
                   scale: float = 0.0, window_lse=None, scores_only: bool = False, with_scores: bool = True,
                   group_agg: int = GROUP_MEAN, qhead_scores=None, window_pos: int = -1,
                   workspace=None, out: dict | None = None, stream=None, gather_stream=None) -> dict:
    """Compress one layer (sgdkv_compress_layer_ex). group_agg selects the plain group mean or an
    Ipt. aggregation with the layer's per-query-head scores; window_pos places the first window
    row (-1: the last obs_window prompt tokens). gather_stream (optional) takes the copy of the
    kept rows into k_c and v_c, which are then complete only on that stream. Returns k_c, v_c,
    kept_pos, offsets, offsets_host, scores (scores: [B, Hkv, window position]). With gather_stream, the
    tensors the copy reads or writes (k, v, k_c, v_c, kept_pos) are marked as in use on that stream (for a
    torch.cuda.Stream; a raw stream handle leaves keeping them alive to the caller), so torch's allocator
    does not hand their memory to other work before the copy is done."""
    import torch
    desc = compress_desc(q_win, k, pool_kernel=pool_kernel, b_sink=b_sink, b_window=b_window, scale=scale)
    B, Hkv, C, d = k.shape
    dev = k.device
    budgets = None if layer_budgets is None else np.ascontiguousarray(np.asarray(layer_budgets, dtype=np.int64))
    if budgets is not None and budgets.size != Hkv:
        raise SgdkvError(ERR_INVALID_ARG, "layer_budgets must hold num_kv_heads values")
    res = dict(out or {})
    if not scores_only:
        T = int(budgets.sum())
        res.setdefault("k_c", torch.empty((B * T, d), dtype=k.dtype, device=dev))
        res.setdefault("v_c", torch.empty((B * T, d), dtype=v.dtype, device=dev))
        res.setdefault("kept_pos", torch.empty(B * T, dtype=torch.int32, device=dev))
        res.setdefault("offsets", torch.empty(B * Hkv + 1, dtype=torch.int64, device=dev))
        res["offsets_host"] = segment_offsets(budgets, B)
    n_scored = C - q_win.shape[2] if window_pos == -1 else int(window_pos)
    if with_scores or scores_only:
        res.setdefault("scores", torch.empty((B, Hkv, max(n_scored, 0)), dtype=torch.float32, device=dev))
    if workspace is None:
        workspace = alloc_workspace(compress_workspace_size(desc), dev)
    qs = None
    if qhead_scores is not None:
        qs = np.ascontiguousarray(np.asarray(qhead_scores, dtype=np.float64).reshape(-1))
        if qs.size != q_win.shape[1]:
            raise SgdkvError(ERR_INVALID_ARG, "qhead_scores must hold num_q_heads values")
    opts = CompressOpts(int(group_agg), 0, None if qs is None else qs.ctypes.data, int(window_pos),
                        None if gather_stream is None else _stream(gather_stream).value)
    st = load_library().sgdkv_compress_layer_ex(
        ctypes.byref(desc), ctypes.byref(opts), None if budgets is None else _np_ptr(budgets), _ptr(q_win), _ptr(k),
        _ptr(v) if v is not None else None, _ptr(window_lse), _ptr(res.get("k_c")), _ptr(res.get("v_c")),
        _ptr(res.get("kept_pos")), _ptr(res.get("offsets")), _ptr(res.get("scores")), _ptr(workspace),
        workspace.numel(), _stream(stream))
    _check(st)
    if isinstance(gather_stream, torch.cuda.Stream) and not scores_only:
        for t in (k, v, res["k_c"], res["v_c"], res["kept_pos"]):
            t.record_stream(gather_stream)
    return res


def decode_desc(q, num_kv_heads: int, out_dtype=None, scale: float = 0.0) -> DecodeDesc:
    B, Hq, d = q.shape
    od = _dtype_code(q) if out_dtype is None else (DTYPE_BF16 if "bfloat16" in str(out_dtype) else DTYPE_F32)
    return DecodeDesc(B, Hq, num_kv_heads, d, _dtype_code(q), od, float(scale))


def decode_workspace_size(desc: DecodeDesc, offsets_host, capacity: int = 0) -> int:
    oh = np.ascontiguousarray(np.asarray(offsets_host, dtype=np.int64))
    n = ctypes.c_size_t(0)
    _check(load_library().sgdkv_decode_workspace_size_ex(ctypes.byref(desc), _np_ptr(oh), int(capacity),
                                                          ctypes.byref(n)))
    return int(n.value)


class DecodeTail(ctypes.Structure):
    _fields_ = [("k_new", ctypes.c_void_p), ("v_new", ctypes.c_void_p), ("capacity", ctypes.c_int64),
                ("n_new", ctypes.c_int64)]


def decode_attention(q, k_c, v_c, offsets, offsets_host, num_kv_heads: int, *, out_dtype=None,
                     scale: float = 0.0, with_lse: bool = True, k_new=None, v_new=None, n_new: int = 0,
                     workspace=None, out=None, lse=None, stream=None, no_alloc: bool = False):
    """One decode step over the ragged cache (sgdkv_decode_attention_ex). k_new/v_new [B, Hkv, capacity, d]
    hold the rows appended since compression, of which the first n_new are attended. no_alloc: call
    sgdkv_decode_attention_noalloc instead, which takes no workspace (its split partials go to the
    library's static device scratch; pass out, and lse if wanted, to allocate nothing here either).
    Returns (out, lse)."""
    import torch
    desc = decode_desc(q, num_kv_heads, out_dtype, scale)
    oh = np.ascontiguousarray(np.asarray(offsets_host, dtype=np.int64))
    B, Hq, d = q.shape
    cap = 0 if k_new is None else int(k_new.shape[2])
    if out is None:
        out = torch.empty((B, Hq, d), dtype=torch.bfloat16 if desc.out_dtype == DTYPE_BF16 else torch.float32,
                          device=q.device)
    if with_lse and lse is None:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=q.device)
    tail = DecodeTail(_ptr(k_new), _ptr(v_new), cap, int(n_new))
    if no_alloc:
        _check(load_library().sgdkv_decode_attention_noalloc(
            ctypes.byref(desc), _ptr(q), _ptr(k_c), _ptr(v_c), _ptr(offsets), _np_ptr(oh), ctypes.byref(tail),
            _ptr(out), _ptr(lse) if with_lse else None, _stream(stream)))
        return out, (lse if with_lse else None)
    if workspace is None:
        workspace = alloc_workspace(decode_workspace_size(desc, oh, cap), q.device)
    st = load_library().sgdkv_decode_attention_ex(
        ctypes.byref(desc), _ptr(q), _ptr(k_c), _ptr(v_c), _ptr(offsets), _np_ptr(oh), ctypes.byref(tail), _ptr(out),
        _ptr(lse) if with_lse else None, _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st)
    return out, (lse if with_lse else None)


def append_kv(q_like, k_step, v_step, k_new, v_new, slot: int, stream=None):
    """Write one generated token's K/V rows [B, Hkv, d] into row `slot` of k_new/v_new [B, Hkv, capacity, d]
    (sgdkv_append_kv). q_like: the decode queries [B, Hq, d] (for the descriptor)."""
    desc = decode_desc(q_like, k_step.shape[1])
    _check(load_library().sgdkv_append_kv(ctypes.byref(desc), _ptr(k_step), _ptr(v_step), _ptr(k_new), _ptr(v_new),
                                          int(k_new.shape[2]), int(slot), _stream(stream)))


# ------------------------------------------------------- kernel timing
def profile_enable(on: bool = True):
    _check(load_library().sgdkv_profile_enable(1 if on else 0))


def profile_reset():
    _check(load_library().sgdkv_profile_reset())


def profile_read(max_entries: int = 64) -> dict:
    """{kernel name: (launches, total ms)} since the last reset (waits for pending events)."""
    names = ctypes.create_string_buffer(max_entries * 64)
    counts = np.zeros(max_entries, dtype=np.int64)
    ms = np.zeros(max_entries, dtype=np.float64)
    n = ctypes.c_int32(0)
    _check(load_library().sgdkv_profile_read(max_entries, names, _np_ptr(counts), _np_ptr(ms), ctypes.byref(n)))
    out = {}
    for i in range(min(n.value, max_entries)):
        name = names.raw[i * 64:(i + 1) * 64].split(b"\0", 1)[0].decode()
        out[name] = (int(counts[i]), float(ms[i]))
    return out
