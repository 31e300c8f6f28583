"""Host-side tests of the C ABI (no GPU needed).

* the library loads and exports every function include/sgdkv.h declares;
* budget allocation (host code) is bit-exact against the oracle;
* every validation error returns its status before any device work, and
  leaves host outputs untouched;
* without a usable GPU, well-formed compress/decode calls fail with
  SGDKV_ERR_HIP only after validation passed.
"""
import ctypes
import os
import re

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
import paper_2609_03235_amd as sg

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _gpu():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


def test_exports_every_declared_symbol():
    header = open(os.path.join(ROOT, "include", "sgdkv.h")).read()
    declared = set(re.findall(r"^\s*(?:sgdkv_status|const char\*|int32_t)\s+(sgdkv_\w+)\(", header, re.M))
    assert declared == set(sg.SYMBOLS)
    lib = sg.load_library()
    for name in declared:
        assert hasattr(lib, name), name
    assert sg.version() == 102


problem = st.integers(min_value=1, max_value=4).flatmap(
    lambda L: st.integers(min_value=1, max_value=8).flatmap(
        lambda H: st.tuples(
            st.just(L), st.just(H),
            st.lists(st.one_of(st.floats(0.0, 1.0), st.floats(0.0, 1e6), st.sampled_from([0.0, 0.5, 1.0])),
                     min_size=L * H, max_size=L * H),
            st.integers(1, 5000), st.integers(0, 64), st.integers(0, 64), st.floats(0.0, 1.0))))


@settings(max_examples=400, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(problem, st.sampled_from([0, 1]))
def test_allocation_bit_exact_vs_oracle(p, mode):
    L, H, scores, C, s, W, frac = p
    if s + W > C:
        return
    n = L * H
    total = n * (s + W) + int(frac * n * (C - s - W))
    got = sg.allocate_budgets(scores, L, H, C, s, W, total, mode)
    ref = oracle.allocate_budgets(np.array(scores), L, H, C, s, W, total, mode)
    assert np.array_equal(got, ref)


def test_allocation_workload_tables_bit_exact():
    import workloads
    for wl in workloads.WORKLOADS.values():
        sc = workloads.head_scores(wl)
        for R in wl.ratios:
            for of_middle in (0, 1):
                t_lib = sg.total_from_ratio(R, wl.layers, wl.num_kv_heads, wl.seq_len, wl.b_sink, wl.b_window,
                                            of_middle)
                t_orc = oracle.total_from_ratio(R, wl.layers, wl.num_kv_heads, wl.seq_len, wl.b_sink,
                                                wl.b_window, of_middle)
                assert t_lib == t_orc
                for mode in (0, 1):
                    got = sg.allocate_budgets(sc, wl.layers, wl.num_kv_heads, wl.seq_len, wl.b_sink,
                                              wl.b_window, t_lib, mode)
                    ref = oracle.allocate_budgets(sc, wl.layers, wl.num_kv_heads, wl.seq_len, wl.b_sink,
                                                  wl.b_window, t_orc, mode)
                    assert np.array_equal(got, ref), (wl.key, R, mode)


def test_reduce_query_head_scores_matches_oracle():
    rng = np.random.Generator(np.random.PCG64(4))
    per_q = rng.random((28, 28))
    assert np.array_equal(sg.reduce_query_head_scores(per_q, 4), oracle.reduce_group_max(per_q, 4))


def test_allocation_errors_leave_output_untouched():
    lib = sg.load_library()
    out = np.full(4, -7, dtype=np.int64)
    P = sg._np_ptr
    bad = [
        (np.array([0.1, -1.0, 0.2, 0.3]), 1, 4, 100, 2, 2, 50, 0),
        (np.array([0.1, np.inf, 0.2, 0.3]), 1, 4, 100, 2, 2, 50, 0),
        (np.array([0.1, np.nan, 0.2, 0.3]), 1, 4, 100, 2, 2, 50, 0),
        (np.array([0.1, 0.1, 0.2, 0.3]), 1, 4, 100, 2, 2, 15, 0),   # below 4*(2+2)
        (np.array([0.1, 0.1, 0.2, 0.3]), 1, 4, 100, 2, 2, 401, 0),  # above 4*100
        (np.array([0.1, 0.1, 0.2, 0.3]), 1, 4, 100, 60, 60, 300, 0),  # s+W > C
        (np.array([0.1, 0.1, 0.2, 0.3]), 1, 4, 100, 2, 2, 50, 2),   # mode
        (np.array([0.1, 0.1, 0.2, 0.3]), 0, 4, 100, 2, 2, 50, 0),   # L
    ]
    for sc, L, H, C, s, W, total, mode in bad:
        rc = lib.sgdkv_allocate_budgets(P(np.ascontiguousarray(sc)), L, H, C, s, W, total, mode, P(out))
        assert rc == sg.ERR_INVALID_ARG, (sc, L, H, C, s, W, total, mode)
        assert lib.sgdkv_last_error()
        assert np.all(out == -7)
    assert lib.sgdkv_allocate_budgets(None, 1, 4, 100, 2, 2, 50, 0, P(out)) == sg.ERR_INVALID_ARG
    with pytest.raises(sg.SgdkvError):
        sg.total_from_ratio(1.5, 1, 4, 100, 2, 2)


@settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(problem, st.sampled_from([0, 1]), st.integers(0, 5), st.floats(0.0, 1.0),
       st.lists(st.one_of(st.floats(0.0, 1.0), st.sampled_from([0.0, 1.0])), min_size=32, max_size=32))
def test_allocation_variants_bit_exact_vs_oracle(p, mode, variant, f, second):
    L, H, scores, C, s, W, frac = p
    if s + W > C:
        return
    n = L * H
    total = n * (s + W) + int(frac * n * (C - s - W))
    sc2 = np.array(second[:n])
    got = sg.allocate_budgets_variant(scores, L, H, C, s, W, total, variant, mode=mode, scores2=sc2,
                                      full_fraction=f)
    ref = oracle.allocate_variant(np.array(scores), L, H, C, s, W, total, variant, mode=mode, scores2=sc2,
                                  full_fraction=f)
    assert np.array_equal(got, ref)


def test_allocation_variant_workloads_bit_exact():
    import workloads
    for wl in workloads.WORKLOADS.values():
        sc = workloads.head_scores(wl)
        sc2 = np.random.Generator(np.random.PCG64(7)).random(sc.size)  # stand-in for R2 scores
        n = sc.size
        for R in wl.ratios:
            total = sg.total_from_ratio(R, wl.layers, wl.num_kv_heads, wl.seq_len, wl.b_sink, wl.b_window)
            for v in range(6):
                args = (sc, wl.layers, wl.num_kv_heads, wl.seq_len, wl.b_sink, wl.b_window, total, v)
                kw = dict(scores2=sc2, full_fraction=0.25)
                got = sg.allocate_budgets_variant(*args, **kw)
                assert np.array_equal(got, oracle.allocate_variant(*args, **kw)), (wl.key, R, v)
                if v == sg.ALLOC_BINARY:
                    assert int((got == wl.seq_len).sum()) == n // 4


def test_allocation_variant_errors_leave_output_untouched():
    lib = sg.load_library()
    out = np.full(4, -7, dtype=np.int64)
    P = sg._np_ptr
    sc = np.array([0.1, 0.4, 0.2, 0.3])
    bad = [
        (sc, None, 100, 2, 2, 50, 0, sg.ALLOC_MIX, 0.0),                             # no second vector
        (sc, np.array([0.1, -1.0, 0.2, 0.3]), 100, 2, 2, 50, 0, sg.ALLOC_MIX, 0.0),  # bad second vector
        (sc, None, 100, 2, 2, 50, 0, sg.ALLOC_BINARY, 1.5),                          # fraction
        (sc, None, 100, 2, 2, 50, 0, sg.ALLOC_BINARY_REVERSE, -0.1),
        (sc, None, 100, 2, 2, 50, 0, 6, 0.0),                                        # variant
        (sc, None, 100, 2, 2, 15, 0, sg.ALLOC_REVERSE, 0.0),                         # total below the reserve
        (sc, None, 100, 2, 2, 50, 3, sg.ALLOC_THR, 0.0),                             # mode
        (np.array([0.1, np.nan, 0.2, 0.3]), None, 100, 2, 2, 50, 0, sg.ALLOC_BINARY, 0.5),
    ]
    for sc1, sc2, C, s, W, total, mode, variant, f in bad:
        sc2p = P(np.ascontiguousarray(sc2)) if sc2 is not None else None
        rc = lib.sgdkv_allocate_budgets_variant(P(np.ascontiguousarray(sc1)), sc2p, 1, 4, C, s, W, total, mode,
                                                variant, f, P(out))
        assert rc == sg.ERR_INVALID_ARG, (variant, f, total, mode)
        assert lib.sgdkv_last_error()
        assert np.all(out == -7)


FAKE = 0x7F0000000000  # 256-aligned stand-in device address; validation never dereferences it


def _desc(**kw):
    base = dict(batch=1, num_q_heads=4, num_kv_heads=2, head_dim=64, obs_window=32, pool_kernel=7,
                seq_len=2048, b_sink=4, b_window=32, dtype=sg.DTYPE_F32, scale=0.0)
    base.update(kw)
    return sg.CompressDesc(**base)


def _compress(desc, budgets, ptrs=None, ws_bytes=None, ws=FAKE):
    lib = sg.load_library()
    ptrs = {**dict(q_win=FAKE, k=FAKE, v=FAKE, lse=None, k_out=FAKE, v_out=FAKE, kept=FAKE, offsets=FAKE,
                   scores=FAKE), **(ptrs or {})}
    need = ctypes.c_size_t(0)
    lib.sgdkv_compress_workspace_size(ctypes.byref(desc), ctypes.byref(need))
    b = None if budgets is None else np.ascontiguousarray(np.asarray(budgets, dtype=np.int64))
    return lib.sgdkv_compress_layer(
        ctypes.byref(desc), None if b is None else sg._np_ptr(b), ptrs["q_win"], ptrs["k"], ptrs["v"],
        ptrs["lse"], ptrs["k_out"], ptrs["v_out"], ptrs["kept"], ptrs["offsets"], ptrs["scores"], ws,
        need.value if ws_bytes is None else ws_bytes, None)


def test_compress_validation():
    good = [512, 512]
    cases = [
        (_desc(batch=0), good, None, None, sg.ERR_INVALID_ARG),
        (_desc(num_q_heads=5), good, None, None, sg.ERR_INVALID_ARG),
        (_desc(head_dim=96), good, None, None, sg.ERR_UNSUPPORTED),
        (_desc(pool_kernel=4), good, None, None, sg.ERR_INVALID_ARG),
        (_desc(b_window=16), good, None, None, sg.ERR_INVALID_ARG),          # W < w
        (_desc(b_sink=2000, b_window=100), good, None, None, sg.ERR_INVALID_ARG),
        (_desc(num_q_heads=64, num_kv_heads=2, obs_window=160, b_window=160), good, None, None,
         sg.ERR_UNSUPPORTED),                                                  # G*w = 5120 > 4096
        (_desc(num_kv_heads=65, num_q_heads=65), [512] * 65, None, None, sg.ERR_UNSUPPORTED),
        (_desc(dtype=5), good, None, None, sg.ERR_INVALID_ARG),
        (_desc(scale=-1.0), good, None, None, sg.ERR_INVALID_ARG),
        (_desc(), [35, 512], None, None, sg.ERR_INVALID_ARG),                  # budget < s+W
        (_desc(), [512, 2049], None, None, sg.ERR_INVALID_ARG),                # budget > C
        (_desc(), None, None, None, sg.ERR_INVALID_ARG),                       # budgets needed
        (_desc(), good, dict(k_out=None), None, sg.ERR_INVALID_ARG),           # partial outputs
        (_desc(), good, dict(k_out=None, v_out=None, kept=None, offsets=None, scores=None), None,
         sg.ERR_INVALID_ARG),                                                  # scores-only needs scores
        (_desc(), good, dict(q_win=FAKE + 4), None, sg.ERR_INVALID_ARG),       # misaligned
        (_desc(), good, dict(k=None), None, sg.ERR_INVALID_ARG),
        (_desc(), good, None, 16, sg.ERR_WORKSPACE),                            # small workspace
    ]
    for desc, budgets, ptrs, ws_bytes, want in cases:
        assert _compress(desc, budgets, ptrs, ws_bytes) == want, (desc.__dict__ if hasattr(desc, "__dict__") else desc)
        assert sg.load_library().sgdkv_last_error()
    assert _compress(_desc(), good, ws=FAKE + 16) == sg.ERR_WORKSPACE  # misaligned workspace
    assert _compress(_desc(), good, ws=None) == sg.ERR_WORKSPACE


def _compress_ex(desc, agg, qs, budgets=(512, 512), window_pos=-1, reserved=0, gather_stream=None):
    lib = sg.load_library()
    need = ctypes.c_size_t(0)
    lib.sgdkv_compress_workspace_size(ctypes.byref(desc), ctypes.byref(need))
    b = np.ascontiguousarray(np.asarray(budgets, dtype=np.int64))
    q = None if qs is None else np.ascontiguousarray(np.asarray(qs, dtype=np.float64))
    opts = sg.CompressOpts(agg, reserved, None if q is None else q.ctypes.data, window_pos, gather_stream)
    return lib.sgdkv_compress_layer_ex(
        ctypes.byref(desc), ctypes.byref(opts), sg._np_ptr(b), FAKE, FAKE, FAKE, None,
        FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need.value, None)


def test_compress_options_validation():
    four = [0.5, 0.2, 0.1, 0.9]  # the default descriptor has 4 query heads
    cases = [
        (_desc(), 4, four, -1, sg.ERR_INVALID_ARG, "group"),                   # unknown aggregation
        (_desc(), -1, four, -1, sg.ERR_INVALID_ARG, "group"),
        (_desc(), sg.GROUP_IPT_MAX, None, -1, sg.ERR_INVALID_ARG, "qhead"),    # scores needed
        (_desc(), sg.GROUP_IPT_MEAN, [0.5, -0.2, 0.1, 0.9], -1, sg.ERR_INVALID_ARG, "qhead"),
        (_desc(), sg.GROUP_IPT_ONLY, [0.5, np.nan, 0.1, 0.9], -1, sg.ERR_INVALID_ARG, "qhead"),
        (_desc(obs_window=20), sg.GROUP_IPT_MAX, four, -1, sg.ERR_UNSUPPORTED, "Ipt"),  # w % 16
        (_desc(num_q_heads=2, obs_window=528, b_window=528), sg.GROUP_IPT_MAX, [0.5, 0.2], -1,
         sg.ERR_UNSUPPORTED, "Ipt"),                                           # one head beyond a split
        (_desc(num_q_heads=320, num_kv_heads=64, obs_window=32), sg.GROUP_IPT_MEAN, [0.1] * 320, -1,
         sg.ERR_UNSUPPORTED, "num_q_heads"),                                   # too many query heads
        (_desc(), 0, None, -2, sg.ERR_INVALID_ARG, "window_pos"),
        (_desc(), 0, None, 2049, sg.ERR_INVALID_ARG, "window position"),      # past C
        (_desc(), 0, None, 1900, sg.ERR_INVALID_ARG, "b_window"),             # W = 32 < C - P0
    ]
    for desc, agg, qs, wp, want, word in cases:
        budgets = (512,) * desc.num_kv_heads
        assert _compress_ex(desc, agg, qs, budgets, window_pos=wp) == want, (agg, qs, wp)
        msg = sg.load_library().sgdkv_last_error().decode()
        assert word in msg, msg
    assert _compress_ex(_desc(), 0, None, reserved=1) == sg.ERR_INVALID_ARG
    # with a gather stream too, arguments are checked before any stream is touched (a bogus
    # handle here would fail if it were used)
    bogus = 0x7F0000001000
    assert _compress_ex(_desc(), 4, None, gather_stream=bogus) == sg.ERR_INVALID_ARG
    assert _compress_ex(_desc(), 0, None, budgets=(512, 9999), gather_stream=bogus) == sg.ERR_INVALID_ARG
    assert "layer_budgets" in sg.load_library().sgdkv_last_error().decode()
    # a window after the prompt needs no recent rows at all: validation passes, then no device
    if not _gpu():
        assert _compress_ex(_desc(b_window=0, b_sink=4), 0, None, budgets=(4, 4), window_pos=2048) == sg.ERR_HIP


def test_workspace_size_independent_of_budgets():
    n = sg.compress_workspace_size(_desc())
    assert n > 0 and n % 256 == 0
    assert sg.compress_workspace_size(_desc(batch=2)) > n


def test_window_rows_beyond_one_workgroup():
    """G*w up to 4096 window rows per KV head: the rows are split over several score workgroups,
    each leaving its own column-sum partial, so the workspace grows with the number of splits."""
    one = sg.compress_workspace_size(_desc(num_q_heads=16, num_kv_heads=2, obs_window=64, b_window=64))  # 512 rows
    two = sg.compress_workspace_size(_desc(num_q_heads=16, num_kv_heads=2, obs_window=128, b_window=128))
    assert two - one >= 2 * 2048 * 4  # a second [B*Hkv][C] fp32 partial, and a larger LSE region
    big = _desc(num_q_heads=64, num_kv_heads=2, obs_window=128, b_window=128)  # 4096 rows: 8 splits
    assert sg.compress_workspace_size(big) > two
    if not _gpu():  # validation passes, then no device
        assert _compress(big, [512, 512]) == sg.ERR_HIP
        assert _compress_ex(big, sg.GROUP_IPT_MAX, [0.5] * 64) == sg.ERR_HIP


def _decode(desc, offsets_host, ptrs=None, ws_bytes=None, ws=FAKE):
    lib = sg.load_library()
    ptrs = {**dict(q=FAKE, k=FAKE, v=FAKE, off=FAKE, out=FAKE, lse=FAKE), **(ptrs or {})}
    oh = np.ascontiguousarray(np.asarray(offsets_host, dtype=np.int64))
    need = ctypes.c_size_t(0)
    lib.sgdkv_decode_workspace_size(ctypes.byref(desc), sg._np_ptr(oh), ctypes.byref(need))
    return lib.sgdkv_decode_attention(ctypes.byref(desc), ptrs["q"], ptrs["k"], ptrs["v"], ptrs["off"],
                                      sg._np_ptr(oh), ptrs["out"], ptrs["lse"], ws,
                                      need.value if ws_bytes is None else ws_bytes, None)


def test_decode_validation():
    d = sg.DecodeDesc(2, 4, 2, 64, 1, 0, 0.0)
    oh = [0, 10, 10, 30, 31]
    assert _decode(sg.DecodeDesc(2, 4, 3, 64, 1, 0, 0.0), oh) == sg.ERR_INVALID_ARG
    assert _decode(sg.DecodeDesc(2, 4, 2, 80, 1, 0, 0.0), oh) == sg.ERR_UNSUPPORTED
    assert _decode(sg.DecodeDesc(1, 34, 2, 64, 1, 0, 0.0), [0, 1, 2]) == sg.ERR_UNSUPPORTED  # G = 17
    assert _decode(d, [0, 10, 9, 30, 31]) == sg.ERR_INVALID_ARG  # decreasing
    assert _decode(d, [-1, 10, 10, 30, 31]) == sg.ERR_INVALID_ARG
    assert _decode(d, oh, dict(out=None)) == sg.ERR_INVALID_ARG
    assert _decode(d, oh, dict(k=FAKE + 8)) == sg.ERR_INVALID_ARG
    assert _decode(d, oh, ws_bytes=8) == sg.ERR_WORKSPACE


def test_append_and_tail_validation():
    lib = sg.load_library()
    desc = sg.DecodeDesc(2, 8, 4, 128, sg.DTYPE_BF16, sg.DTYPE_F32, 0.0)
    oh = np.array([0, 10, 20, 30, 40, 50, 60, 70, 80], dtype=np.int64)
    P = sg._np_ptr
    need = ctypes.c_size_t(0)
    assert lib.sgdkv_decode_workspace_size_ex(ctypes.byref(desc), P(oh), -1, ctypes.byref(need)) == sg.ERR_INVALID_ARG
    assert lib.sgdkv_decode_workspace_size_ex(ctypes.byref(desc), P(oh), 0, ctypes.byref(need)) == sg.OK
    n0 = need.value
    assert lib.sgdkv_decode_workspace_size_ex(ctypes.byref(desc), P(oh), 1000, ctypes.byref(need)) == sg.OK
    assert need.value > n0
    ws = need.value

    def dec(tail, ws_bytes=ws):
        return lib.sgdkv_decode_attention_ex(ctypes.byref(desc), FAKE, FAKE, FAKE, FAKE, P(oh), ctypes.byref(tail),
                                             FAKE, None, FAKE, ws_bytes, None)
    assert dec(sg.DecodeTail(FAKE, FAKE, 100, 101)) == sg.ERR_INVALID_ARG      # n_new > capacity
    assert dec(sg.DecodeTail(FAKE, FAKE, 100, -1)) == sg.ERR_INVALID_ARG
    assert dec(sg.DecodeTail(None, FAKE, 100, 5)) == sg.ERR_INVALID_ARG        # k_new missing
    assert dec(sg.DecodeTail(FAKE + 8, FAKE, 100, 5)) == sg.ERR_INVALID_ARG    # misaligned
    assert dec(sg.DecodeTail(FAKE, FAKE, 1000, 5), ws_bytes=n0) == sg.ERR_WORKSPACE  # planned for no tail
    assert dec(sg.DecodeTail(FAKE, FAKE, 1 << 40, 5)) == sg.ERR_UNSUPPORTED    # region over 4 GiB

    def app(cap, slot, ptrs=(FAKE, FAKE, FAKE, FAKE)):
        return lib.sgdkv_append_kv(ctypes.byref(desc), *ptrs, cap, slot, None)
    assert app(10, 10) == sg.ERR_INVALID_ARG
    assert app(10, -1) == sg.ERR_INVALID_ARG
    assert app(10, 3, (FAKE, None, FAKE, FAKE)) == sg.ERR_INVALID_ARG
    assert app(10, 3, (FAKE, FAKE, FAKE + 4, FAKE)) == sg.ERR_INVALID_ARG
    assert app(1 << 40, 3) == sg.ERR_UNSUPPORTED
    bad = sg.DecodeDesc(0, 8, 4, 128, sg.DTYPE_BF16, sg.DTYPE_F32, 0.0)
    assert lib.sgdkv_append_kv(ctypes.byref(bad), FAKE, FAKE, FAKE, FAKE, 10, 3, None) == sg.ERR_INVALID_ARG
    if not _gpu():
        assert app(10, 3) == sg.ERR_HIP  # validation passed; no device here


@settings(max_examples=200, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(st.lists(st.integers(0, 1 << 20), min_size=1, max_size=64), st.integers(1, 40))
def test_segment_offsets_lay_out_segments_in_order(budgets, B):
    """The ragged cache holds segment (b, h) after every segment before it in (b, h) order."""
    got = sg.segment_offsets(budgets, B)
    row, want = 0, []
    for b in range(B):
        for n in budgets:
            want.append(row)
            row += n
    want.append(row)
    assert got.tolist() == want


def test_segment_offsets_match_the_oracle_cache():
    rng = np.random.Generator(np.random.PCG64(5))
    B, Hq, Hkv, d, C, w, s, W = 3, 6, 3, 64, 300, 8, 2, 16
    q_win = rng.standard_normal((B, Hq, w, d))
    k, v = rng.standard_normal((B, Hkv, C, d)), rng.standard_normal((B, Hkv, C, d))
    budgets = np.array([s + W, C, s + W + 77])
    orc = oracle.compress(q_win, k, v, budgets, w=w, kp=3, s=s, W=W)
    assert np.array_equal(sg.segment_offsets(budgets, B), orc["offsets"])


def test_segment_offsets_errors():
    lib = sg.load_library()
    out = np.full(5, -7, dtype=np.int64)
    P = sg._np_ptr
    assert lib.sgdkv_segment_offsets(P(np.array([1, -1], dtype=np.int64)), 2, 2, P(out)) == sg.ERR_INVALID_ARG
    assert lib.sgdkv_segment_offsets(P(np.array([1, 1], dtype=np.int64)), 0, 2, P(out)) == sg.ERR_INVALID_ARG
    assert lib.sgdkv_segment_offsets(P(np.array([1, 1], dtype=np.int64)), 2, 0, P(out)) == sg.ERR_INVALID_ARG
    assert lib.sgdkv_segment_offsets(None, 2, 2, P(out)) == sg.ERR_INVALID_ARG
    assert lib.sgdkv_segment_offsets(P(np.array([1 << 61, 1 << 61], dtype=np.int64)), 2, 2, P(out)) \
        == sg.ERR_INVALID_ARG
    assert np.all(out == -7)


def test_noalloc_decode_rejects_partials_beyond_the_static_scratch():
    """The static scratch holds 64 MiB of split partials; a decode that needs more is refused
    before anything is enqueued (validation precedes the device check, so no GPU is needed).
    Beyond 512 segments every segment holds the slots of the longest one: 1024 segments with one
    of 2^23 rows need gigabytes."""
    lib = sg.load_library()
    desc = sg.DecodeDesc(128, 64, 8, 128, sg.DTYPE_BF16, sg.DTYPE_F32, 0.0)
    oh = np.full(128 * 8 + 1, 1 << 23, dtype=np.int64)
    oh[0] = 0  # one segment of 2^23 rows, the others empty
    assert sg.decode_workspace_size(desc, oh) > 64 << 20
    P = sg._np_ptr
    st = lib.sgdkv_decode_attention_noalloc(ctypes.byref(desc), FAKE, FAKE, FAKE, FAKE, P(oh), None, FAKE, None,
                                            None)
    assert st == sg.ERR_UNSUPPORTED
    assert b"static scratch" in lib.sgdkv_last_error()
    small = np.array([0, 10, 10, 30, 31], dtype=np.int64)
    d2 = sg.DecodeDesc(2, 4, 2, 64, 1, 0, 0.0)
    assert lib.sgdkv_decode_attention_noalloc(ctypes.byref(d2), FAKE, FAKE, FAKE, FAKE, P(np.array([0, 10, 9, 30, 31])),
                                              None, FAKE, None, None) == sg.ERR_INVALID_ARG
    if not _gpu():
        assert lib.sgdkv_decode_attention_noalloc(ctypes.byref(d2), FAKE, FAKE, FAKE, FAKE, P(small), None, FAKE,
                                                  None, None) == sg.ERR_HIP


def test_decode_workspace_follows_the_splits_not_the_longest_segment():
    """With up to 512 segments the split partials are one slot per launched decode workgroup
    (G*(d+2) floats): about 12288 splits over the batch, four per workgroup, plus at most one
    part-filled workgroup per segment and half a round (256) of rounding to whole rounds of the
    device, however unequal the segments. One segment of 2^23 rows
    among 511 empty ones needs the same few megabytes as equal segments of the same total, and
    both fit the 64 MiB static scratch."""
    G, d = 8, 128
    per_wg = G * (d + 2) * 4
    for lens in ([1 << 23] + [0] * 511, [(1 << 23) // 512] * 512, [1 << 14] * 7 + [1 << 22]):
        n = len(lens)
        desc = sg.DecodeDesc(n // 8, 8 * G, 8, d, sg.DTYPE_BF16, sg.DTYPE_F32, 0.0)
        oh = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        need = sg.decode_workspace_size(desc, oh)
        wgs = need // per_wg
        assert need <= 64 << 20 and wgs <= 12288 // 4 + n + 256 + 1, (lens[:3], need)
        assert wgs >= sum(lens) // (1 << 16)  # at least one workgroup per 4 splits of at most 16384 rows
    # appended regions add their workgroups per segment
    desc = sg.DecodeDesc(2, 16, 2, d, sg.DTYPE_BF16, sg.DTYPE_F32, 0.0)
    oh = np.array([0, 1000, 1000, 5000, 5000], dtype=np.int64)
    assert sg.decode_workspace_size(desc, oh, 4096) > sg.decode_workspace_size(desc, oh)


def test_decode_workgroups_fill_whole_rounds():
    """Beyond one round of decode workgroups (the 512 an MI355X runs at once), the compact grid's
    workgroups are shared out over the segments so that they fill a whole number of rounds:
    one workgroup slot each, so the workspace holds a multiple of 512 slots. One round or less
    keeps a workgroup per four splits of the planned length."""
    G, d = 7, 128
    per_wg = G * (d + 2) * 4
    rng = np.random.Generator(np.random.PCG64(5))
    for n, hi in [(32, 70000), (128, 140000), (512, 3000), (37, 50000)]:
        lens = rng.integers(0, hi, size=n)
        lens[::9] = 0
        lens[1::13] = 1
        desc = sg.DecodeDesc(1, n * G, n, d, sg.DTYPE_BF16, sg.DTYPE_F32, 0.0)
        oh = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
        wgs = sg.decode_workspace_size(desc, oh) // per_wg
        assert wgs % 512 == 0 and wgs >= int(np.count_nonzero(lens)), (n, hi, wgs)
    lens = [300, 0, 1000, 5]  # under one round: four splits per workgroup (64 rows each, a batch this small)
    desc = sg.DecodeDesc(1, 4 * G, 4, d, sg.DTYPE_BF16, sg.DTYPE_F32, 0.0)
    oh = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    assert sg.decode_workspace_size(desc, oh) // per_wg == 2 + 0 + 4 + 1


def test_decode_workspace_with_appended_rows():
    """Appended-row workgroups (one per segment for up to 4 x 256 rows at this size) count toward the
    whole rounds while they come to at most half a round, so a capacity of 64 rows needs no more
    slots than none: 32 segments of 32768 rows plan 1024 workgroups, and with one appended each 992
    + 32. Past half a round the plan is the one without them, plus every appended slot."""
    G, d = 7, 128
    per_wg = G * (d + 2) * 4
    desc = sg.DecodeDesc(8, 4 * G, 4, d, sg.DTYPE_BF16, sg.DTYPE_F32, 0.0)
    oh = np.arange(33, dtype=np.int64) * 32768
    assert sg.decode_workspace_size(desc, oh) // per_wg == 1024
    assert sg.decode_workspace_size(desc, oh, 64) // per_wg == 1024
    assert sg.decode_workspace_size(desc, oh, 1024) // per_wg == 1024
    cap = 300000  # ceil(ceil(300000 / 256) / 4) = 293 appended workgroups per segment
    assert sg.decode_workspace_size(desc, oh, cap) // per_wg == 1024 + 32 * 293


@pytest.mark.skipif(_gpu(), reason="checks the no-device path")
def test_no_device_fails_after_validation():
    assert _compress(_desc(), [512, 512]) == sg.ERR_HIP
    assert _decode(sg.DecodeDesc(2, 4, 2, 64, 1, 0, 0.0), [0, 10, 10, 30, 31]) == sg.ERR_HIP


def test_allocation_extreme_scales_bit_exact():
    for sc, L, H, C, total in [([0.0, 0.0, 0.0, 1.0, 1.0, 2.225073858507203e-309], 2, 3, 8, 18),
                               ([1e300, 1e299, 3e298, 0.0], 1, 4, 1000, 1500),
                               ([5e-324, 5e-324, 0.0], 1, 3, 10, 17)]:
        for mode in (0, 1):
            got = sg.allocate_budgets(sc, L, H, C, 0, 0, total, mode)
            ref = oracle.allocate_budgets(np.array(sc), L, H, C, 0, 0, total, mode)
            assert np.array_equal(got, ref), (sc, mode, got, ref)
            assert np.all(got >= 0) and int(got.sum()) == total
