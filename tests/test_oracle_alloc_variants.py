"""Pins of the oracle's allocation variants (Appendix A.7, Table 5).

Hand-worked values (tests/golden/alloc_variants_hand.json), closed forms
(Reverse mirrors each head about the middle), brute-force orderings (the
binary variants) and exact-arithmetic identities (a mix of a vector with
itself is the plain allocation of the normalised vector).
"""
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "alloc_variants_hand.json")
VARIANT = {"plain": oracle.ALLOC_PLAIN, "thr": oracle.ALLOC_THR, "reverse": oracle.ALLOC_REVERSE,
           "mix": oracle.ALLOC_MIX, "binary": oracle.ALLOC_BINARY, "binary_reverse": oracle.ALLOC_BINARY_REVERSE}


@pytest.mark.parametrize("case", json.load(open(GOLDEN))["cases"], ids=lambda c: f"{c['variant']}-{c['mode']}")
def test_hand_examples(case):
    b = oracle.allocate_variant(np.array(case["scores"]), case["L"], case["H"], case["C"], case["s"], case["W"],
                                case["total"], VARIANT[case["variant"]], mode=case["mode"],
                                scores2=np.array(case["scores2"]) if "scores2" in case else None,
                                full_fraction=case.get("full_fraction", 0.0))
    assert b.tolist() == case["budgets"], case["note"]


heads = st.integers(1, 3).flatmap(lambda L: st.integers(1, 5).flatmap(lambda H: st.tuples(
    st.just(L), st.just(H),
    st.lists(st.one_of(st.floats(0.0, 1.0), st.sampled_from([0.0, 0.5, 1.0])), min_size=L * H, max_size=L * H),
    st.lists(st.one_of(st.floats(0.0, 1.0), st.sampled_from([0.0, 0.5, 1.0])), min_size=L * H, max_size=L * H),
    st.integers(8, 300), st.integers(0, 3), st.integers(0, 3), st.floats(0.0, 1.0), st.sampled_from([0, 1]))))


def _total(n, C, s, W, frac):
    lo, hi = n * (s + W), n * C
    return lo + int(round(frac * (hi - lo)))


@settings(max_examples=200, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(heads)
def test_reverse_mirrors_each_head(p):
    L, H, sc, _, C, s, W, frac, mode = p
    n, M = L * H, C - s - W
    total = _total(n, C, s, W, frac)
    sc = np.array(sc)
    b = oracle.allocate_budgets(sc, L, H, C, s, W, total, mode)
    r = oracle.allocate_variant(sc, L, H, C, s, W, total, oracle.ALLOC_REVERSE, mode=mode)
    assert np.all(r + b == 2 * (s + W) + M)
    assert int(r.sum()) == n * (C + s + W) - total


@settings(max_examples=200, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(heads)
def test_thr_zeroes_below_mean(p):
    L, H, sc, _, C, s, W, frac, mode = p
    n, M = L * H, C - s - W
    total = _total(n, C, s, W, frac)
    sc = np.array(sc)
    b = oracle.allocate_variant(sc, L, H, C, s, W, total, oracle.ALLOC_THR, mode=mode)
    assert int(b.sum()) == total and np.all(b >= s + W) and np.all(b <= C)
    # the threshold is the mean of all L*H scores, here in exact rational arithmetic; a score
    # within an ulp of it may fall on either side of the fp64 mean, so such draws pin nothing
    mean = sum(Fraction(x) for x in sc.tolist()) / n
    ulp = Fraction(math.ulp(float(mean))) if mean > 0 else Fraction(0)
    if any(abs(Fraction(x) - mean) <= ulp for x in sc.tolist()) and len(set(sc.tolist())) > 1:
        return
    kept = [Fraction(x) >= mean for x in sc.tolist()]
    # without caps, the shares of the surviving heads are exact rationals and a zeroed head gets nothing
    T = total - n * (s + W)
    tot = sum(Fraction(x) for x, k in zip(sc.tolist(), kept) if k)
    if tot > 0:
        x = [Fraction(v) * T / tot if k else Fraction(0) for v, k in zip(sc.tolist(), kept)]
        if all(v <= M - 1 for v in x):
            m = b - (s + W)
            for h in range(n):
                assert abs(Fraction(int(m[h])) - x[h]) < 1
                if not kept[h]:
                    assert m[h] == 0
    # equal scores: nothing is below the mean, so thr is the plain allocation
    u = np.full(n, 0.375)
    assert np.array_equal(oracle.allocate_variant(u, L, H, C, s, W, total, oracle.ALLOC_THR, mode=mode),
                          oracle.allocate_budgets(u, L, H, C, s, W, total, mode))


@settings(max_examples=200, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(heads)
def test_mix_identities(p):
    L, H, sc, sc2, C, s, W, frac, mode = p
    n = L * H
    total = _total(n, C, s, W, frac)
    a, b2 = np.array(sc), np.array(sc2)
    ab = oracle.allocate_variant(a, L, H, C, s, W, total, oracle.ALLOC_MIX, mode=mode, scores2=b2)
    ba = oracle.allocate_variant(b2, L, H, C, s, W, total, oracle.ALLOC_MIX, mode=mode, scores2=a)
    assert np.array_equal(ab, ba)  # the average is symmetric
    assert int(ab.sum()) == total
    # mixing a vector with itself: (S + S) / 2 == S exactly, so it is the plain allocation of S
    tot = 0.0
    for x in sc:
        tot += x
    S = np.array([x / tot for x in sc]) if tot > 0 else np.full(n, 1.0 / n)
    aa = oracle.allocate_variant(a, L, H, C, s, W, total, oracle.ALLOC_MIX, mode=mode, scores2=a)
    assert np.array_equal(aa, oracle.allocate_budgets(S, L, H, C, s, W, total, mode))


@settings(max_examples=200, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(heads, st.floats(0.0, 1.0))
def test_binary_is_a_top_k_by_score(p, f):
    L, H, sc, _, C, s, W, frac, mode = p
    n = L * H
    total = _total(n, C, s, W, frac)
    sc = np.array(sc)
    order = sorted(range(n), key=lambda h: (-sc[h], h))  # brute force: stable sort by score
    k = int(np.floor(f * n))
    top = oracle.allocate_variant(sc, L, H, C, s, W, total, oracle.ALLOC_BINARY, full_fraction=f)
    bot = oracle.allocate_variant(sc, L, H, C, s, W, total, oracle.ALLOC_BINARY_REVERSE, full_fraction=f)
    assert sorted(np.flatnonzero(top == C).tolist()) == sorted(order[:k]) or C == s + W
    assert sorted(np.flatnonzero(bot == C).tolist()) == sorted(order[n - k:]) or C == s + W
    assert np.all((top == C) | (top == s + W)) and np.all((bot == C) | (bot == s + W))


def test_variant_errors():
    sc = np.array([1.0, 2.0])
    with pytest.raises(oracle.OracleError):
        oracle.allocate_variant(sc, 1, 2, 10, 1, 1, 10, oracle.ALLOC_MIX)  # no second vector
    with pytest.raises(oracle.OracleError):
        oracle.allocate_variant(sc, 1, 2, 10, 1, 1, 10, oracle.ALLOC_MIX, scores2=np.array([1.0, -1.0]))
    with pytest.raises(oracle.OracleError):
        oracle.allocate_variant(sc, 1, 2, 10, 1, 1, 10, oracle.ALLOC_BINARY, full_fraction=1.5)
    with pytest.raises(oracle.OracleError):
        oracle.allocate_variant(sc, 1, 2, 10, 1, 1, 10, 6)
