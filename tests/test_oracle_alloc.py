"""Pins for the oracle's head-budget allocation (Sec. 3.3 Eq. 2, Appendix A.1 Algorithm 1).

The paper prints no allocation example, so these pin the oracle against
hand-derived cases (tests/golden), exact rational shares, and the properties
that Eq. 2 and Algorithm 1 fix: integer budgets summing to the total, bounds,
monotonicity in the score, scale invariance of the normalisation, the cap
condition stated with Algorithm 1, and the greedy order of redistribution.
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_examples():
    with open(os.path.join(GOLDEN, "alloc_hand_example.json")) as f:
        fx = json.load(f)
    for case in fx["cases"]:
        b = oracle.allocate_budgets(case["scores"], case["L"], case["H"], case["C"], case["s"],
                                    case["W"], case["total"], case["mode"])
        assert b.tolist() == case["budgets"], case["note"]


def test_reduce_group_max():
    # Appendix A.7: per-attention-head scores reduce to one per KV head by max over the group
    per_q = np.array([[0.1, 0.7, 0.3, 0.2, 0.9, 0.0], [5.0, 4.0, 3.0, 2.0, 1.0, 0.5]])
    out = oracle.reduce_group_max(per_q, 2)  # G = 3
    assert out.tolist() == [[0.7, 0.9], [5.0, 2.0]]
    out3 = oracle.reduce_group_max(per_q, 3)  # G = 2
    assert out3.tolist() == [[0.7, 0.3, 0.9], [5.0, 3.0, 1.0]]


def test_total_from_ratio():
    # R of all rows: the tiny workload's "25 % of 2 x 2048 rows"
    assert oracle.total_from_ratio(0.25, 1, 2, 2048, 4, 32, of_middle=0) == 1024
    # 112 heads at 128K, 10/25/50 %
    assert oracle.total_from_ratio(0.10, 28, 4, 131072, 1024, 1024) == 1468006
    assert oracle.total_from_ratio(0.25, 28, 4, 131072, 1024, 1024) == 3670016
    assert oracle.total_from_ratio(0.50, 28, 4, 131072, 1024, 1024) == 7340032
    # Eq. 2 summed: L*H*(s+W) + floor(R*L*H*M)
    assert oracle.total_from_ratio(0.25, 1, 2, 2048, 4, 32, of_middle=1) == 2 * 36 + 1006
    with pytest.raises(oracle.OracleError):
        oracle.total_from_ratio(0.001, 1, 2, 2048, 4, 32, of_middle=0)  # below sink + window


def _exact_shares(scores, T):
    fs = [Fraction(float(x)) for x in scores]
    tot = sum(fs)
    if tot == 0:
        return [Fraction(T, len(fs))] * len(fs)
    return [x * T / tot for x in fs]


def _rank_key(scores, h):
    return (-float(scores[h]), h)


problem = st.integers(min_value=1, max_value=3).flatmap(
    lambda L: st.integers(min_value=1, max_value=6).flatmap(
        lambda H: st.tuples(
            st.just(L), st.just(H),
            st.lists(st.one_of(st.floats(0.0, 1.0), st.sampled_from([0.0, 0.25, 0.5, 1.0])),
                     min_size=L * H, max_size=L * H),
            st.integers(8, 400), st.integers(0, 4), st.integers(0, 4), st.floats(0.0, 1.0))))


def _instance(p):
    L, H, scores, C, s, W, frac = p
    n = L * H
    lo, hi = n * (s + W), n * C
    total = lo + int(round(frac * (hi - lo)))
    return L, H, np.array(scores, dtype=np.float64), C, s, W, total


@settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(problem, st.sampled_from([0, 1]))
def test_invariants(p, mode):
    L, H, scores, C, s, W, total = _instance(p)
    n = L * H
    M = C - s - W
    b = oracle.allocate_budgets(scores, L, H, C, s, W, total, mode)
    assert b.dtype == np.int64
    assert int(b.sum()) == total
    assert np.all(b >= s + W) and np.all(b <= C)
    # monotone in the score
    for a in range(n):
        for c in range(n):
            if scores[a] > scores[c]:
                assert b[a] >= b[c], (scores, b)
    # normalisation makes the allocation invariant under scaling by a power of two, wherever
    # that scaling is exact (a denormal score scaled down can round or flush to zero)
    for k in (-7, 3):
        scaled = scores * (2.0 ** k)
        if np.array_equal(scaled * (2.0 ** -k), scores):
            b2 = oracle.allocate_budgets(scaled, L, H, C, s, W, total, mode)
            assert np.array_equal(b, b2)
    # without any capping the budgets are the exact shares rounded by largest remainder
    T = total - n * (s + W)
    x = _exact_shares(scores, T)
    m = b - (s + W)
    if all(v <= M - 1 for v in x):
        for h in range(n):
            assert abs(Fraction(int(m[h])) - x[h]) < 1
        up = [h for h in range(n) if Fraction(int(m[h])) > x[h]]
        down = [h for h in range(n) if Fraction(int(m[h])) < x[h]]
        if up and down:
            # every rounded-up head has a fractional part at least that of every rounded-down one
            fu = min(x[h] - (int(m[h]) - 1) for h in up)
            fd = max(x[h] - int(m[h]) for h in down)
            assert float(fu) >= float(fd) - 1e-9


@settings(max_examples=300, deadline=None, suppress_health_check=[HealthCheck.too_slow])
@given(problem)
def test_greedy_redistribution_order(p):
    """Algorithm 1 (mode 0): capped heads sit at M and excess goes to the top-scoring heads first."""
    L, H, scores, C, s, W, total = _instance(p)
    n = L * H
    M = C - s - W
    b = oracle.allocate_budgets(scores, L, H, C, s, W, total, 0)
    m = b - (s + W)
    T = total - n * (s + W)
    x = _exact_shares(scores, T)
    order = sorted(range(n), key=lambda h: _rank_key(scores if scores.sum() > 0 else np.ones(n), h))
    # a head whose exact share reaches M is full
    for h in range(n):
        if x[h] >= M:
            assert m[h] == M
    # heads that received redistributed rows (more than their rounded-up share) come in score
    # order: every head ranked before such a head is full, and at most one of them is partial
    received = [h for h in range(n) if m[h] > max(0, -(-x[h].numerator // x[h].denominator))]
    for h in received:
        for g in order[: order.index(h)]:
            assert m[g] == M, (scores, m, h, g)
    assert sum(1 for h in received if m[h] < M) <= 1


@settings(max_examples=200, deadline=None)
@given(problem)
def test_water_level_mode(p):
    """Mode 1: x_h = min(lambda*sigma_h, M) summing to T; lambda found by bisection here."""
    L, H, scores, C, s, W, total = _instance(p)
    n = L * H
    M = C - s - W
    T = total - n * (s + W)
    sg = [Fraction(float(v)) for v in scores]
    if sum(sg) == 0:
        sg = [Fraction(1)] * n
    pos = [v for v in sg if v > 0]
    target = min(T, M * len(pos))

    def level(lam):
        return sum(min(lam * v, M) for v in sg)

    lo, hi = Fraction(0), Fraction(0)
    if target > 0:
        hi = Fraction(1)
        while level(hi) < target:
            hi *= 2
        for _ in range(100):
            mid = (lo + hi) / 2
            if level(mid) < target:
                lo = mid
            else:
                hi = mid
    x = [min(hi * v, Fraction(M)) for v in sg]
    rest = T - target  # rows that only zero-score heads can take: a flat level over them
    zeros = [h for h in range(n) if sg[h] == 0]
    if rest > 0:
        for h in zeros:
            x[h] = Fraction(rest, len(zeros))
    b = oracle.allocate_budgets(scores, L, H, C, s, W, total, 1)
    m = b - (s + W)
    assert int(m.sum()) == T
    for h in range(n):
        assert abs(Fraction(int(m[h])) - x[h]) < 1 + Fraction(1, 10**6), (scores, m, [float(v) for v in x])


def test_extremes_and_uniform():
    sc = np.array([0.3, 0.1, 0.9, 0.4, 0.0, 0.2])
    L, H, C, s, W = 2, 3, 50, 3, 5
    for mode in (0, 1):
        assert oracle.allocate_budgets(sc, L, H, C, s, W, 6 * C, mode).tolist() == [C] * 6
        assert oracle.allocate_budgets(sc, L, H, C, s, W, 6 * (s + W), mode).tolist() == [s + W] * 6
    # uniform scores: floor/ceil of T/n with the extra rows on the lowest indices
    T = 6 * 7 + 4
    b = oracle.allocate_budgets(np.full(6, 0.37), L, H, C, s, W, 6 * (s + W) + T, 0)
    assert (b - s - W).tolist() == [8, 8, 8, 8, 7, 7]


def test_cap_condition():
    """Appendix A.1: heads with S_h*L*H*R > 1 exceed the middle length and end capped at M."""
    L, H, C, s, W = 1, 8, 1000, 10, 10
    M = C - s - W
    R = 0.25
    total = oracle.total_from_ratio(R, L, H, C, s, W, of_middle=1)  # Eq. 2 summed over heads
    sc = np.array([0.7, 0.1, 0.05, 0.05, 0.04, 0.03, 0.02, 0.01])
    S = sc / sc.sum()
    b = oracle.allocate_budgets(sc, L, H, C, s, W, total, 0)
    for h in range(L * H):
        if S[h] * L * H * R > 1:
            assert b[h] - s - W == M
    # the one capped head's excess lands on the next head in score order
    assert S[0] * L * H * R > 1 and S[1] * L * H * R < 1
    x1 = S[1] * L * H * R * M
    excess = S[0] * L * H * R * M - M
    assert abs((b[1] - s - W) - (x1 + excess)) <= 1


def test_invalid_inputs():
    sc = np.array([0.5, 0.5])
    with pytest.raises(oracle.OracleError):
        oracle.allocate_budgets(np.array([0.5, -1.0]), 1, 2, 100, 1, 1, 50)
    with pytest.raises(oracle.OracleError):
        oracle.allocate_budgets(np.array([0.5, np.nan]), 1, 2, 100, 1, 1, 50)
    with pytest.raises(oracle.OracleError):
        oracle.allocate_budgets(sc, 1, 2, 100, 1, 1, 3)  # below 2*(1+1)
    with pytest.raises(oracle.OracleError):
        oracle.allocate_budgets(sc, 1, 2, 100, 1, 1, 201)  # above 2*100
    with pytest.raises(oracle.OracleError):
        oracle.allocate_budgets(sc, 1, 2, 100, 60, 60, 150)  # s + W > C


def test_extreme_score_scales():
    """Denormal and huge scores: shares are formed from normalised scores, so nothing overflows.
    Heads 3 and 4 exceed M = 8 and are capped; the 2 rows left go to the denormal head."""
    sc = np.array([0.0, 0.0, 0.0, 1.0, 1.0, 2.225073858507203e-309])
    for mode in (0, 1):
        b = oracle.allocate_budgets(sc, 2, 3, 8, 0, 0, 18, mode)
        assert b.tolist() == [0, 0, 0, 8, 8, 2], (mode, b)
    big = np.array([1e300, 1e299, 3e298, 0.0])
    for mode in (0, 1):
        b = oracle.allocate_budgets(big, 1, 4, 1000, 0, 0, 1500, mode)
        assert int(b.sum()) == 1500 and np.all(b >= 0) and np.all(b <= 1000)
        assert b[0] == 1000 and b[1] >= b[2] >= b[3]
