"""Pins for quotas and the shared ranking (Algorithm 1, Theorem 3.4 ordering)."""
import numpy as np
import pytest

from oracle import rank


def test_quotas_round_half_up():
    assert rank.quotas(10, 30, 100, 588 * 588) == (34574, 103724)
    assert rank.quotas(25, 25, 100, 8) == (2, 2)
    assert rank.quotas(25, 25, 100, 10) == (3, 2)          # 2.5 -> 3, 5.0 -> 5
    assert rank.quotas(100, 0, 100, 77) == (77, 0)
    assert rank.quotas(0, 40, 100, 345744) == (0, 138298)
    assert rank.quotas(5, 25, 100, 1980 ** 2) == (196020, 980100)


def _brute(scores, T8, T4):
    order = sorted(range(len(scores)), key=lambda i: (-float(scores[i]), i))
    cls = [0] * len(scores)
    for r, i in enumerate(order):
        cls[i] = 8 if r < T8 else (4 if r < T8 + T4 else 0)
    return np.array(cls, np.uint8)


@pytest.mark.parametrize("seed", range(5))
def test_head_scope_brute_force(seed):
    rng = np.random.default_rng(seed)
    R = 9
    A = rng.random((R, R)).astype(np.float32)
    A[rng.random((R, R)) < 0.3] = np.float32(0.25)          # many exact ties
    cls = rank.rank_head(A, 20, 30, 100, "head")
    T8, T4 = rank.quotas(20, 30, 100, R * R)
    np.testing.assert_array_equal(cls.reshape(-1), _brute(A.reshape(-1), T8, T4))
    assert (cls == 8).sum() == T8 and (cls == 4).sum() == T4


def test_row_scope_brute_force():
    rng = np.random.default_rng(7)
    R = 12
    A = rng.integers(0, 4, (R, R)).astype(np.float32)       # heavy ties
    cls = rank.rank_head(A, 25, 25, 100, "row")
    T8, T4 = rank.quotas(25, 25, 100, R)
    for a in range(R):
        np.testing.assert_array_equal(cls[a], _brute(A[a], T8, T4))


def test_monotone_classes_and_tie_break():
    """Theorem 3.4 ordering: every 8-bit pair scores >= every 4-bit pair >= every
    skipped pair; among equal scores the lower pair index is ranked first."""
    rng = np.random.default_rng(3)
    R = 16
    A = np.round(rng.random((R, R)) * 8).astype(np.float32) / 8
    cls = rank.rank_head(A, 10, 30, 100, "head").reshape(-1)
    a = A.reshape(-1)
    idx = np.arange(a.size)
    for hi, lo in ((8, 4), (4, 0)):
        s_hi, s_lo = a[cls == hi], a[cls == lo]
        assert s_hi.min() >= s_lo.max()
        tie = s_hi.min()
        if tie == s_lo.max():
            assert idx[(cls == hi) & (a == tie)].max() < idx[(cls == lo) & (a == tie)].min()


def test_key_lists_ascending():
    cls = np.array([0, 4, 8, 4, 0, 8, 8], np.uint8)
    l4, l8 = rank.key_lists(cls)
    assert list(l4) == [1, 3] and list(l8) == [2, 5, 6]


def test_quotas3_cumulative_against_exact_rationals():
    """T16, T8, T4 from cumulative counts rounded half up, checked with exact
    fractions; num16 = 0 reproduces the two-path quotas."""
    from fractions import Fraction
    rng = np.random.default_rng(11)
    for _ in range(200):
        den = int(rng.integers(1, 200))
        n16, n8 = (int(x) for x in rng.integers(0, den + 1, 2))
        n4 = int(rng.integers(0, den + 1))
        if n16 + n8 + n4 > den:
            continue
        M = int(rng.integers(1, 5000))
        half = lambda num: int(Fraction(num * M, den) + Fraction(1, 2))   # floor(x + 1/2), x >= 0
        c16, c168, c1684 = half(n16), half(n16 + n8), half(n16 + n8 + n4)
        assert rank.quotas3(n16, n8, n4, den, M) == (c16, c168 - c16, c1684 - c168)
        assert rank.quotas3(0, n8, n4, den, M)[1:] == rank.quotas(n8, n4, den, M)
    # 0.2, 0.3, 0.6 of 345,744: 69,148.8 -> 69,149; 103,723.2 -> 103,723; 207,446.4 -> 207,446
    assert rank.quotas3(20, 10, 30, 100, 588 * 588) == (69149, 34574, 103723)


def _brute3(scores, T16, T8, T4):
    order = sorted(range(len(scores)), key=lambda i: (-float(scores[i]), i))
    cls = [0] * len(scores)
    for r, i in enumerate(order):
        cls[i] = 16 if r < T16 else 8 if r < T16 + T8 else 4 if r < T16 + T8 + T4 else 0
    return np.array(cls, np.uint8)


@pytest.mark.parametrize("scope", ["head", "row"])
def test_sixteen_bit_quota_brute_force(scope):
    """Algorithm 1 with all three quotas: first T16 -> 16, next T8 -> 8, next
    T4 -> 4, on tie-heavy scores, against a pure-Python sort."""
    rng = np.random.default_rng(5)
    R = 11
    A = (rng.integers(0, 6, (R, R)) / 6).astype(np.float32)
    cls = rank.rank_head(A, 20, 25, 100, scope, num16=15)
    if scope == "head":
        T16, T8, T4 = rank.quotas3(15, 20, 25, 100, R * R)
        np.testing.assert_array_equal(cls.reshape(-1), _brute3(A.reshape(-1), T16, T8, T4))
        assert [(cls == c).sum() for c in (16, 8, 4)] == [T16, T8, T4]
    else:
        T16, T8, T4 = rank.quotas3(15, 20, 25, 100, R)
        for a in range(R):
            np.testing.assert_array_equal(cls[a], _brute3(A[a], T16, T8, T4))
    a = A.reshape(-1) if scope == "head" else A[0]
    c = cls.reshape(-1) if scope == "head" else cls[0]
    for hi, lo in ((16, 8), (8, 4), (4, 0)):
        if (c == hi).any() and (c == lo).any():
            assert a[c == hi].min() >= a[c == lo].max()


def test_key_lists_all_segments():
    cls = np.array([16, 4, 8, 4, 0, 16, 8], np.uint8)
    l4, l8, l16 = rank.key_lists_all(cls)
    assert list(l4) == [1, 3] and list(l8) == [2, 6] and list(l16) == [0, 5]
