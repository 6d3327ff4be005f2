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
