"""Pins for pooling and the draft map (descriptor equation, Definition 3.1,
Remark on bilinearity)."""
import numpy as np
import pytest
from scipy.special import softmax

from oracle import draft, partition


def _tiny(seed=0, T=2, Hg=13, Wg=11, d=16):
    rng = np.random.default_rng(seed)
    N = T * Hg * Wg
    Q = rng.standard_normal((N, d)).astype(np.float32)
    K = (rng.standard_normal((N, d)) * 2).astype(np.float32)
    return Q, K, partition.tile_partition(T, Hg, Wg)


def test_pool_brute_force_loops():
    Q, _, (slot2tok, n_a, _) = _tiny()
    T, Hg, Wg = 2, 13, 11
    mean, mx = draft.pool(Q, slot2tok, n_a)
    a = 0
    for t in range(T):
        for i in range(0, Hg, 8):
            for j in range(0, Wg, 8):
                rows = [Q[t * Hg * Wg + y * Wg + x].astype(np.float64)
                        for y in range(i, min(i + 8, Hg)) for x in range(j, min(j + 8, Wg))]
                for c in range(Q.shape[1]):
                    s = 0.0
                    m = -np.inf
                    for r in rows:
                        s += r[c]
                        m = max(m, r[c])
                    assert mean[a, c] == pytest.approx(s / len(rows), rel=1e-15, abs=1e-15)
                    assert mx[a, c] == m
                a += 1


@pytest.mark.parametrize("lam", [0.0, 0.2, 1.0])
def test_draft_rows_sum_to_one_and_branches(lam):
    Q, K, (slot2tok, n_a, _) = _tiny(1)
    A32, p = draft.draft_head(Q, K, slot2tok, n_a, lam)
    A = p["A64"]
    np.testing.assert_allclose(A.sum(axis=1), 1.0, rtol=0, atol=1e-14)
    d = Q.shape[1]
    avg = softmax(p["Qbar"] @ p["Kbar"].T / np.sqrt(d), axis=1)
    mxb = softmax(p["Qmax"] @ p["Kmax"].T / np.sqrt(d), axis=1)
    np.testing.assert_allclose(A, (1 - lam) * avg + lam * mxb, rtol=1e-13, atol=1e-16)
    if lam == 0.0:
        np.testing.assert_allclose(A, avg, rtol=1e-13)
    assert A32.dtype == np.float32 and np.array_equal(A32, A.astype(np.float32))


def test_bilinearity_mean_token_pair_logit():
    """Qbar_a . Kbar_b / sqrt d equals the mean token-pair logit between the regions."""
    Q, K, (slot2tok, n_a, _) = _tiny(2)
    Qbar, _ = draft.pool(Q, slot2tok, n_a)
    Kbar, _ = draft.pool(K, slot2tok, n_a)
    d = Q.shape[1]
    for a, b in [(0, 0), (1, 3), (5, 2), (7, 7)]:
        qa = Q[slot2tok[a * 64:a * 64 + n_a[a]]].astype(np.float64)
        kb = K[slot2tok[b * 64:b * 64 + n_a[b]]].astype(np.float64)
        pair_mean = (qa @ kb.T / np.sqrt(d)).mean()
        assert Qbar[a] @ Kbar[b] / np.sqrt(d) == pytest.approx(pair_mean, rel=1e-12, abs=1e-12)


def test_max_branch_sees_what_mean_hides():
    """Two key regions with equal means but different channel maxima get equal
    average-branch scores and different max-branch scores."""
    d = 4
    Qbar = np.ones((1, d))
    Qmax = np.ones((1, d))
    Kbar = np.zeros((2, d))
    Kmax = np.array([[0.1] * d, [3.0] * d])
    A0 = draft.draft_map(Qbar, Kbar, Qmax, Kmax, 0.0)
    A1 = draft.draft_map(Qbar, Kbar, Qmax, Kmax, 0.5)
    assert A0[0, 0] == A0[0, 1] == 0.5
    assert A1[0, 1] > A1[0, 0]
