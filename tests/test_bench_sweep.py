"""Host-side pieces of the operator sweep in bench.py: budgets of the sweep
points and the dense reference rows of its error metric (checked against the
oracle's textbook dense attention)."""
import numpy as np

import bench
from oracle import attention


def test_sweep_budgets_follow_mix_and_retained_fraction():
    pts = bench.sweep_points()
    assert len(pts) == len(set(pts))
    for lam, mix, rho, fmt4 in pts:
        n16, n8, n4 = bench.sweep_budgets(mix, rho)
        total = n16 + n8 + n4
        assert 0 < total <= bench.SWEEP_DEN
        assert abs(total - rho * bench.SWEEP_DEN) <= 1.5      # rounding of up to three shares
        for n, pct in zip((n16, n8, n4), bench.SWEEP_MIXES[mix]):
            assert (n == 0) == (pct == 0)
        assert fmt4 == "nvfp4" or bench.SWEEP_MIXES[mix][2] > 0   # MXFP4 only where a 4-bit share exists
    assert bench.sweep_budgets("4/8/16", 1.0) == (100, 300, 600)


def test_dense_rows_equal_textbook_attention():
    rng = np.random.default_rng(3)
    Q = rng.standard_normal((50, 32)).astype(np.float32) * 3
    K = rng.standard_normal((300, 32)).astype(np.float32) * 3
    V = rng.standard_normal((300, 32)).astype(np.float32)
    rows = np.array([0, 7, 49])
    np.testing.assert_allclose(bench.dense_rows(Q[rows], K, V), attention.dense_attention(Q, K, V)[rows],
                               rtol=1e-12, atol=1e-12)
