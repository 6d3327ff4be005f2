"""The parity harness's rounding-flip diagnostics (host only)."""
import numpy as np

from gpu_harness import boundary_distance, compare_outputs
from oracle import formats


def test_boundary_distance_on_e2m1_midpoints_and_values():
    mids = np.array([0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0])
    assert np.all(boundary_distance(mids, formats.E2M1_VALUES) == 0)
    assert np.all(boundary_distance(-mids, formats.E2M1_VALUES) == 0)
    # a representable value sits half a step from its nearest boundary
    np.testing.assert_allclose(boundary_distance(np.array([1.0, 3.0, 6.0]), formats.E2M1_VALUES),
                               [0.25, 0.5 / 3, 1.0 / 6])


def test_boundary_distance_on_e4m3_table():
    table = formats.e4m3_decode(np.arange(256))
    x = np.array([1.0625, 448.0, 400.0])   # midpoint of 1 and 1.125; the top finite value; midpoint of 384 and 416
    d = boundary_distance(x, table)
    assert d[0] == 0 and d[2] == 0
    np.testing.assert_allclose(d[1], 16.0 / 448.0)   # 448 lies 16 above the 416/448 midpoint


def test_failed_comparison_reports_worst_rows_first():
    got = np.zeros((2, 3, 4))
    ref = np.zeros((2, 3, 4))
    got[1, 2] = 1.0
    got[0, 1] = 0.5
    seen = []
    try:
        compare_outputs(got, ref, "planted", lambda rows: seen.extend(rows))
    except AssertionError:
        pass
    assert [tuple(int(i) for i in r) for r in seen[:2]] == [(1, 2), (0, 1)]
