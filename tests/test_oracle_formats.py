"""Pins for the oracle's number formats (E4M3, E2M1, INT8 rounding).

Format definitions: OCP FP8 E4M3FN (bias 7, 3 mantissa bits, max 448, codes
0x7F/0xFF are NaN) and OCP FP4 E2M1 (values 0, .5, 1, 1.5, 2, 3, 4, 6), as
used by the paper's format appendix; INT8 rounds ties away from zero (INT8
paragraph of the same appendix).
"""
import decimal
import struct

import numpy as np
import pytest
import torch

from oracle import formats as F


def _e4m3_table():
    """All finite E4M3 codes and values, built from the bit-field definition."""
    codes, vals = [], []
    for c in range(256):
        if c & 0x7F == 0x7F:
            continue
        s = -1.0 if c & 0x80 else 1.0
        e, m = (c >> 3) & 15, c & 7
        v = (m / 8) * 2.0 ** -6 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7)
        codes.append(c)
        vals.append(s * v)
    return np.array(codes), np.array(vals)


def test_e4m3_exhaustive_codes():
    codes, vals = _e4m3_table()
    assert np.max(vals) == 448.0 and np.min(vals) == -448.0
    np.testing.assert_array_equal(F.e4m3(vals), vals)
    np.testing.assert_array_equal(F.e4m3_code(vals), codes)
    np.testing.assert_array_equal(F.e4m3_decode(codes), vals)


def test_e4m3_midpoints_round_to_even():
    _, vals = _e4m3_table()
    pos = np.unique(vals[vals >= 0])
    for lo, hi in zip(pos[:-1], pos[1:]):
        mid = (lo + hi) / 2
        even = lo if F.e4m3_code(lo) % 2 == 0 else hi
        assert F.e4m3(mid) == even
        assert F.e4m3(-mid) == -even
        eps = (hi - lo) * 1e-6
        assert F.e4m3(mid - eps) == lo and F.e4m3(mid + eps) == hi


def test_e4m3_saturates_never_nan():
    for x in (448.0, 449.0, 464.0, 480.0, 1e6, 3.4e38):
        assert F.e4m3(x) == 448.0 and F.e4m3(-x) == -448.0


def test_e4m3_matches_torch_float8_in_range():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(20000) * 10.0,
                        rng.uniform(-448, 448, 20000),
                        rng.uniform(-2 ** -6, 2 ** -6, 20000)]).astype(np.float32)
    t = torch.from_numpy(x).to(torch.float8_e4m3fn).to(torch.float64).numpy()
    np.testing.assert_array_equal(F.e4m3(x.astype(np.float64)), t)


def _e2m1_nearest_even(x):
    """Brute force: nearest E2M1 magnitude, ties to the even code."""
    a = abs(x)
    if a >= 6.0:
        return float(np.copysign(6.0, x))
    best = None
    for code, v in enumerate(F.E2M1_VALUES):
        dist = abs(a - v)
        if best is None or dist < best[0] or (dist == best[0] and code % 2 == 0):
            best = (dist, code, v)
    return float(np.copysign(best[2], x))


def test_e2m1_table_and_ties():
    np.testing.assert_array_equal(F.e2m1(F.E2M1_VALUES), F.E2M1_VALUES)
    np.testing.assert_array_equal(F.e2m1_code(F.E2M1_VALUES), np.arange(8))
    np.testing.assert_array_equal(F.e2m1_code(-F.E2M1_VALUES[1:]), np.arange(1, 8) | 8)
    ties = {0.25: 0.0, 0.75: 1.0, 1.25: 1.0, 1.75: 2.0, 2.5: 2.0, 3.5: 4.0, 5.0: 4.0}
    for x, want in ties.items():
        assert F.e2m1(x) == want and F.e2m1(-x) == -want
    assert F.e2m1(7.0) == 6.0 and F.e2m1(1e9) == 6.0


def test_e2m1_brute_force_random():
    rng = np.random.default_rng(1)
    x = np.concatenate([rng.uniform(-7, 7, 3000), rng.uniform(-1, 1, 1000)])
    want = np.array([_e2m1_nearest_even(v) for v in x])
    np.testing.assert_array_equal(F.e2m1(x), want)


def test_half_away_matches_decimal():
    rng = np.random.default_rng(2)
    y = np.concatenate([rng.uniform(-130, 130, 5000).astype(np.float32),
                        np.arange(-127, 128) + np.float32(0.5),
                        np.arange(-127, 128) - np.float32(0.5)]).astype(np.float64)
    want = [float(decimal.Decimal(float(v)).quantize(decimal.Decimal(1), rounding=decimal.ROUND_HALF_UP))
            for v in y]
    np.testing.assert_array_equal(F.half_away(y), np.array(want))


def test_f32_single_rounding():
    for v in (1 / 3, 0.1, 2.0 ** -140, 1e30):
        assert float(F.f32(v)) == struct.unpack("f", struct.pack("f", v))[0]
