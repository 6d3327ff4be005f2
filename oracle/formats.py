"""Number formats used by the mixed-precision paths (oracle; test infrastructure).

Paper: appendix "Quantization Formats and Scales" and Table "Operand and
accumulator formats". E4M3 is the OCP FP8 E4M3FN format (max finite 448, no
infinities); E2M1 is the OCP FP4 format (max 6). The paper does not state a
rounding mode for its casts; the reading used here is round to nearest,
ties to even, saturating at the largest finite magnitude (never NaN).

INT8 rounds to nearest with ties away from zero, as the INT8 paragraph of
the format appendix states.

Everything here works on float64 arrays whose values are exact copies of
the float32 inputs the format definition applies to.
"""
import numpy as np

E4M3_MBITS, E4M3_EMIN, E4M3_MAX = 3, -6, 448.0
E2M1_MBITS, E2M1_EMIN, E2M1_MAX = 1, 0, 6.0

# Magnitudes of the 8 non-negative E2M1 codes, code = index.
E2M1_VALUES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def round_float_format(x, mbits, emin, maxval):
    """Round to a binary float format with ``mbits`` fraction bits and
    minimum normal exponent ``emin`` (subnormals below), ties to even,
    saturating at ``maxval``. Sign is preserved (including -0)."""
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    _, e = np.frexp(a)                 # a = f * 2**e with f in [0.5, 1)
    e = np.maximum(e - 1, emin)        # exponent of the binade (clamped to subnormal range)
    ulp = np.ldexp(1.0, e - mbits)
    q = np.rint(a / ulp) * ulp         # a/ulp is exact (power-of-two scaling); rint ties to even
    q = np.minimum(q, maxval)
    return np.copysign(q, x)


def e4m3(x):
    """Value of x after a round-to-nearest-even, saturating cast to E4M3."""
    return round_float_format(x, E4M3_MBITS, E4M3_EMIN, E4M3_MAX)


def e2m1(x):
    """Value of x after a round-to-nearest-even, saturating cast to E2M1."""
    return round_float_format(x, E2M1_MBITS, E2M1_EMIN, E2M1_MAX)


def e4m3_code(v):
    """Byte code of E4M3 values ``v`` (already representable): sign bit 7,
    exponent bits 6..3 (bias 7), mantissa bits 2..0."""
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    _, e = np.frexp(a)
    e = e - 1
    normal = a >= 2.0 ** E4M3_EMIN
    exp_field = np.where(normal, e + 7, 0)
    mant = np.where(normal, a / np.ldexp(1.0, e) - 1.0, a / 2.0 ** (E4M3_EMIN)) * 8.0
    code = (exp_field.astype(np.int64) << 3) | np.rint(mant).astype(np.int64)
    code = np.where(a == 0, 0, code)
    return (code | (np.signbit(v).astype(np.int64) << 7)).astype(np.uint8)


def e4m3_decode(code):
    """Value of each E4M3 byte code (0x7F / 0xFF, the NaN codes, map to NaN)."""
    c = np.asarray(code, dtype=np.int64)
    s = np.where(c & 0x80, -1.0, 1.0)
    ef = (c >> 3) & 0xF
    m = c & 7
    mag = np.where(ef == 0, m / 8.0 * 2.0 ** E4M3_EMIN, (1.0 + m / 8.0) * np.ldexp(1.0, ef - 7))
    mag = np.where((c & 0x7F) == 0x7F, np.nan, mag)
    return s * mag


def e2m1_code(v):
    """4-bit code of E2M1 values ``v`` (already representable): sign bit 3."""
    v = np.asarray(v, dtype=np.float64)
    a = np.abs(v)
    idx = np.searchsorted(E2M1_VALUES, a)
    return (idx | (np.signbit(v).astype(np.int64) << 3)).astype(np.uint8)


def half_away(y):
    """Round to nearest integer, ties away from zero (exact for float32 inputs)."""
    y = np.asarray(y, dtype=np.float64)
    return np.sign(y) * np.floor(np.abs(y) + 0.5)


def f32(x):
    """Round to float32 (the single rounding of one IEEE fp32 operation)."""
    return np.asarray(x, dtype=np.float64).astype(np.float32)
