"""The rounding identity the INT8 encoder relies on (operand preparation):
for every float32 y with |y| <= 130, truncating the float32 sum
y + copysign(0.5 - 2^-25, y) equals y rounded half away from zero. Checked
exhaustively with numpy's IEEE float32 arithmetic against the definition
computed in float64 (the device probe test runs the encoder's own function on
every tie and its neighbours)."""
import numpy as np

from oracle import formats as F


def test_round_half_away_identity_exhaustive():
    c = np.nextafter(np.float32(0.5), np.float32(0))
    assert c == np.float32(0.49999997)
    hi = int(np.float32(130.0).view(np.uint32))
    chunk = 1 << 25
    bad = 0
    for start in range(0, hi + 1, chunk):
        y = np.arange(start, min(start + chunk, hi + 1), dtype=np.uint32).view(np.float32)
        for ys in (y, -y):
            got = np.trunc(ys + np.copysign(c, ys))
            bad += int(np.count_nonzero(got != F.half_away(ys)))
    assert bad == 0
