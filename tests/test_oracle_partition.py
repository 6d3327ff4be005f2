"""Pins for the region layout: 8x8 tiles, compact valid slots, inverse map."""
import numpy as np
import pytest

from oracle import partition as P


@pytest.mark.parametrize("T,Hg,Wg", [(2, 16, 16), (2, 13, 11), (1, 8, 8), (3, 7, 17), (21, 30, 52)])
def test_tiles_brute_force(T, Hg, Wg):
    slot2tok, n_a, tok2slot = P.tile_partition(T, Hg, Wg)
    nI, nJ = -(-Hg // 8), -(-Wg // 8)
    assert n_a.size == T * nI * nJ
    # every token exactly once, and tok2slot inverts slot2tok
    valid = slot2tok[slot2tok >= 0]
    assert np.array_equal(np.sort(valid), np.arange(T * Hg * Wg))
    assert np.array_equal(slot2tok[tok2slot], np.arange(T * Hg * Wg))
    # brute force over tokens: block id, and slot = row-major rank within the tile's valid rectangle
    for n in range(0, T * Hg * Wg, max(1, T * Hg * Wg // 500)):
        t, rem = divmod(n, Hg * Wg)
        y, x = divmod(rem, Wg)
        a = (t * nI + y // 8) * nJ + x // 8
        w = min(8, Wg - (x // 8) * 8)
        assert tok2slot[n] == a * 64 + (y % 8) * w + (x % 8)
    # valid slots come first in each block
    for a in range(n_a.size):
        blk = slot2tok[a * 64:(a + 1) * 64]
        assert np.all(blk[:n_a[a]] >= 0) and np.all(blk[n_a[a]:] == -1)


def test_mid_layer_tile_sizes():
    slot2tok, n_a, _ = P.tile_partition(21, 30, 52)
    assert n_a.size == 588
    assert set(np.unique(n_a)) == {24, 32, 48, 64}
    assert abs(1 - n_a.sum() / (588 * 64) - 0.1295) < 1e-3
