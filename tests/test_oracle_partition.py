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


RAGGED_FRAMES = [(30, 52), (45, 80), (16, 16), (13, 21), (2, 100), (100, 2), (7, 17), (1, 1), (1, 130), (65, 1),
                 (9, 9), (24, 40), (33, 7)]


def _components(mask):
    """Number of 4-connected components of a boolean mask (breadth-first search)."""
    seen = np.zeros_like(mask)
    n = 0
    for y0, x0 in zip(*np.nonzero(mask)):
        if seen[y0, x0]:
            continue
        n += 1
        stack = [(y0, x0)]
        seen[y0, x0] = True
        while stack:
            y, x = stack.pop()
            for yy, xx in ((y + 1, x), (y - 1, x), (y, x + 1), (y, x - 1)):
                if 0 <= yy < mask.shape[0] and 0 <= xx < mask.shape[1] and mask[yy, xx] and not seen[yy, xx]:
                    seen[yy, xx] = True
                    stack.append((yy, xx))
    return n


@pytest.mark.parametrize("H,W", RAGGED_FRAMES)
def test_ragged_counts_padding_connectivity(H, W):
    """Ragged-padding equation: R_f = ceil(HW/C) regions, 0 <= R_f C - HW < C;
    every region holds at most C tokens and is connected."""
    lab = P.ragged_frame_labels(H, W)
    Rf = int(lab.max()) + 1
    assert Rf == -(-H * W // 64)
    assert 0 <= Rf * 64 - H * W < 64
    counts = np.bincount(lab.reshape(-1), minlength=Rf)
    assert counts.min() > 0 and counts.max() <= 64
    for r in range(Rf):
        assert _components(lab == r) == 1, (H, W, r)


@pytest.mark.parametrize("H,W", RAGGED_FRAMES)
def test_ragged_perimeter_identity(H, W):
    """Region-perimeter equation: the unit boundary edges of all regions sum to
    2(H+W) + 2 E_cut, counted here region by region."""
    lab = P.ragged_frame_labels(H, W)
    pad = np.pad(lab, 1, constant_values=-1)
    total = 0
    for r in range(int(lab.max()) + 1):
        m = pad == r
        total += int((m[1:-1, 1:-1] & (pad[:-2, 1:-1] != r)).sum() + (m[1:-1, 1:-1] & (pad[2:, 1:-1] != r)).sum()
                     + (m[1:-1, 1:-1] & (pad[1:-1, :-2] != r)).sum() + (m[1:-1, 1:-1] & (pad[1:-1, 2:] != r)).sum())
    assert total == 2 * (H + W) + 2 * P.cut_edges(lab)


@pytest.mark.parametrize("T,H,W", [(2, 16, 16), (1, 24, 40), (3, 8, 8)])
def test_ragged_is_the_tiling_when_8_divides_the_frame(T, H, W):
    """With 8 | H and 8 | W the smallest perimeter among the candidates is the
    8x8 tiling (a square has the least perimeter for its area), so both
    partitions coincide, block numbering and slot order included."""
    r = P.ragged_partition(T, H, W)
    t = P.tile_partition(T, H, W)
    for x, y in zip(r, t):
        np.testing.assert_array_equal(x, y)


def test_ragged_mid_layer_block_count():
    """21x30x52 latent: 25 regions per frame (ceil(1560/64)) instead of 28 tiles,
    region sizes 62 or 63, five bands of six rows."""
    slot2tok, n_a, tok2slot = P.ragged_partition(21, 30, 52)
    assert n_a.size == 21 * 25
    assert set(np.unique(n_a)) <= {62, 63}
    lab = P.ragged_frame_labels(30, 52)
    assert all(len(np.unique(lab[6 * b:6 * b + 6])) == 5 for b in range(5))
    valid = slot2tok >= 0
    assert np.array_equal(np.sort(slot2tok[valid]), np.arange(21 * 30 * 52))
    assert np.array_equal(tok2slot[slot2tok[valid]], np.nonzero(valid)[0])
