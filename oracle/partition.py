"""Spatial regions and slot maps (oracle; test infrastructure).

Paper: "Spatial grouping" (each frame split into connected regions whose
token count is bounded by the attention block capacity C), the fused
preparation section (each region packed into one contiguous block; the
inverse index map restores token order) and the routing appendix (valid
counts n_a exclude padding).

Two partitions (C = 64), both with the slots of a block holding its valid
tokens in row-major order, followed by padding; tokens are numbered
frame-major raster: n = t*Hg*Wg + y*Wg + x.

* 8x8 tiles (the configured hot path): block a = t*nI*nJ + i*nJ + j with
  nI = ceil(Hg/8), nJ = ceil(Wg/8).
* Ragged (fused-reordering paragraph; ragged-padding and region-perimeter
  equations): R_f = ceil(Hg*Wg/C) connected regions per frame with less
  than one block of padding, chosen for the smallest total perimeter.
  Reading (the paper names the criteria, not an algorithm): the candidates
  split the frame into nb bands of balanced height (the larger bands first),
  along rows or along columns; each band is walked in a snake order (down
  one column, up the next; for column bands, along one row and back the
  next) and cut into consecutive runs of balanced size (the larger runs
  first), ceil(band/C) runs per band. A candidate is valid when its run
  count equals R_f. Among valid candidates the smallest total perimeter
  wins, then row bands before column bands, then fewer bands. Regions are
  numbered band by band, run by run; block a = t*R_f + region.
"""
import numpy as np

TILE = 8
CAP = TILE * TILE


def tile_partition(T, Hg, Wg):
    """Return (slot2tok [R*64] int64 with -1 for padding, n_a [R], tok2slot [N])."""
    nI = -(-Hg // TILE)
    nJ = -(-Wg // TILE)
    R = T * nI * nJ
    slot2tok = np.full(R * CAP, -1, dtype=np.int64)
    n_a = np.zeros(R, dtype=np.int64)
    for t in range(T):
        for i in range(nI):
            for j in range(nJ):
                a = (t * nI + i) * nJ + j
                ys = np.arange(i * TILE, min(i * TILE + TILE, Hg))
                xs = np.arange(j * TILE, min(j * TILE + TILE, Wg))
                toks = (t * Hg * Wg + ys[:, None] * Wg + xs[None, :]).reshape(-1)
                slot2tok[a * CAP: a * CAP + toks.size] = toks
                n_a[a] = toks.size
    tok2slot = np.full(T * Hg * Wg, -1, dtype=np.int64)
    valid = slot2tok >= 0
    tok2slot[slot2tok[valid]] = np.nonzero(valid)[0]
    return slot2tok, n_a, tok2slot


def _snake_band_labels(h, w, runs, first_label):
    """Labels [h, w] of one band of h rows: snake walk down/up the columns,
    cut into ``runs`` consecutive runs of balanced size (larger first)."""
    n = h * w
    sizes = [n // runs + (1 if k < n % runs else 0) for k in range(runs)]
    walk = []
    for x in range(w):
        ys = range(h) if x % 2 == 0 else range(h - 1, -1, -1)
        walk.extend((y, x) for y in ys)
    lab = np.empty((h, w), dtype=np.int64)
    pos = 0
    for k, size in enumerate(sizes):
        for (y, x) in walk[pos:pos + size]:
            lab[y, x] = first_label + k
        pos += size
    return lab


def cut_edges(lab):
    """Number of horizontally or vertically adjacent cell pairs with different labels."""
    return int((lab[:, 1:] != lab[:, :-1]).sum() + (lab[1:, :] != lab[:-1, :]).sum())


def _band_candidate(H, W, nb, C):
    """Labels [H, W] of the row-band candidate with nb bands, or None if its
    run count differs from ceil(H*W/C)."""
    Rf = -(-H * W // C)
    heights = [H // nb + (1 if i < H % nb else 0) for i in range(nb)]
    runs = [-(-h * W // C) for h in heights]
    if sum(runs) != Rf:
        return None
    bands, label = [], 0
    for h, r in zip(heights, runs):
        bands.append(_snake_band_labels(h, W, r, label))
        label += r
    return np.concatenate(bands, axis=0)


def ragged_frame_labels(H, W, C=CAP):
    """Region label of every cell of one H x W frame (ragged partition)."""
    best = None
    for orient in (0, 1):                       # 0: row bands, 1: column bands
        h, w = (H, W) if orient == 0 else (W, H)
        for nb in range(1, h + 1):
            lab = _band_candidate(h, w, nb, C)
            if lab is None:
                continue
            lab = lab if orient == 0 else lab.T
            key = (cut_edges(lab), orient, nb)   # total perimeter = 2(H+W) + 2 E_cut
            if best is None or key < best[0]:
                best = (key, lab)
    return best[1]


def ragged_partition(T, Hg, Wg):
    """Return (slot2tok [R*64] int64 with -1 for padding, n_a [R], tok2slot [N])
    of the ragged partition (same frame labels in every frame)."""
    lab = ragged_frame_labels(Hg, Wg)
    Rf = int(lab.max()) + 1
    R = T * Rf
    slot2tok = np.full(R * CAP, -1, dtype=np.int64)
    n_a = np.zeros(R, dtype=np.int64)
    for t in range(T):
        for r in range(Rf):
            ys, xs = np.nonzero(lab == r)            # row-major order
            toks = t * Hg * Wg + ys * Wg + xs
            a = t * Rf + r
            slot2tok[a * CAP: a * CAP + toks.size] = toks
            n_a[a] = toks.size
    tok2slot = np.full(T * Hg * Wg, -1, dtype=np.int64)
    valid = slot2tok >= 0
    tok2slot[slot2tok[valid]] = np.nonzero(valid)[0]
    return slot2tok, n_a, tok2slot


def make_partition(kind, T, Hg, Wg):
    """``kind`` = "tiles8" or "ragged"."""
    if kind == "tiles8":
        return tile_partition(T, Hg, Wg)
    if kind == "ragged":
        return ragged_partition(T, Hg, Wg)
    raise ValueError(kind)


def gather_slots(X, slot2tok):
    """X [N, d] -> [R, 64, d] in slot order, padding slots set to 0."""
    R = slot2tok.size // CAP
    out = np.zeros((slot2tok.size, X.shape[1]), dtype=X.dtype)
    valid = slot2tok >= 0
    out[valid] = X[slot2tok[valid]]
    return out.reshape(R, CAP, X.shape[1])
