"""Spatial regions and slot maps (oracle; test infrastructure).

Paper: "Spatial grouping" (each frame split into connected regions whose
token count is bounded by the attention block capacity C), the fused
preparation section (each region packed into one contiguous block; the
inverse index map restores token order) and the routing appendix (valid
counts n_a exclude padding).

This build fixes the regions to 8x8 spatial tiles per frame (C = 64):
block a = t*nI*nJ + i*nJ + j with nI = ceil(Hg/8), nJ = ceil(Wg/8). The
slots of a block hold its valid tokens in row-major order, followed by
padding. Tokens are numbered frame-major raster: n = t*Hg*Wg + y*Wg + x.
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


def gather_slots(X, slot2tok):
    """X [N, d] -> [R, 64, d] in slot order, padding slots set to 0."""
    R = slot2tok.size // CAP
    out = np.zeros((slot2tok.size, X.shape[1]), dtype=X.dtype)
    valid = slot2tok >= 0
    out[valid] = X[slot2tok[valid]]
    return out.reshape(R, CAP, X.shape[1])
