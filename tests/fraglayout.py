"""Index shuffles between the oracle's slot-ordered arrays [R, 64, d] and the
fragment order of the encoded-operand sections documented in include/da2.h.

Pure indexing: no arithmetic of the method happens here."""
import numpy as np


def kappa(j, r):
    return 32 * j + 16 * ((r // 4) % 2) + 4 * (r // 8) + r % 4


def _lanes():
    lane = np.arange(64)
    return lane % 32, lane // 32


def index_q4(d, permute_keys):
    """(slot, ch) index arrays [2, d/16, 64, 8] of the Q4 / K4 sections."""
    r, g = _lanes()
    jq = np.arange(2)[:, None, None, None]
    s = np.arange(d // 16)[None, :, None, None]
    e = np.arange(8)[None, None, None, :]
    rr, gg = r[None, None, :, None], g[None, None, :, None]
    slot = kappa(jq, rr) if permute_keys else 32 * jq + rr
    ch = 16 * s + 8 * gg + e
    return np.broadcast_arrays(slot, ch)


def index_q8(d, permute_keys):
    """(slot, ch) index arrays [2, d/32, 64, 16] of the Q8 / K8 sections."""
    r, g = _lanes()
    jq = np.arange(2)[:, None, None, None]
    s = np.arange(d // 32)[None, :, None, None]
    e = np.arange(16)[None, None, None, :]
    rr, gg = r[None, None, :, None], g[None, None, :, None]
    slot = kappa(jq, rr) if permute_keys else 32 * jq + rr
    ch = 32 * s + 16 * gg + e
    return np.broadcast_arrays(slot, ch)


def index_v4(d):
    """(slot, ch) index arrays [d/32, 4, 64, 8] of the V4 section."""
    r, g = _lanes()
    t = np.arange(d // 32)[:, None, None, None]
    s = np.arange(4)[None, :, None, None]
    e = np.arange(8)[None, None, None, :]
    rr, gg = r[None, None, :, None], g[None, None, :, None]
    slot = 32 * (s // 2) + 16 * gg + 8 * (s % 2) + e
    ch = 32 * t + rr
    return np.broadcast_arrays(slot, ch)


def index_v8(d):
    """(slot, ch) index arrays [d/32, 2, 64, 16] of the V8 section."""
    r, g = _lanes()
    t = np.arange(d // 32)[:, None, None, None]
    h = np.arange(2)[None, :, None, None]
    e = np.arange(16)[None, None, None, :]
    rr, gg = r[None, None, :, None], g[None, None, :, None]
    slot = 32 * h + 16 * gg + e
    ch = 32 * t + rr
    return np.broadcast_arrays(slot, ch)


def kappa_mx(j, r):
    return 32 * ((r // 4) % 2) + 16 * j + 4 * (r // 8) + r % 4


def index_mx_qk(d, permute_keys):
    """(slot, ch) index arrays [2, d/64, 64, 32] of the codes in the data
    fragments of the Q4mx / K4mx sections (tile, step, lane, code)."""
    r, g = _lanes()
    jq = np.arange(2)[:, None, None, None]
    s = np.arange(d // 64)[None, :, None, None]
    i = np.arange(32)[None, None, None, :]
    rr, gg = r[None, None, :, None], g[None, None, :, None]
    slot = kappa_mx(jq, rr) if permute_keys else 32 * jq + rr
    ch = 64 * s + 32 * gg + i
    return np.broadcast_arrays(slot, ch)


def index_mx_v(d):
    """(slot, ch) index arrays [d/32, 64, 32] of the V4mx data codes."""
    r, g = _lanes()
    t = np.arange(d // 32)[:, None, None]
    i = np.arange(32)[None, None, :]
    rr, gg = r[None, :, None], g[None, :, None]
    return np.broadcast_arrays(32 * gg + i, 32 * t + rr)


def _pack_nibbles(codes):
    """[..., 32] 4-bit codes -> [..., 16] bytes, code 2b in the low nibble of byte b."""
    c = codes.astype(np.uint8)
    return (c[..., 0::2] & 0xF) | ((c[..., 1::2] & 0xF) << 4)


def mx_section(kind, codes, kexp):
    """Bytes [R, (d/32 + 1) * 1024] of an MXFP4 section.

    kind "Q", "K": codes [R, 64, d] (slot ordered), kexp [R, 64, d/32] block
    exponents of (slot, 32-channel block); kind "V": codes [R, 64, d],
    kexp [R, 2, d] of (32-slot block, channel)."""
    R, _, d = codes.shape
    r, g = _lanes()
    words = np.zeros((R, 64, 4), np.uint32)
    if kind in ("Q", "K"):
        slot, ch = index_mx_qk(d, kind == "K")
        data = codes[:, slot, ch]                                     # [R, 2, d/64, 64, 32]
        data = data.reshape(R, 2 * (d // 64), 64, 32)
        for jq in range(2):
            for s in range(d // 64):
                srow = kappa_mx(jq, r) if kind == "K" else 32 * jq + r
                words[:, :, jq * (d // 64) + s] = kexp[:, srow, 2 * s + g] + 127
    else:
        slot, ch = index_mx_v(d)
        data = codes[:, slot, ch]                                     # [R, d/32, 64, 32]
        for t in range(d // 32):
            words[:, :, t] = kexp[:, g, 32 * t + r] + 127
    frags = np.concatenate([_pack_nibbles(data), words.view(np.uint8).reshape(R, 1, 64, 16)], axis=1)
    return frags.reshape(R, -1)


SECTIONS = {
    "Q4": (lambda d: index_q4(d, False), np.float16),
    "K4": (lambda d: index_q4(d, True), np.float16),
    "V4": (index_v4, np.float16),
    "Q8": (lambda d: index_q8(d, False), np.int8),
    "K8": (lambda d: index_q8(d, True), np.int8),
    "V8": (index_v8, np.uint8),
    "Q16": (lambda d: index_q4(d, False), np.float16),   # 16-bit path: the Q4 / K4 / V4 layouts
    "K16": (lambda d: index_q4(d, True), np.float16),
    "V16": (index_v4, np.float16),
}


def to_frag(name, X):
    """Slot-ordered X [R, 64, d] -> fragment order [R, 64*d] of section ``name``."""
    idx, dtype = SECTIONS[name]
    slot, ch = idx(X.shape[2])
    return X[:, slot, ch].reshape(X.shape[0], -1).astype(dtype)


def from_frag(name, F, d):
    """Fragment order [R, 64*d] -> slot-ordered [R, 64, d]."""
    idx, dtype = SECTIONS[name]
    slot, ch = idx(d)
    out = np.zeros((F.shape[0], 64, d), dtype=F.dtype)
    out[:, slot, ch] = F.reshape((F.shape[0],) + slot.shape)
    return out
