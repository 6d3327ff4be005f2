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
    """[..., 2n] 4-bit codes -> [..., n] bytes, code 2b in the low nibble of byte b."""
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


def nv_section(kind, codes, scodes):
    """Bytes [R, 36 d] of a packed NVFP4 section.

    kind "Q", "K": codes [R, 64, d] E2M1 codes (slot ordered), scodes
    [R, 64, d/16] E4M3 codes of the (slot, 16-channel group) scales; kind
    "V": codes [R, 64, d], scodes [R, 4, d] E4M3 codes of the (16-slot group,
    channel) scales. The order is that of include/da2.h: per attention thread
    (wave w, lane) its code dwords, then the scale bytes."""
    R, _, d = codes.shape
    ns, nt = d // 16, d // 32
    r, g = _lanes()
    if kind in ("Q", "K"):
        slot, ch = index_q4(d, kind == "K")                           # [2, ns, 64, 8]
        frag = codes[:, slot, ch]                                     # [R, 2, ns, 64, 8]
        frag = frag.transpose(0, 1, 3, 2, 4)                          # [R, w, lane, s, 8]
        code_bytes = _pack_nibbles(frag).reshape(R, -1)                 # 32 d bytes
        w = np.arange(2)[:, None, None]
        rr = np.arange(32)[None, :, None]
        sg = np.arange(ns)[None, None, :]
        row = kappa(w, rr) if kind == "K" else 32 * w + rr
        scale_bytes = scodes[:, row, sg].reshape(R, -1)               # [R, 2*32*ns]
    else:
        slot, ch = index_v4(d)                                        # [nt, 4, 64, 8]
        frag = codes[:, slot, ch].reshape(R, 2, nt // 2, 4, 64, 8)    # [R, w, t2, s, lane, 8]
        frag = frag.transpose(0, 1, 4, 2, 3, 5)                       # [R, w, lane, t2, s, 8]
        code_bytes = _pack_nibbles(frag).reshape(R, -1)
        w = np.arange(2)[:, None, None, None]
        lane = np.arange(64)[None, :, None, None]
        t2 = np.arange(nt // 2)[None, None, :, None]
        h = np.arange(2)[None, None, None, :]
        t = w * (nt // 2) + t2
        kg = 2 * h + lane // 32
        scale_bytes = scodes[:, kg, 32 * t + lane % 32].reshape(R, -1)  # [R, 2*64*(nt/2)*2]
    out = np.concatenate([code_bytes, scale_bytes], axis=1).astype(np.uint8)
    assert out.shape[1] == 36 * d
    return out


SECTIONS = {
    "Q8": (lambda d: index_q8(d, False), np.int8),
    "K8": (lambda d: index_q8(d, True), np.int8),
    "V8": (index_v8, np.uint8),
    "Q16": (lambda d: index_q4(d, False), np.float16),   # 16-bit path: the fp16 fragment orders
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
