"""Pins for the operand encodings (format appendix, NVFP4 quantization
equation, uniform-quantizer bound of the reconstructed-operand appendix).

The scalar reference below is an independent brute-force transcription
with Python floats: float32 rounding through ``struct``, E4M3 / E2M1 casts
by exhaustive nearest search with ties to the even code.
"""
import struct

import numpy as np
import pytest

from oracle import encode, formats as F, partition


def r32(x):
    return struct.unpack("f", struct.pack("f", float(x)))[0]


def _nearest(grid_codes, x):
    a = abs(x)
    best = None
    for code, v in grid_codes:
        dist = abs(a - v)
        if best is None or dist < best[0] or (dist == best[0] and code % 2 == 0):
            best = (dist, code, v)
    return best[2] if x >= 0 else -best[2]


E4M3_GRID = [(c, (c & 7) / 8 * 2.0 ** -6 if (c >> 3) == 0 else (1 + (c & 7) / 8) * 2.0 ** ((c >> 3) - 7))
             for c in range(0x7F)]
E2M1_GRID = list(enumerate([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]))


def e4m3_bf(x):
    return 448.0 if x >= 448 else (-448.0 if x <= -448 else _nearest(E4M3_GRID, x))


def e2m1_bf(x):
    return 6.0 if x >= 6 else (-6.0 if x <= -6 else _nearest(E2M1_GRID, x))


def _tiny(seed=0, T=1, Hg=13, Wg=11, d=32):
    rng = np.random.default_rng(seed)
    N = T * Hg * Wg
    X = (rng.standard_normal((N, d)) * rng.uniform(0.1, 3, d)).astype(np.float32)
    return X, partition.tile_partition(T, Hg, Wg)


def test_int8_scalar_brute_force_and_half_step_bound():
    X, (slot2tok, n_a, _) = _tiny()
    Xs = partition.gather_slots(X, slot2tok)
    q, delta = encode.int8_blocks(Xs, n_a)
    for a in range(n_a.size):
        vals = [float(v) for v in Xs[a, :n_a[a]].reshape(-1)]
        amax = max(abs(v) for v in vals)
        dl = r32(r32(amax / 127.0) + r32(1e-7))
        assert delta[a] == np.float32(dl)
        inv = r32(1.0 / dl)
        for k, v in enumerate(vals[:300]):
            y = r32(v * inv)
            want = int(abs(y) + 0.5) * (1 if y >= 0 else -1)
            assert q[a].reshape(-1)[k] == want
        rec = q[a, :n_a[a]].astype(np.float64) * float(delta[a])
        # uniform quantizer: error at most half a step (up to the float32 rounding of x*inv)
        assert np.all(np.abs(rec - Xs[a, :n_a[a]]) <= float(delta[a]) * (0.5 + 1e-6))
        assert np.all(q[a, n_a[a]:] == 0)


def test_e4m3_v_scalar_brute_force():
    X, (slot2tok, n_a, _) = _tiny(1)
    X[:, 3] = 0.0                                    # an all-zero channel
    Vs = partition.gather_slots(X, slot2tok)
    v8, dV = encode.e4m3_values_per_channel(Vs, n_a)
    for c in range(X.shape[1]):
        amax = max(abs(float(v)) for v in X[:, c])
        dl = r32(amax / 2.25)
        assert dV[c] == np.float32(dl)
        if dl == 0:
            assert np.all(v8[:, :, c] == 0)
            continue
        inv = r32(1.0 / dl)
        for a in range(0, n_a.size):
            for s in range(0, 64, 7):
                assert v8[a, s, c] == e4m3_bf(r32(float(Vs[a, s, c]) * inv))
    assert np.abs(v8).max() <= 2.25 + 1e-6


def _nvfp4_group_bf(xs, g):
    amax = max(abs(float(x)) for x in xs)
    sixg = r32(6.0 * g)
    sigma = e4m3_bf(r32(amax / sixg))
    if sigma == 0:
        return sigma, [0.0] * len(xs)
    inv = r32(1.0 / r32(g * sigma))
    return sigma, [e2m1_bf(r32(float(x) * inv)) for x in xs]


def test_nvfp4_qk_and_v_scalar_brute_force():
    X, (slot2tok, n_a, _) = _tiny(2)
    X[5, :16] = 0.0                                  # a zero group
    enc = encode.encode_head(X, X, X, slot2tok, n_a)
    g = float(enc["gQ"])
    assert enc["gQ"] == np.float32(r32(float(np.abs(X).max()) / 2688.0))
    Xs = partition.gather_slots(X, slot2tok)
    for a in range(n_a.size):
        for s in range(0, 64, 5):
            for k in range(X.shape[1] // 16):
                sig, e = _nvfp4_group_bf(Xs[a, s, 16 * k:16 * k + 16], g)
                assert enc["sQ"][a, s, k] == sig
                assert list(enc["eQ"][a, s, 16 * k:16 * k + 16]) == e
        for c in range(0, X.shape[1], 3):
            for k in range(4):
                sig, e = _nvfp4_group_bf(Xs[a, 16 * k:16 * k + 16, c], float(enc["gV"]))
                assert enc["sV"][a, k, c] == sig
                assert list(enc["eV"][a, 16 * k:16 * k + 16, c]) == e


def test_nvfp4_reconstruction_error_bound():
    """Each reconstructed value is within half an E2M1 step of the group's
    scale: |x - g sigma e| <= g sigma * step/2 with step <= 2 (saturation aside,
    the scale rounding can push x/(g sigma) up to 6 * (1 + 2^-4))."""
    X, (slot2tok, n_a, _) = _tiny(3)
    enc = encode.encode_head(X, X, X, slot2tok, n_a)
    rec = encode.reconstruct(enc)
    Xs = partition.gather_slots(X, slot2tok).astype(np.float64)
    s = np.repeat(enc["sQ"], 16, axis=2) * float(enc["gQ"])
    err = np.abs(rec["Qh4"] - Xs)
    assert np.all(err <= s * 1.0 + s * 6 * 2 ** -4 + 1e-12)
    assert np.all(np.abs(rec["Qh4"]) <= 6 * s + 1e-12)
    # the f16 container holds sigma*e exactly
    se = np.repeat(enc["sQ"], 16, axis=2) * enc["eQ"]
    assert np.array_equal(se.astype(np.float16).astype(np.float64), se)


def test_padding_encodes_to_zero():
    X, (slot2tok, n_a, _) = _tiny(4)
    enc = encode.encode_head(X, X, X, slot2tok, n_a)
    for a in np.nonzero(n_a < 64)[0]:
        for key in ("q8", "k8", "v8", "eQ", "eK", "eV"):
            assert np.all(enc[key][a, n_a[a]:] == 0)


def test_fp16_operands_are_half_casts():
    """16-bit path operands: the slot-ordered values cast to IEEE half
    (checked with Python's half packing); padding slots are zero."""
    X, layout = _tiny(4)
    slot2tok, n_a, _ = layout
    enc = encode.encode_head(X, X, X, slot2tok, n_a)
    Xs = partition.gather_slots(X, slot2tok)
    for key in ("q16", "k16", "v16"):
        got = enc[key].astype(np.float64)
        assert got.dtype == np.float64 and enc[key].dtype == np.float16
        for idx in zip(*np.nonzero(np.ones(Xs.shape[:2], bool))):
            row = Xs[idx]
            want = [struct.unpack("e", struct.pack("e", float(v)))[0] for v in row[:4]]
            assert list(got[idx][:4]) == want
        pad = np.arange(64)[None, :] >= n_a[:, None]
        assert np.all(got[pad] == 0)


def _mx_brute(block):
    """OCP MX block of E2M1 elements, scalar Python: X = 2^(floor(log2 amax) - 2)."""
    import math
    amax = max(abs(float(v)) for v in block)
    if amax == 0:
        return -127, [0.0] * len(block)
    m, e = math.frexp(amax)            # amax = m 2^e, m in [0.5, 1)
    k = max(-127, min(127, e - 1 - 2))
    return k, [e2m1_bf(float(v) / 2.0 ** k) for v in block]


def test_mx_scalar_brute_force_and_top_code():
    """MXFP4 blocks against a scalar transcription of the OCP rule; the block
    maximum always lands on E2M1 4 or 6 (amax / X in [4, 8), 6 saturating)."""
    rng = np.random.default_rng(21)
    X = (rng.standard_normal((40, 32)) * np.exp(rng.uniform(-8, 8, (40, 1)))).astype(np.float32)
    X[0] = 0.0
    X[1, :] = 0.0
    X[1, 5] = -3.0
    k, e = encode.mx_groups(X.astype(np.float64))
    for i in range(X.shape[0]):
        kb, eb = _mx_brute(X[i])
        assert k[i] == kb
        assert list(e[i]) == eb
        if np.abs(X[i]).max() > 0:
            assert np.abs(e[i]).max() in (4.0, 6.0)


def test_mx_head_encoding_layout_and_reconstruction():
    """Q/K blocks run along channels (32 per token), V blocks along 32 key slots
    per channel; padding stays zero; |x - x_hat| <= 2X (half the top step is X,
    saturation of (6, 8) adds at most 2X)."""
    X, layout = _tiny(7, d=64)
    slot2tok, n_a, _ = layout
    enc = encode.encode_head_mx(X, X, X, slot2tok, n_a)
    rec = encode.reconstruct_mx(enc)
    Xs = partition.gather_slots(X, slot2tok).astype(np.float64)
    R = Xs.shape[0]
    kq, eq = encode.mx_groups(Xs.reshape(R, 64, 2, 32))
    np.testing.assert_array_equal(enc["kQ"], kq)
    np.testing.assert_array_equal(rec["Qh4"], np.ldexp(1.0, np.repeat(kq, 32, axis=2)) * eq.reshape(R, 64, 64))
    for a in range(R):
        for c in (0, 17, 63):
            for g in range(2):
                kb, eb = _mx_brute(Xs[a, 32 * g:32 * g + 32, c])
                assert enc["kV"][a, g, c] == kb
                assert list(enc["eV"][a, 32 * g:32 * g + 32, c]) == eb
    bound_q = 2 * np.ldexp(1.0, np.repeat(enc["kQ"], 32, axis=2))
    assert np.all(np.abs(rec["Qh4"] - Xs) <= bound_q)
    pad = np.arange(64)[None, :] >= n_a[:, None]
    assert np.all(rec["Vh4"][pad] == 0) and np.all(rec["Qh4"][pad] == 0)
