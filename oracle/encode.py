"""Operand encodings of the 8-bit and 4-bit paths (oracle; test infrastructure).

Paper: appendix "Quantization Formats and Scales".

* INT8 Q/K: one float32 scale per query block / physical key block,
  delta = max|X| / 127 + 1e-7, codes = X / delta rounded to nearest, ties
  away from zero.
* E4M3 V (probability-value product of the INT8 path): per-channel scale
  delta_c = max_v |V_vc| / 2.25 over all valid keys of the head; all-zero
  channels encode to zero.
* FP16 Q/K/V (16-bit path, INT8-and-FP16 paragraph): the values cast to
  IEEE half precision, round to nearest even.
* MXFP4 (a 4-bit alternative that gfx950's matrix cores take natively; not
  a format of the paper): OCP microscaling with blocks of 32 along the
  reduction dimension (channels for Q and K, key slots within a block for
  V), a power-of-two scale X = 2^(floor(log2 max|x|) - 2) clamped to
  [2^-127, 2^127] (2^-127 for an all-zero block), elements E2M1(x / X)
  rounded to nearest even with saturation.
* NVFP4 (NVFP4 quantization equation): E2M1 values with an E4M3 scale per
  group of 16 along the reduction dimension (channels for Q and K, key
  slots within a block for V), a positive per-tensor scale g_X,
  sigma = E4M3(max|x| / (6 g)), x_hat = g sigma E2M1(x / (g sigma)); a group
  whose scale encodes to zero is all zeros.

Readings (the paper leaves these open):
* Scales and codes are evaluated with float32 operations in this fixed
  order, each rounded once: delta = f32(f32(amax/127) + f32(1e-7));
  division by a scale is a multiplication by its float32 reciprocal,
  y = f32(x * f32(1/scale)), and the cast is applied to y.
* g_X = f32(max|X| / 2688) per (batch, head), so that local scales can use
  the whole E4M3 range (2688 = 6 * 448); g_X = 1 for an all-zero tensor.
* The per-channel delta_c and g_X are per (batch, head), the unit the
  paper's analysis works in.
* Padding slots are zero and encode to zero in every format.
"""
import numpy as np

from .formats import e4m3, e2m1, half_away, f32
from .partition import CAP, gather_slots

GROUP = 16


def _recip(x):
    return f32(np.float32(1.0) / np.asarray(x, np.float32))


def int8_blocks(Xs, n_a):
    """INT8 codes and per-block scales. Xs: [R, 64, d] float32 (padding 0)."""
    R = Xs.shape[0]
    amax = np.abs(Xs).reshape(R, -1).max(axis=1).astype(np.float32)
    delta = f32(f32(amax / np.float32(127.0)) + np.float32(1e-7))
    y = f32(Xs * _recip(delta)[:, None, None])
    q = np.clip(half_away(y), -127, 127).astype(np.int8)
    return q, delta


def e4m3_values_per_channel(Vs, n_a):
    """E4M3 values of V/delta_c and the per-channel scales delta_c [d]."""
    amax_c = np.abs(Vs).reshape(-1, Vs.shape[2]).max(axis=0).astype(np.float32)
    delta = f32(amax_c / np.float32(2.25))
    zero = delta == 0
    inv = np.where(zero, np.float32(0.0), _recip(np.where(zero, np.float32(1.0), delta)))
    y = f32(Vs * inv[None, None, :])
    v8 = e4m3(y)
    v8 = np.where(zero[None, None, :], 0.0, v8)
    return v8, delta


def nvfp4_global_scale(amax):
    g = f32(np.float32(amax) / np.float32(2688.0))
    return np.float32(1.0) if g == 0 else np.float32(g)


def nvfp4_groups(x, g):
    """NVFP4-encode ``x`` [..., G, 16] (groups on the last axis) with global
    scale g. Returns (sigma [..., G] E4M3 values, e [..., G, 16] E2M1 values)."""
    amax = np.abs(x).max(axis=-1).astype(np.float32)
    sixg = f32(np.float32(6.0) * np.float32(g))
    sigma = e4m3(f32(amax / sixg))
    zero = sigma == 0
    den = f32(np.float32(g) * np.where(zero, 1.0, sigma).astype(np.float32))
    inv = _recip(den)
    e = e2m1(f32(x * inv[..., None]))
    e = np.where(zero[..., None], 0.0, e)
    return sigma, e


MX_GROUP = 32


def mx_scale_exponents(amax):
    """E8M0 exponents k of the MX blocks: floor(log2 amax) - 2, clamped to
    [-127, 127]; -127 for a zero block."""
    amax = np.asarray(amax, dtype=np.float64)
    _, e = np.frexp(np.where(amax > 0, amax, 1.0))          # amax = f 2^e, f in [0.5, 1)
    k = (e - 1) - 2
    return np.where(amax > 0, np.clip(k, -127, 127), -127).astype(np.int64)


def mx_groups(x):
    """MXFP4-encode ``x`` [..., G, 32] (blocks on the last axis). Returns
    (k [..., G] scale exponents, e [..., G, 32] E2M1 values)."""
    k = mx_scale_exponents(np.abs(x).max(axis=-1))
    e = e2m1(np.asarray(x, np.float64) / np.ldexp(1.0, k)[..., None])
    return k, e


def encode_head_mx(Q, K, V, slot2tok, n_a):
    """MXFP4 operands of one head, slot ordered: kQ, kK [R,64,d/32] and
    eQ, eK [R,64,d]; kV [R,2,d] (32-slot blocks per channel) and eV [R,64,d]."""
    Qs, Ks, Vs = (gather_slots(X.astype(np.float32), slot2tok) for X in (Q, K, V))
    R, _, d = Qs.shape
    out = {}
    for name, Xs in (("Q", Qs), ("K", Ks)):
        k, e = mx_groups(Xs.reshape(R, CAP, d // MX_GROUP, MX_GROUP))
        out["k" + name], out["e" + name] = k, e.reshape(R, CAP, d)
    vt = Vs.reshape(R, CAP // MX_GROUP, MX_GROUP, d).transpose(0, 1, 3, 2)   # [R, 2, d, 32]
    k, e = mx_groups(vt)
    out["kV"] = k
    out["eV"] = e.transpose(0, 1, 3, 2).reshape(R, CAP, d)
    return out


def reconstruct_mx(enc):
    """MXFP4 operands in original units: Qh4/Kh4/Vh4 = 2^k e."""
    R, _, d = enc["eQ"].shape
    rec = {}
    for name in ("Q", "K"):
        rec[name + "h4"] = np.ldexp(1.0, np.repeat(enc["k" + name], MX_GROUP, axis=2)) * enc["e" + name]
    rec["Vh4"] = np.ldexp(1.0, np.repeat(enc["kV"], MX_GROUP, axis=1)) * enc["eV"]
    return rec


def encode_head(Q, K, V, slot2tok, n_a, amaxQ=None, amaxK=None, amaxV=None):
    """All operand encodings of one head. Q, K, V: [N, d] float32 values.

    Returns a dict with slot-ordered arrays (R blocks of 64 slots):
      q8, k8 int8 [R,64,d]; dQ, dK float32 [R]
      v8 E4M3 values [R,64,d]; dV float32 [d]
      gQ, gK, gV float32; sQ, sK E4M3 values [R,64,d/16]; eQ, eK [R,64,d];
      sV E4M3 values [R,4,d] (16-slot groups per channel); eV [R,64,d]
      q16, k16, v16 float16 [R,64,d] (16-bit path)
    """
    Qs, Ks, Vs = (gather_slots(X.astype(np.float32), slot2tok) for X in (Q, K, V))
    R, _, d = Qs.shape
    q8, dQ = int8_blocks(Qs, n_a)
    k8, dK = int8_blocks(Ks, n_a)
    v8, dV = e4m3_values_per_channel(Vs, n_a)
    out = dict(q8=q8, dQ=dQ, k8=k8, dK=dK, v8=v8, dV=dV,
               q16=Qs.astype(np.float16), k16=Ks.astype(np.float16), v16=Vs.astype(np.float16))
    amaxes = {"Q": amaxQ, "K": amaxK, "V": amaxV}
    for name, Xs, X in (("Q", Qs, Q), ("K", Ks, K)):
        amax = amaxes[name] if amaxes[name] is not None else np.abs(X).max()
        g = nvfp4_global_scale(amax)
        s, e = nvfp4_groups(Xs.reshape(R, CAP, d // GROUP, GROUP), g)
        out["g" + name], out["s" + name], out["e" + name] = g, s, e.reshape(R, CAP, d)
    amax = amaxV if amaxV is not None else np.abs(V).max()
    g = nvfp4_global_scale(amax)
    # V groups run along key slots: [R, 4 groups, 16 slots, d] -> groups on the slot axis.
    vt = Vs.reshape(R, CAP // GROUP, GROUP, d).transpose(0, 1, 3, 2)   # [R, 4, d, 16]
    s, e = nvfp4_groups(vt, g)                                          # s [R,4,d], e [R,4,d,16]
    out["gV"], out["sV"] = g, s
    out["eV"] = e.transpose(0, 1, 3, 2).reshape(R, CAP, d)
    return out


def reconstruct(enc):
    """Operands in original units (float64), as the attention uses them.

    Qh8/Kh8: delta * q; Vh8: delta_c * v8; Qh4/Kh4/Vh4: g * sigma * e;
    Qh16/Kh16/Vh16: the half-precision values."""
    R, _, d = enc["q8"].shape
    rec = {
        "Qh8": enc["q8"].astype(np.float64) * enc["dQ"].astype(np.float64)[:, None, None],
        "Kh8": enc["k8"].astype(np.float64) * enc["dK"].astype(np.float64)[:, None, None],
        "Vh8": enc["v8"] * enc["dV"].astype(np.float64)[None, None, :],
        "Qh16": enc["q16"].astype(np.float64),
        "Kh16": enc["k16"].astype(np.float64),
        "Vh16": enc["v16"].astype(np.float64),
    }
    for name in ("Q", "K"):
        s = np.repeat(enc["s" + name], GROUP, axis=2)                   # [R,64,d]
        rec[name + "h4"] = float(enc["g" + name]) * s * enc["e" + name]
    sV = np.repeat(enc["sV"], GROUP, axis=1)                            # [R,64,d]
    rec["Vh4"] = float(enc["gV"]) * sV * enc["eV"]
    return rec
