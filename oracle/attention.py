"""Phased mixed-precision attention with one shared online-softmax state
(oracle; test infrastructure).

Paper: "Phased execution" and "Cross-precision accumulation" (retained key
blocks of a query block are grouped into an NVFP4 segment, an INT8 segment
and a 16-bit segment, processed in that order; all blocks share the row
maxima, the denominator and the output numerator; one normalization at the
end), the NVFP4 probability equation, the INT8 and FP16 paragraph of the
format appendix, the precision-state-conversion equation (Enter / Exit),
the phased-execution appendix (the FP16 phase continues in the common
scale), "Weight Quantization under Shared Normalization" and the
reconstructed-output equation.

For one query region a with retained key blocks L = [list4 ascending ;
list8 ascending ; list16 ascending] and valid query u:

  s_uv  = Qhat_u . Khat_v / sqrt(d)     (reconstructed operands, float64)
  m_j   = max(m_{j-1}, max_{v in block j} s_uv)        (running maximum)
  Pt_uv = exp(s_uv - m_j)                              (unnormalized weight)
  4-bit block: sigma_P = E4M3(448 max_{v in G} Pt_uv) over 16-slot groups,
               w_uv = sigma_P / 2688 * E2M1(2688 Pt_uv / sigma_P)
  8-bit block: w_uv = eta * E4M3(Pt_uv / eta), eta = 2^-8.807
  16-bit block: w_uv = FP16(Pt_uv), Qhat, Khat, Vhat the FP16 values
  l = sum_j e^{m_j - m} sum_v Pt_uv,  U = sum_j e^{m_j - m} sum_v w_uv Vhat_v,
  O_u = U / l   (0 for a row with no retained block),  m = m_last.

The closed form above is the online recurrence with its rescalings
multiplied out (the shared-normalization appendix); ``attend_sequential``
runs the recurrence block by block with the Enter / Exit unit changes and
is used to check the closed form.

Readings: the running maximum is updated once per 64-slot key block; the
denominator takes the float32-before-conversion weights (here exact);
eta = 2^-8.807 exactly, the value the printed 0.0022326917 rounds; key
blocks ascend within a phase; padded key slots carry no weight; the FP16
weight is the round-to-nearest-even half-precision value of the exact Pt.
"""
import numpy as np

from .formats import e4m3, e2m1
from .partition import CAP

ETA = 2.0 ** -8.807
AMP = 2.0 ** 8.807          # 1 / ETA
FP4_P_SCALE = 2688.0        # 6 * 448
GROUP = 16


def quant_weights_fp4(Pt):
    """NVFP4 weights for Pt [..., 64] (16-slot groups on the last axis)."""
    g = Pt.reshape(Pt.shape[:-1] + (CAP // GROUP, GROUP))
    sigma = e4m3(448.0 * g.max(axis=-1))
    safe = np.where(sigma == 0, 1.0, sigma)
    e = e2m1(FP4_P_SCALE * g / safe[..., None])
    w = np.where(sigma[..., None] == 0, 0.0, sigma[..., None] / FP4_P_SCALE * e)
    return w.reshape(Pt.shape)


def quant_weights_fp8(Pt):
    """INT8-path weights: eta * E4M3(Pt / eta)."""
    return ETA * e4m3(AMP * Pt)


MX_GROUP = 32


def quant_weights_mx(Pt):
    """MXFP4 weights for Pt [..., 64]: 32-slot blocks, X = 2^(floor(log2 max) - 2)
    (clamped to [2^-127, 2^127]), w = X E2M1(Pt / X); a zero block stays zero."""
    g = np.asarray(Pt, np.float64).reshape(Pt.shape[:-1] + (CAP // MX_GROUP, MX_GROUP))
    amax = g.max(axis=-1)
    _, e = np.frexp(np.where(amax > 0, amax, 1.0))
    k = np.where(amax > 0, np.clip((e - 1) - 2, -127, 127), -127)
    X = np.ldexp(1.0, k)[..., None]
    return (X * e2m1(g / X)).reshape(Pt.shape)


def quant_weights_fp16(Pt):
    """16-bit path weights: Pt cast to IEEE half precision (round to nearest even)."""
    return np.asarray(Pt, np.float64).astype(np.float16).astype(np.float64)


def identity_weights(Pt):
    return Pt


class Operands:
    """Per-phase reconstructed operands of one head, slot ordered [R, 64, d].

    ``phases`` maps 4, 8 and 16 to (Qhat, Khat, Vhat, weight_quantizer)."""

    def __init__(self, n_a, phases):
        self.n_a = n_a
        self.phases = phases

    @classmethod
    def quantized(cls, rec, n_a, rec_mx=None):
        """Quantized operands; with ``rec_mx`` (reconstruct_mx) the 4-bit phase
        runs on MXFP4 operands and weights instead of NVFP4."""
        if rec_mx is not None:
            return cls(n_a, {4: (rec_mx["Qh4"], rec_mx["Kh4"], rec_mx["Vh4"], quant_weights_mx),
                             8: (rec["Qh8"], rec["Kh8"], rec["Vh8"], quant_weights_fp8),
                             16: (rec["Qh16"], rec["Kh16"], rec["Vh16"], quant_weights_fp16)})
        return cls(n_a, {4: (rec["Qh4"], rec["Kh4"], rec["Vh4"], quant_weights_fp4),
                         8: (rec["Qh8"], rec["Kh8"], rec["Vh8"], quant_weights_fp8),
                         16: (rec["Qh16"], rec["Kh16"], rec["Vh16"], quant_weights_fp16)})

    @classmethod
    def exact(cls, Qs, Ks, Vs, n_a):
        """No-quant mode: the original values on both paths, unquantized weights."""
        Q, K, V = (np.asarray(x, np.float64) for x in (Qs, Ks, Vs))
        return cls(n_a, {4: (Q, K, V, identity_weights), 8: (Q, K, V, identity_weights),
                         16: (Q, K, V, identity_weights)})


def _segment(ops, a, blocks, phase):
    """Logits [nq, nb, 64] (padding -inf), Vhat [nb, 64, d] and quantizer of one phase."""
    Qh, Kh, Vh, quant = ops.phases[phase]
    nq, d = ops.n_a[a], Qh.shape[2]
    blocks = np.asarray(blocks, dtype=np.int64)
    S = (Qh[a, :nq] @ Kh[blocks].reshape(-1, d).T / np.sqrt(d)).reshape(nq, blocks.size, CAP)
    pad = np.arange(CAP)[None, :] >= ops.n_a[blocks][:, None]           # [nb, 64]
    S = np.where(pad[None], -np.inf, S)
    return S, Vh[blocks], quant


def attend(ops, a, list4, list8, list16=(), return_parts=False):
    """Output rows [n_a[a], d] of query region a (closed form)."""
    nq = ops.n_a[a]
    d = ops.phases[4][0].shape[2]
    segs = [(_segment(ops, a, lst, p), p) for lst, p in ((list4, 4), (list8, 8), (list16, 16)) if len(lst)]
    if not segs:
        return np.zeros((nq, d))
    S = np.concatenate([s[0] for s, _ in segs], axis=1)                # [nq, nb, 64]
    m = np.maximum.accumulate(S.max(axis=2), axis=1)                    # running max per block
    Pt = np.exp(S - m[:, :, None])
    W = np.empty_like(Pt)
    Vh = np.concatenate([s[1] for s, _ in segs], axis=0)               # [nb, 64, d]
    j = 0
    for (Sp, _, quant), _p in segs:
        nb = Sp.shape[1]
        W[:, j:j + nb] = quant(Pt[:, j:j + nb])
        j += nb
    f = np.exp(m - m[:, -1:])                                           # e^{m_j - m_last}
    ell = (f * Pt.sum(axis=2)).sum(axis=1)
    U = (W * f[:, :, None]).reshape(nq, -1) @ Vh.reshape(-1, d)
    O = U / ell[:, None]
    if return_parts:
        return O, dict(S=S, m=m, Pt=Pt, W=W, f=f, ell=ell, U=U)
    return O


def attend_sequential(ops, a, list4, list8, dV, gV, list16=(), mx=False):
    """The online recurrence block by block, with the phase unit changes.

    Phase 4 accumulates U in units of g_V/2688 (its matrix products take
    sigma_P e_P and sigma_V e_V); Enter converts the state to the INT8
    path's units (U / (eta delta_c), l / eta); phase 8 accumulates the
    amplified weights Pt/eta and E4M3 codes times the E4M3 V codes; Exit
    converts back (precision-state-conversion equation); phase 16 then
    accumulates FP16 weights times FP16 values in the common units. With
    ``mx`` the 4-bit phase is MXFP4, whose power-of-two block scales the
    matrix products apply, so it accumulates in the common units."""
    nq = ops.n_a[a]
    d = ops.phases[4][0].shape[2]
    dV = np.asarray(dV, np.float64)
    m = np.full(nq, -np.inf)
    ell = np.zeros(nq)
    U = np.zeros((nq, d))
    unit4 = 1.0 if mx else FP4_P_SCALE / gV
    if len(list4):
        U = U * unit4                                                   # into phase-4 units
        for b in list4:
            S, Vh, quant = _segment(ops, a, [b], 4)
            S, Vh = S[:, 0], Vh[0]
            m_new = np.maximum(m, S.max(axis=1))
            alpha = np.exp(m - m_new)
            Pt = np.exp(S - m_new[:, None])
            ell = ell * alpha + Pt.sum(axis=1)
            U = U * alpha[:, None] + (quant(Pt) @ Vh) * unit4
            m = m_new
        U = U / unit4                                                   # back to common units
    if len(list8):
        scale = np.where(dV == 0, 0.0, 1.0 / (ETA * np.where(dV == 0, 1.0, dV)))
        U = U * scale[None, :]                                          # Enter
        ell = ell / ETA
        for b in list8:
            S, Vh, quant = _segment(ops, a, [b], 8)
            S, Vh = S[:, 0], Vh[0]
            m_new = np.maximum(m, S.max(axis=1))
            alpha = np.exp(m - m_new)
            Pamp = np.exp(S - m_new[:, None]) * AMP
            ell = ell * alpha + Pamp.sum(axis=1)
            v8 = np.where(dV == 0, 0.0, Vh / np.where(dV == 0, 1.0, dV))  # E4M3 codes' values
            U = U * alpha[:, None] + e4m3(Pamp) @ v8
            m = m_new
        U = U * (ETA * dV)[None, :]                                     # Exit
        ell = ell * ETA
    for b in list16:
        S, Vh, quant = _segment(ops, a, [b], 16)
        S, Vh = S[:, 0], Vh[0]
        m_new = np.maximum(m, S.max(axis=1))
        alpha = np.exp(m - m_new)
        Pt = np.exp(S - m_new[:, None])
        ell = ell * alpha + Pt.sum(axis=1)
        U = U * alpha[:, None] + quant(Pt) @ Vh
        m = m_new
    if not (len(list4) or len(list8) or len(list16)):
        return np.zeros((nq, d))
    return U / ell[:, None]


def dense_attention(Q, K, V):
    """Textbook softmax(QK^T / sqrt d) V in float64 (dense-operator equation)."""
    Q, K, V = (np.asarray(x, np.float64) for x in (Q, K, V))
    S = Q @ K.T / np.sqrt(Q.shape[1])
    P = np.exp(S - S.max(axis=1, keepdims=True))
    return (P / P.sum(axis=1, keepdims=True)) @ V


def lemma_bound(ops, exact, a, list4, list8, Qtok, Ktok, Vtok, slot2tok, list16=()):
    """Both sides of the block form of Lemma 3.2 for every valid query of region a.

    lhs_u = ||O_dense_u - Ohat_u||,
    rhs_u = 2 Vmax delta_u + e^{alpha_u} sum_b m_ub c_ub with
    c_ub = 2 Vmax (e^alpha_ub - 1) + e^alpha_ub [nu_ub + (Vmax + nu_ub) omega_ub],
    residuals measured on the actual operands (error-model and
    reconstructed-operand appendices)."""
    nq = ops.n_a[a]
    Qtok, Ktok, Vtok = (np.asarray(x, np.float64) for x in (Qtok, Ktok, Vtok))
    d = Qtok.shape[1]
    Oh, parts = attend(ops, a, list4, list8, list16, return_parts=True)
    toks_q = slot2tok[a * CAP: a * CAP + nq]
    Od = dense_attention(Qtok[toks_q], Ktok, Vtok)
    lhs = np.linalg.norm(Od - Oh, axis=1)
    Vmax = np.linalg.norm(Vtok, axis=1).max()
    blocks = list(list4) + list(list8) + list(list16)
    # exact logits of the retained blocks, same slot layout
    Se, _, _ = _segment(exact, a, blocks, 4)
    S, m, W, f = parts["S"], parts["m"], parts["W"], parts["f"]
    h = m[:, -1]
    w = np.exp(S - h[:, None, None])                                    # float weights at final reference
    what = W * f[:, :, None]                                            # reconstructed weights, same reference
    Pw = np.exp(Se - Se.max(axis=(1, 2), keepdims=True))
    Pomega = Pw / Pw.sum(axis=(1, 2), keepdims=True)
    m_ub = Pomega.sum(axis=2)
    valid = np.isfinite(S)
    with np.errstate(invalid="ignore"):
        alpha_ub = np.where(valid, np.abs(S - Se), 0.0).max(axis=2)
    segs = ((list4, 4), (list8, 8), (list16, 16))
    Vh = np.concatenate([ops.phases[p][2][lst] for lst, p in segs if len(lst)])
    Vx = np.concatenate([exact.phases[p][2][lst] for lst, p in segs if len(lst)])
    nu_b = np.linalg.norm(Vh - Vx, axis=2).max(axis=1)                  # [nb]
    nu_ub = np.broadcast_to(nu_b[None, :], m_ub.shape)
    omega_ub = np.abs(what - w).sum(axis=2) / np.maximum(w.sum(axis=2), 1e-300)
    c_ub = 2 * Vmax * np.expm1(alpha_ub) + np.exp(alpha_ub) * (nu_ub + (Vmax + nu_ub) * omega_ub)
    S_all = Qtok[toks_q] @ Ktok.T / np.sqrt(d)
    P_all = np.exp(S_all - S_all.max(axis=1, keepdims=True))
    P_all /= P_all.sum(axis=1, keepdims=True)
    keep = np.zeros(Ktok.shape[0], bool)
    kslots = np.concatenate([np.arange(b * CAP, b * CAP + ops.n_a[b]) for b in blocks])
    keep[slot2tok[kslots]] = True
    delta_u = P_all[:, ~keep].sum(axis=1)
    rhs = 2 * Vmax * delta_u + np.exp(alpha_ub.max(axis=1)) * (m_ub * c_ub).sum(axis=1)
    return lhs, rhs
