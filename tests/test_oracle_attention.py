"""Pins for the phased attention of the oracle.

* No-quant mode with nothing skipped equals textbook dense attention
  (dense-operator equation).
* Skipping a block removes exactly its mass: O^Omega = (O^dense - sum_{v in b}
  P_uv V_v) / (1 - delta_u) (support-removal step of the Lemma 3.2 proof).
* In no-quant mode the order of blocks does not matter (online rescaling
  is exact), and V == 1 gives O == 1 (rows sum to one).
* The closed form equals the block-by-block recurrence with the Enter /
  Exit unit changes (precision-state-conversion equation).
* Lemma 3.2 (block form) holds for every query with residuals measured on
  the actual operands.
* Hand-derived closed forms: equal logits make every unnormalized weight
  1; NVFP4 then reproduces 1 exactly and the INT8 path gives
  E4M3(2^8.807) * 2^-8.807 = 448 / 2^8.807.
* Scalar brute force of the two weight quantizers (NVFP4 probability
  equation; eta * E4M3(P / eta) of the INT8 path).
"""
import struct

import numpy as np
import pytest

from oracle import attention as att, encode, partition, rank
from test_oracle_encode import e4m3_bf, e2m1_bf


def _case(seed=0, T=2, Hg=13, Wg=11, d=32, scale=1.0):
    rng = np.random.default_rng(seed)
    N = T * Hg * Wg
    Q = (rng.standard_normal((N, d)) * scale).astype(np.float32)
    K = (rng.standard_normal((N, d)) * scale).astype(np.float32)
    V = rng.standard_normal((N, d)).astype(np.float32)
    layout = partition.tile_partition(T, Hg, Wg)
    return Q, K, V, layout


def _exact_ops(Q, K, V, layout):
    slot2tok, n_a, _ = layout
    return att.Operands.exact(*(partition.gather_slots(X, slot2tok) for X in (Q, K, V)), n_a)


def _quant_ops(Q, K, V, layout):
    slot2tok, n_a, _ = layout
    enc = encode.encode_head(Q, K, V, slot2tok, n_a)
    return enc, att.Operands.quantized(encode.reconstruct(enc), n_a)


def _rows(layout, a):
    slot2tok, n_a, _ = layout
    return slot2tok[a * 64: a * 64 + n_a[a]]


def test_noquant_dense_equivalence():
    Q, K, V, layout = _case()
    ops = _exact_ops(Q, K, V, layout)
    R = layout[1].size
    Od = att.dense_attention(Q, K, V)
    for a in range(R):
        blocks = np.arange(R)
        O4 = att.attend(ops, a, blocks, [])
        O8 = att.attend(ops, a, [], blocks)
        Om = att.attend(ops, a, blocks[::2], blocks[1::2])
        for O in (O4, O8, Om):
            np.testing.assert_allclose(O, Od[_rows(layout, a)], rtol=1e-12, atol=1e-12)


def test_skip_removes_exactly_its_mass():
    Q, K, V, layout = _case(1, scale=1.5)
    slot2tok, n_a, _ = layout
    ops = _exact_ops(Q, K, V, layout)
    R = n_a.size
    S = Q.astype(np.float64) @ K.T.astype(np.float64) / np.sqrt(Q.shape[1])
    P = np.exp(S - S.max(axis=1, keepdims=True))
    P /= P.sum(axis=1, keepdims=True)
    Od = P @ V.astype(np.float64)
    for a, skip in [(0, 3), (2, 0), (5, 5)]:
        keep = [b for b in range(R) if b != skip]
        O = att.attend(ops, a, keep[:3], keep[3:])
        q = _rows(layout, a)
        kb = _rows(layout, skip)
        delta = P[q][:, kb].sum(axis=1)
        want = (Od[q] - P[q][:, kb] @ V[kb].astype(np.float64)) / (1 - delta)[:, None]
        np.testing.assert_allclose(O, want, rtol=1e-12, atol=1e-12)


def test_noquant_order_invariance_and_unit_rows():
    Q, K, V, layout = _case(2, scale=2.0)
    slot2tok, n_a, _ = layout
    R = n_a.size
    ops = _exact_ops(Q, K, V, layout)
    rng = np.random.default_rng(0)
    for a in range(R):
        blocks = rng.permutation(R)[:5]
        O1 = att.attend(ops, a, sorted(blocks[:2]), sorted(blocks[2:]))
        O2 = att.attend(ops, a, sorted(blocks[3:]), sorted(blocks[:3]))
        np.testing.assert_allclose(O1, O2, rtol=1e-12, atol=1e-13)
    ones = att.Operands.exact(partition.gather_slots(Q, slot2tok), partition.gather_slots(K, slot2tok),
                              np.ones((R, 64, Q.shape[1])), n_a)
    for a in range(R):
        np.testing.assert_allclose(att.attend(ones, a, [0, 2], [1, 3]), 1.0, rtol=0, atol=1e-14)


@pytest.mark.parametrize("lists", [([0, 2, 5], [1, 3]), ([], [0, 4]), ([1, 2], []), ([0], [0]), ([], [])])
def test_closed_form_equals_sequential_enter_exit(lists):
    Q, K, V, layout = _case(3, scale=1.5)
    enc, ops = _quant_ops(Q, K, V, layout)
    l4, l8 = lists
    for a in range(layout[1].size):
        O1 = att.attend(ops, a, l4, l8)
        O2 = att.attend_sequential(ops, a, l4, l8, enc["dV"], float(enc["gV"]))
        np.testing.assert_allclose(O1, O2, rtol=1e-12, atol=1e-13)
        if not (l4 or l8):
            assert np.all(O1 == 0)


def test_lemma_bound_holds():
    Q, K, V, layout = _case(4, scale=1.8)
    slot2tok, n_a, _ = layout
    enc, ops = _quant_ops(Q, K, V, layout)
    exact = _exact_ops(Q, K, V, layout)
    rng = np.random.default_rng(1)
    R = n_a.size
    for a in range(R):
        perm = rng.permutation(R)
        l8, l4 = sorted(perm[:2]), sorted(perm[2:5])
        lhs, rhs = att.lemma_bound(ops, exact, a, l4, l8, Q, K, V, slot2tok)
        assert np.all(lhs <= rhs * (1 + 1e-9) + 1e-12), (a, (lhs - rhs).max())


def test_equal_logits_closed_forms():
    """Q = 0 makes every logit 0, so every unnormalized weight is 1."""
    Q, K, V, layout = _case(5)
    Q[:] = 0.0
    slot2tok, n_a, _ = layout
    enc, ops = _quant_ops(Q, K, V, layout)
    rec = encode.reconstruct(enc)
    R = n_a.size
    for a in (0, 3):
        q = _rows(layout, a)
        blocks = [1, 2]
        kslots = np.concatenate([np.arange(b * 64, b * 64 + n_a[b]) for b in blocks])
        O4 = att.attend(ops, a, blocks, [])
        mean4 = rec["Vh4"].reshape(-1, Q.shape[1])[kslots].mean(axis=0)
        np.testing.assert_allclose(O4, np.broadcast_to(mean4, O4.shape), rtol=1e-13, atol=1e-14)
        O8 = att.attend(ops, a, [], blocks)
        mean8 = rec["Vh8"].reshape(-1, Q.shape[1])[kslots].mean(axis=0)
        np.testing.assert_allclose(O8, np.broadcast_to(mean8 * 448.0 / 2 ** 8.807, O8.shape),
                                   rtol=1e-13, atol=1e-14)


def test_weight_quantizers_scalar_brute_force():
    rng = np.random.default_rng(6)
    Pt = np.exp(-rng.exponential(3.0, (7, 64)))
    Pt[0, :16] = 0.0                                 # zero group
    W4 = att.quant_weights_fp4(Pt)
    W8 = att.quant_weights_fp8(Pt)
    eta = 2.0 ** -8.807
    for u in range(Pt.shape[0]):
        for k in range(4):
            grp = Pt[u, 16 * k:16 * k + 16]
            sig = e4m3_bf(448.0 * max(grp))
            for i, p in enumerate(grp):
                want = 0.0 if sig == 0 else sig / 2688.0 * e2m1_bf(2688.0 * p / sig)
                assert W4[u, 16 * k + i] == pytest.approx(want, rel=1e-15, abs=0)
        for v in range(64):
            assert W8[u, v] == pytest.approx(eta * e4m3_bf(Pt[u, v] / eta), rel=1e-15, abs=0)
    # the printed dequantization scale agrees with 2^-8.807 to the digits given
    assert abs(0.0022326917 - eta) < 5e-10


def test_precision_ordering_of_error():
    """Nothing skipped: all-8-bit is closer to dense than mixed, which is closer
    than all-4-bit (same inputs)."""
    Q, K, V, layout = _case(7, scale=1.5)
    enc, ops = _quant_ops(Q, K, V, layout)
    R = layout[1].size
    Od = att.dense_attention(Q, K, V)
    err = {}
    for name, split in (("8", 0), ("mix", R // 2), ("4", R)):
        num = den = 0.0
        for a in range(R):
            blocks = np.arange(R)
            O = att.attend(ops, a, blocks[:split], blocks[split:])
            ref = Od[_rows(layout, a)]
            num += ((O - ref) ** 2).sum()
            den += (ref ** 2).sum()
        err[name] = np.sqrt(num / den)
    assert err["8"] < err["mix"] < err["4"]
    assert err["8"] < 0.05 and err["4"] < 0.3


def test_noquant_dense_equivalence_with_sixteen_bit_segment():
    """No-quant mode: any split of all blocks over the three phases, including
    the 16-bit one, is textbook dense attention."""
    Q, K, V, layout = _case(8)
    ops = _exact_ops(Q, K, V, layout)
    R = layout[1].size
    Od = att.dense_attention(Q, K, V)
    for a in range(R):
        b = np.arange(R)
        for split in ((b, [], []), ([], [], b), (b[0::3], b[1::3], b[2::3])):
            O = att.attend(ops, a, *split)
            np.testing.assert_allclose(O, Od[_rows(layout, a)], rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("lists", [([0, 2], [1], [3, 5]), ([], [], [0, 1, 4]), ([1], [], [2]), ([], [3], [0])])
def test_closed_form_equals_sequential_three_phases(lists):
    """The closed form equals the block recurrence whose 16-bit phase follows
    the INT8 Exit (or the NVFP4 phase) in the common units."""
    Q, K, V, layout = _case(9, scale=1.5)
    enc, ops = _quant_ops(Q, K, V, layout)
    l4, l8, l16 = lists
    for a in range(layout[1].size):
        O1 = att.attend(ops, a, l4, l8, l16)
        O2 = att.attend_sequential(ops, a, l4, l8, enc["dV"], float(enc["gV"]), l16)
        np.testing.assert_allclose(O1, O2, rtol=1e-12, atol=1e-13)


def test_sixteen_bit_only_is_dense_on_half_operands_within_weight_rounding():
    """All blocks on the 16-bit path: the output is dense attention over the
    half-precision Q, K, V except that the numerator uses half-precision
    weights. Each normal half weight is within 2^-11 of its value relative,
    a subnormal one within 2^-25 absolute, and the denominator is at least 1
    (the weight of the final maximum), so |O - O_dense16| <= (2^-11 +
    n_keys 2^-25) max|V|."""
    Q, K, V, layout = _case(10, scale=1.2)
    slot2tok, n_a, _ = layout
    enc, ops = _quant_ops(Q, K, V, layout)
    Q16, K16, V16 = (X.astype(np.float16).astype(np.float64) for X in (Q, K, V))
    Od = att.dense_attention(Q16, K16, V16)
    R = n_a.size
    bound = (2.0 ** -11 + K.shape[0] * 2.0 ** -25) * np.abs(V16).max()
    worst = 0.0
    for a in range(R):
        O = att.attend(ops, a, [], [], np.arange(R))
        err = np.abs(O - Od[_rows(layout, a)]).max()
        worst = max(worst, err)
        assert err <= bound, (a, err, bound)
    assert worst > 0          # the weight rounding is really applied


def test_fp16_weights_scalar():
    """The 16-bit path's weight is the nearest half (ties to even), checked
    with Python's own IEEE half packing."""
    rng = np.random.default_rng(12)
    Pt = np.concatenate([np.exp(-rng.exponential(4.0, 500)), [1.0, 2.0 ** -24, 3 * 2.0 ** -26, 1 + 2.0 ** -11]])
    W = att.quant_weights_fp16(Pt)
    for p, w in zip(Pt, W):
        assert w == struct.unpack("e", struct.pack("e", float(p)))[0]


def _mx_ops(Q, K, V, layout):
    slot2tok, n_a, _ = layout
    enc = encode.encode_head(Q, K, V, slot2tok, n_a)
    encm = encode.encode_head_mx(Q, K, V, slot2tok, n_a)
    return enc, att.Operands.quantized(encode.reconstruct(enc), n_a, encode.reconstruct_mx(encm)), encm


@pytest.mark.parametrize("lists", [([0, 2, 5], [1, 3], []), ([1, 4], [], [2]), ([0], [3], [1])])
def test_mx_closed_form_equals_sequential(lists):
    """With MXFP4 the 4-bit phase accumulates in the common units; the closed
    form still equals the recurrence with Enter / Exit."""
    Q, K, V, layout = _case(13, scale=1.5)
    enc, ops, _ = _mx_ops(Q, K, V, layout)
    l4, l8, l16 = lists
    for a in range(layout[1].size):
        O1 = att.attend(ops, a, l4, l8, l16)
        O2 = att.attend_sequential(ops, a, l4, l8, enc["dV"], float(enc["gV"]), l16, mx=True)
        np.testing.assert_allclose(O1, O2, rtol=1e-12, atol=1e-13)


def test_mx_equal_logits_give_exact_mean():
    """Equal logits: every Pt is 1, X = 2^-2, Pt / X = 4 is an E2M1 value, so
    every MX weight is exactly 1 and O is the mean of the MX values."""
    Q, K, V, layout = _case(14)
    Q[:] = 0.0
    slot2tok, n_a, _ = layout
    _, ops, encm = _mx_ops(Q, K, V, layout)
    rec = encode.reconstruct_mx(encm)
    blocks = [0, 3]
    kslots = np.concatenate([np.arange(b * 64, b * 64 + n_a[b]) for b in blocks])
    O = att.attend(ops, 1, blocks, [])
    mean = rec["Vh4"].reshape(-1, Q.shape[1])[kslots].mean(axis=0)
    np.testing.assert_allclose(O, np.broadcast_to(mean, O.shape), rtol=1e-13, atol=1e-14)


def test_mx_weights_scalar_brute_force():
    from test_oracle_encode import _mx_brute
    rng = np.random.default_rng(15)
    Pt = np.exp(-rng.exponential(3.0, (9, 64)))
    Pt[0, :32] = 0.0
    Pt[1, 32:] = 2.0 ** -140                      # below the smallest scale
    W = att.quant_weights_mx(Pt)
    for u in range(Pt.shape[0]):
        for g in range(2):
            k, e = _mx_brute(Pt[u, 32 * g:32 * g + 32])
            assert list(W[u, 32 * g:32 * g + 32]) == [2.0 ** k * v for v in e]
