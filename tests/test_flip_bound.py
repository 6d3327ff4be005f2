"""The full-size GPU parity tests accept a row beyond the max-abs bar only
when the deviation is within the bar plus the flip bound (tests/oracle_pool.py):
what the weights whose quantizer inputs lie within FLIP_EPS of a rounding
midpoint can move the output. These CPU checks pin that bound: it is zero when
no weight is that close, it covers a planted flip of the closest weight, and it
does not cover a defect (a key block left out)."""
import numpy as np
import pytest

import oracle_pool
from oracle import attention, encode, formats, partition, rank
from synth import configs, gen
from gpu_harness import TOL_MAX_ABS


def _setup(w, h=0):
    Q, K, V = gen.generate(w, heads=[h])
    slot2tok, n_a, _ = partition.make_partition(w.partition, w.T, w.Hg, w.Wg)
    from oracle import draft
    A32, _ = draft.draft_head(Q[0, 0], K[0, 0], slot2tok, n_a, w.lam)
    cls = rank.rank_head(A32, *w.budgets, w.scope)
    enc = encode.encode_head(Q[0, 0], K[0, 0], V[0, 0], slot2tok, n_a)
    return attention.Operands.quantized(encode.reconstruct(enc), n_a), cls


W = configs.Workload("flip-2x16x32-h1-d64", B=1, H=1, d=64, T=2, Hg=16, Wg=32, dtype="fp32",
                     budgets=(30, 40, 100), scope="head", head_scale=True, seed=31)


def _closest_nvfp4_weight(ops, a, lists):
    """(query, block, slot, relative distance, step width, sigma) of the NVFP4
    weight whose quantizer input lies closest to an E2M1 midpoint."""
    _, parts = attention.attend(ops, a, *lists, return_parts=True)
    n4 = len(lists[0])
    g = parts["Pt"][:, :n4].reshape(parts["Pt"].shape[0], n4, 4, 16)
    sigma = formats.e4m3(448.0 * g.max(axis=-1))
    y = attention.FP4_P_SCALE * g / np.where(sigma > 0, sigma, 1.0)[..., None]
    t = formats.E2M1_VALUES
    mids, widths = (t[1:] + t[:-1]) / 2, t[1:] - t[:-1]
    dist = np.abs(y[..., None] - mids) / np.maximum(y[..., None], 1e-300)
    dist = np.where((sigma[..., None, None] > 0) & (y[..., None] > 0), dist, np.inf)
    i = np.unravel_index(np.argmin(dist), dist.shape)
    q, b, grp, e, m = i
    return q, b, 16 * grp + e, float(dist[i]), float(widths[m]), float(sigma[q, b, grp]), parts


@pytest.mark.parametrize("a", [3, 9])
def test_flip_bound_covers_a_planted_flip_and_nothing_else(monkeypatch, a):
    ops, cls = _setup(W)
    lists = rank.key_lists_all(cls[a])
    assert len(lists[0]) > 0
    q, b, v, dist, width, sigma, parts = _closest_nvfp4_weight(ops, a, lists)
    O = parts["U"] / parts["ell"][:, None]
    # the output with that one weight rounded to the other neighbour
    Vh = ops.phases[4][2][lists[0][b], v]
    dw = width * sigma / attention.FP4_P_SCALE
    O_flip = O.copy()
    O_flip[q] += dw * parts["f"][q, b] * Vh / parts["ell"][q]
    # no weight counts as near a midpoint: the bound is zero
    monkeypatch.setattr(oracle_pool, "FLIP_EPS", 0.0)
    _, B0, n0 = oracle_pool.flip_bound(ops, a, lists)
    assert n0 == 0 and np.all(B0 == 0)
    # a window just wide enough for the closest weight: the planted flip is covered
    monkeypatch.setattr(oracle_pool, "FLIP_EPS", dist * 1.0001)
    _, B1, n1 = oracle_pool.flip_bound(ops, a, lists)
    assert n1 >= 1
    assert np.all(np.abs(O_flip - O) <= B1 + 1e-12)
    assert np.abs(O_flip - O).max() > 0
    # a defect is not covered: the row's first 4-bit key block left out
    monkeypatch.setattr(oracle_pool, "FLIP_EPS", 1e-4)
    O_ref, B, _ = oracle_pool.flip_bound(ops, a, lists)
    O_bad = attention.attend(ops, a, lists[0][1:], lists[1], lists[2])
    assert (np.abs(O_bad - O_ref) - TOL_MAX_ABS - B).max() > 0
