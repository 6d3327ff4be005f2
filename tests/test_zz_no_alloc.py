"""The allocation-free ranking entry point against the workspace one, through
the C ABI: identical classes, counts, key lists and work-order permutation,
on two calls in a row (the second on a smaller problem, so the shared fixed
scratch holds the first call's contents when the second starts), in head and
row scope; and the size limit is reported as DA2_ERR_WORKSPACE."""
import numpy as np
import pytest
import torch

from gpu_harness import SMALL, lists_of, log, problem_of
from paper_2609_32628_amd import _lib, api
from synth import configs

pytestmark = pytest.mark.gpu


def _scores(BH, R, seed):
    rng = np.random.default_rng(seed)
    A = rng.random((BH, R, R)).astype(np.float32)
    A[rng.random((BH, R, R)) < 0.3] = np.float32(0.25)     # many ties
    return A


def _rank_both(w, scope, budgets16, seed):
    p = problem_of(w)
    R = api.da2_sizes(p, scope)["R"]
    BH = w.B * w.H
    A = torch.from_numpy(_scores(BH, R, seed)).cuda().reshape(w.B, w.H, R, R)
    outs = []
    for noalloc in (False, True):
        buf = api.alloc(p, scope)
        buf.cls.fill_(0xEE)
        buf.lists.fill_(0xA5)
        if noalloc:
            api.da2_rank_assign_noalloc(A, p, *budgets16, scope, buf.cls, buf.lists)
        else:
            api.da2_rank_assign(A, p, *budgets16, scope, buf.cls, buf.lists, buf.ws_rank)
        torch.cuda.synchronize()
        keys, counts, order = lists_of(buf, p)
        n = counts[:, :3].sum(axis=1)
        outs.append((buf.cls.cpu().numpy(), counts.copy(), np.sort(order),
                     [keys[r, :n[r]].copy() for r in range(n.size)]))
    (c0, n0, o0, k0), (c1, n1, o1, k1) = outs
    assert np.array_equal(c0, c1)
    assert np.array_equal(n0, n1)
    assert np.array_equal(o0, o1) and np.array_equal(o0, np.arange(BH * R))
    assert all(np.array_equal(a, b) for a, b in zip(k0, k1))
    return int((c1 == 8).sum()), int((c1 == 4).sum())


@pytest.mark.parametrize("scope", ["head", "row"])
def test_noalloc_rank_matches_workspace_rank(scope):
    big = configs.MID if scope == "head" else SMALL
    small = SMALL if scope == "head" else configs.TINY
    for w, budgets, seed in ((big, (0, 10, 30, 100), 1), (small, (5, 20, 30, 100), 2)):
        log(f"noalloc rank {scope} {w.name} {budgets}")
        n8, n4 = _rank_both(w, scope, budgets, seed)
        log(f"  identical: {n8} 8-bit, {n4} 4-bit pairs")


def test_noalloc_rank_rejects_problems_beyond_its_scratch():
    # head scope on the mid layer's grid with 128 heads: the per-head
    # histograms and candidate lists need more than the fixed scratch (the
    # size is checked on the host before any launch)
    p = api.problem(1, 128, 128, 21, 30, 52)
    assert api.da2_sizes(p, "head")["ws_rank_bytes"] > _lib.DA2_RANK_NOALLOC_MAX_BYTES
    A = torch.empty(1, dtype=torch.float32, device="cuda")
    with pytest.raises(_lib.Da2Error) as e:
        api.da2_rank_assign_noalloc(A, p, 0, 10, 30, 100, "head", A, A)
    assert e.value.status == _lib.DA2_ERR_WORKSPACE
