"""Oracle work of the full-size GPU parity tests, one (batch, head) per task in
a pool of fresh CPU processes (test infrastructure).

Workers are started with the "spawn" method, so they share nothing with the
parent that holds the GPU: each one regenerates its head's inputs from the
seeded generator (the draws of a head do not depend on the other heads) and
runs the oracle on one BLAS thread. Nothing here touches the library or the
GPU."""
import os
from dataclasses import asdict
from multiprocessing import get_context

import numpy as np


def _init():
    try:
        from threadpoolctl import threadpool_limits
        threadpool_limits(1)
    except ImportError:
        pass


def _workload(wd):
    from synth import configs
    return configs.Workload(**wd)


def _head_inputs(w, h):
    from synth import gen
    Q, K, V = gen.generate(w, heads=[h])
    return Q[0, 0], K[0, 0], V[0, 0]


def _masks(task):
    """Draft map and class map of one head (b = 0)."""
    from oracle import draft, partition, rank
    wd, h = task
    w = _workload(wd)
    q, k, _ = _head_inputs(w, h)
    slot2tok, n_a, _ = partition.make_partition(w.partition, w.T, w.Hg, w.Wg)
    A32, _ = draft.draft_head(q, k, slot2tok, n_a, w.lam)
    return h, A32, rank.rank_head(A32, *w.budgets, w.scope, num16=w.num16)


def _outputs(task):
    """Draft map, class map and the output rows of one head: every query
    block of ``rows`` (None: all), each with the oracle's own class row, or
    with the class row given for it in ``given`` (block -> class row)."""
    from oracle import attention, draft, encode, partition, rank
    wd, h, rows, given = task
    w = _workload(wd)
    q, k, v = _head_inputs(w, h)
    layout = partition.make_partition(w.partition, w.T, w.Hg, w.Wg)
    slot2tok, n_a, _ = layout
    A32, _ = draft.draft_head(q, k, slot2tok, n_a, w.lam)
    cls = rank.rank_head(A32, *w.budgets, w.scope, num16=w.num16)
    enc = encode.encode_head(q, k, v, slot2tok, n_a)
    rec_mx = encode.reconstruct_mx(encode.encode_head_mx(q, k, v, slot2tok, n_a)) if w.fmt4 == "mxfp4" else None
    ops = attention.Operands.quantized(encode.reconstruct(enc), n_a, rec_mx)
    O = np.full(q.shape, np.nan)
    for a in (range(n_a.size) if rows is None else rows):
        row = given.get(a, cls[a]) if given else cls[a]
        toks = slot2tok[a * partition.CAP:a * partition.CAP + n_a[a]]
        O[toks] = attention.attend(ops, a, *rank.key_lists_all(row))
    return h, A32, cls, O


def _pool_map(fn, tasks, timeout=900):
    """fn over tasks in spawned workers; raises (instead of waiting forever)
    if a worker dies or the work takes longer than ``timeout`` seconds."""
    workers = max(1, min(len(tasks), 16, os.cpu_count() or 1))
    with get_context("spawn").Pool(workers, initializer=_init) as pool:
        return pool.map_async(fn, tasks, chunksize=1).get(timeout)


def masks(w, heads):
    """{head: (A32, cls)} for batch 0 of workload ``w``."""
    return {h: (A, c) for h, A, c in _pool_map(_masks, [(asdict(w), h) for h in heads])}


def outputs(w, heads, rows=None, given=None):
    """{head: (A32, cls, O)}; ``given`` maps head -> {block: class row}."""
    tasks = [(asdict(w), h, rows, (given or {}).get(h)) for h in heads]
    return {h: (A, c, O) for h, A, c, O in _pool_map(_outputs, tasks)}


# Relative error bound of the kernel's float32 unquantized weights against the
# exact ones: at most 8 float32 accumulation steps of exact products on logits
# of at most ~40 in log2 units (~3e-5), plus the exp2 / log2 roundings, with
# a factor of 3 to spare. A quantizer input this close to a rounding midpoint
# may legitimately round either way in the kernel.
FLIP_EPS = 1e-4


def _midpoint_steps(x, table):
    """For each |x|: whether it lies within FLIP_EPS (relative) of a rounding
    midpoint of the magnitude table, and the width of that step."""
    t = np.unique(np.abs(table[np.isfinite(table)]))
    mids = (t[1:] + t[:-1]) / 2
    widths = t[1:] - t[:-1]
    ax = np.abs(np.asarray(x, np.float64))
    i = np.clip(np.searchsorted(mids, ax), 1, mids.size - 1)
    near_lo = np.abs(ax - mids[i - 1]) <= FLIP_EPS * ax
    near_hi = np.abs(ax - mids[i]) <= FLIP_EPS * ax
    width = np.where(near_lo, widths[i - 1], np.where(near_hi, widths[i], 0.0))
    return near_lo | near_hi, width


def flip_bound(ops, a, lists):
    """Oracle output of block a and, per (query, channel), a bound on how far
    the output can move when the weights whose quantizer inputs lie within
    FLIP_EPS of a rounding midpoint round the other way: NVFP4 weight codes
    (E2M1 of 2688 Pt / sigma_P), the group scales sigma_P (E4M3 of 448 max Pt;
    all 16 weights of the group recomputed with the neighbouring scale) and
    the INT8 path's weights (E4M3 of Pt / eta)."""
    from oracle import attention, formats
    O, parts = attention.attend(ops, a, *lists, return_parts=True)
    Pt, f, ell = parts["Pt"], parts["f"], parts["ell"]              # [nq, nb, 64], [nq, nb], [nq]
    n4, n8 = len(lists[0]), len(lists[1])
    blocks = list(lists[0]) + list(lists[1]) + list(lists[2])
    Vh = np.concatenate([ops.phases[p][2][np.asarray(lst, np.int64)]
                         for lst, p in zip(lists, (4, 8, 16)) if len(lst)])  # [nb, 64, d]
    dW = np.zeros_like(Pt)
    mx = ops.phases[4][3] is attention.quant_weights_mx
    if n4 and not mx:
        g = Pt[:, :n4].reshape(Pt.shape[0], n4, 4, 16)
        x = 448.0 * g.max(axis=-1)
        sigma = formats.e4m3(x)
        safe = np.where(sigma > 0, sigma, 1.0)
        y = attention.FP4_P_SCALE * g / safe[..., None]
        near, width = _midpoint_steps(y, formats.E2M1_VALUES)
        d4 = np.where(near & (sigma[..., None] > 0), width * sigma[..., None] / attention.FP4_P_SCALE, 0.0)
        # the group scale on the other side of its own midpoint
        e4 = formats.e4m3_decode(np.arange(256))
        snear, _ = _midpoint_steps(x, e4)
        t = np.unique(np.abs(e4[np.isfinite(e4)]))
        lo = t[np.clip(np.searchsorted(t, sigma, side="left") - 1, 0, t.size - 1)]
        hi = t[np.clip(np.searchsorted(t, sigma, side="right"), 0, t.size - 1)]
        alt = np.where(x >= sigma, hi, lo)
        w_now = np.where(sigma[..., None] > 0, sigma[..., None] / attention.FP4_P_SCALE *
                         formats.e2m1(attention.FP4_P_SCALE * g / safe[..., None]), 0.0)
        alt_safe = np.where(alt > 0, alt, 1.0)
        w_alt = np.where(alt[..., None] > 0, alt[..., None] / attention.FP4_P_SCALE *
                         formats.e2m1(attention.FP4_P_SCALE * g / alt_safe[..., None]), 0.0)
        d4 = np.maximum(d4, np.where(snear[..., None], np.abs(w_alt - w_now), 0.0))
        dW[:, :n4] = d4.reshape(Pt.shape[0], n4, 64)
    if n4 and mx:
        g = Pt[:, :n4].reshape(Pt.shape[0], n4, 2, 32)
        amax = g.max(axis=-1)
        _, e = np.frexp(np.where(amax > 0, amax, 1.0))
        k = np.where(amax > 0, np.clip((e - 1) - 2, -127, 127), -127)
        X = np.ldexp(1.0, k)[..., None]
        near, width = _midpoint_steps(g / X, formats.E2M1_VALUES)
        dm = np.where(near, width * X, 0.0)
        # the block exponent one step the other way when the maximum sits at a power of two
        frac = amax / np.ldexp(1.0, k + 2)                               # in [1, 2)
        knear = (np.abs(frac - 1.0) <= FLIP_EPS) | (np.abs(frac - 2.0) <= 2 * FLIP_EPS)
        k_alt = np.where(frac < 1.5, k - 1, k + 1)
        X_alt = np.ldexp(1.0, k_alt)[..., None]
        w_now = X * formats.e2m1(g / X)
        w_alt = X_alt * formats.e2m1(g / X_alt)
        dm = np.maximum(dm, np.where(knear[..., None], np.abs(w_alt - w_now), 0.0))
        dW[:, :n4] = dm.reshape(Pt.shape[0], n4, 64)
    if n8:
        x = attention.AMP * Pt[:, n4:n4 + n8]
        near, width = _midpoint_steps(x, formats.e4m3_decode(np.arange(256)))
        dW[:, n4:n4 + n8] = np.where(near, width * attention.ETA, 0.0)
    B = np.einsum("qbk,kbd->qd", dW * f[:, :, None], np.abs(Vh).transpose(1, 0, 2)) / ell[:, None]
    return O, B, int((dW > 0).sum())


def _flip_task(task):
    """Rows of block list ``blocks`` of one head: the largest excess of the
    GPU rows' deviation over TOL + flip bound, the largest deviation, and the
    number of near-midpoint weights."""
    from oracle import attention, encode, partition, rank
    wd, h, items, tol = task
    w = _workload(wd)
    q, k, v = _head_inputs(w, h)
    slot2tok, n_a, _ = partition.make_partition(w.partition, w.T, w.Hg, w.Wg)
    enc = encode.encode_head(q, k, v, slot2tok, n_a)
    rec_mx = encode.reconstruct_mx(encode.encode_head_mx(q, k, v, slot2tok, n_a)) if w.fmt4 == "mxfp4" else None
    ops = attention.Operands.quantized(encode.reconstruct(enc), n_a, rec_mx)
    out = []
    for a, cls_row, O_gpu in items:
        O, B, nflip = flip_bound(ops, a, rank.key_lists_all(cls_row))
        dev = np.abs(O_gpu.astype(np.float64) - O)
        out.append((a, float((dev - tol - B).max()), float(dev.max()), nflip, float(B.max())))
    return h, out


def flip_check(w, items_by_head, tol):
    """{head: [(block, max excess over tol + bound, max deviation, near-midpoint
    weights, max bound)]} for the GPU rows items_by_head[h] = [(block, class
    row, GPU output rows [n_a, d])]."""
    tasks = [(asdict(w), h, items, tol) for h, items in items_by_head.items()]
    return dict(_pool_map(_flip_task, tasks))
