"""The four stages end to end for one workload (oracle; test infrastructure).

Stage order follows the paper's pipeline figure and hardware section:
region layout -> pooled draft map -> shared ranking -> operand encoding ->
phased attention -> inverse index map back to token order.
"""
import numpy as np

from . import attention, draft, encode, partition, rank


def run_head(Q, K, V, layout, lam, budgets, scope, rows=None, mode="quant", num16=0, fmt4="nvfp4"):
    """One (batch, head). Q, K, V: [N, d] float32 values; budgets
    (num8, num4, den) plus num16/den for the 16-bit path; fmt4 selects the
    4-bit encoding ("nvfp4" or "mxfp4").

    ``rows`` restricts the attention to a subset of query regions (the draft,
    ranking and encodings always cover the whole head). Returns a dict with
    A32, cls, enc, and O [N, d] float64 (rows not computed are NaN)."""
    slot2tok, n_a, _ = layout
    A32, pooled = draft.draft_head(Q, K, slot2tok, n_a, lam)
    cls = rank.rank_head(A32, *budgets, scope, num16=num16)
    enc = encode.encode_head(Q, K, V, slot2tok, n_a)
    enc_mx = encode.encode_head_mx(Q, K, V, slot2tok, n_a) if fmt4 == "mxfp4" else None
    if mode == "quant":
        rec_mx = None if enc_mx is None else encode.reconstruct_mx(enc_mx)
        ops = attention.Operands.quantized(encode.reconstruct(enc), n_a, rec_mx)
    else:
        ops = attention.Operands.exact(*(partition.gather_slots(X, slot2tok) for X in (Q, K, V)), n_a)
    R = n_a.size
    O = np.full(Q.shape, np.nan)
    for a in (range(R) if rows is None else rows):
        l4, l8, l16 = rank.key_lists_all(cls[a])
        toks = slot2tok[a * partition.CAP: a * partition.CAP + n_a[a]]
        O[toks] = attention.attend(ops, a, l4, l8, l16)
    return dict(A32=A32, pooled=pooled, cls=cls, enc=enc, enc_mx=enc_mx, O=O)


def run(w, Q, K, V, heads=None, rows=None, mode="quant"):
    """Whole workload ``w`` (synth.configs.Workload). Q, K, V: [B, H, N, d]."""
    layout = partition.make_partition(w.partition, w.T, w.Hg, w.Wg)
    out = []
    for b in range(Q.shape[0]):
        for h in (range(Q.shape[1]) if heads is None else heads):
            out.append(run_head(Q[b, h], K[b, h], V[b, h], layout, w.lam, w.budgets,
                                w.scope, rows=rows, mode=mode, num16=w.num16, fmt4=w.fmt4))
    return layout, out
