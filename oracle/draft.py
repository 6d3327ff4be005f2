"""Pooled descriptors and the draft map (oracle; test infrastructure).

Paper: descriptor equation (region mean and channel-wise maximum of Q and
K over the valid tokens of a region), Definition 3.1 / draft equation

    A = (1 - lambda) softmax_row(Qbar Kbar^T / sqrt d)
        + lambda softmax_row(Qmax Kmax^T / sqrt d),

with both branches normalized over key regions (routing appendix). All of
it is computed in float64; the softmax subtracts the row maximum first,
which leaves its value unchanged. The result is rounded once to float32,
the type the ranking consumes.
"""
import numpy as np

from .partition import CAP


def pool(X, slot2tok, n_a):
    """Region mean and channel-wise max of X [N, d] (float64 of the inputs).

    Returns (mean [R, d], max [R, d]) in float64; padding never enters."""
    R = n_a.size
    d = X.shape[1]
    mean = np.empty((R, d))
    mx = np.empty((R, d))
    for a in range(R):
        toks = slot2tok[a * CAP: a * CAP + n_a[a]]
        rows = X[toks].astype(np.float64)
        mean[a] = rows.sum(axis=0) / n_a[a]
        mx[a] = rows.max(axis=0)
    return mean, mx


def softmax_rows(S):
    """Row softmax in float64 with the row maximum subtracted."""
    S = np.asarray(S, dtype=np.float64)
    e = np.exp(S - S.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def draft_map(Qbar, Kbar, Qmax, Kmax, lam):
    """Draft map A (float64, [R, R]) of one head."""
    d = Qbar.shape[1]
    s1 = Qbar @ Kbar.T / np.sqrt(d)
    s2 = Qmax @ Kmax.T / np.sqrt(d)
    return (1.0 - lam) * softmax_rows(s1) + lam * softmax_rows(s2)


def draft_head(Q, K, slot2tok, n_a, lam):
    """Pool one head's Q, K [N, d] and return (A32 [R, R] float32, pooled dict)."""
    Qbar, Qmax = pool(Q, slot2tok, n_a)
    Kbar, Kmax = pool(K, slot2tok, n_a)
    A = draft_map(Qbar, Kbar, Qmax, Kmax, lam)
    return A.astype(np.float32), dict(Qbar=Qbar, Qmax=Qmax, Kbar=Kbar, Kmax=Kmax, A64=A)
