"""Integer quotas and the shared ranking (oracle; test infrastructure).

Paper: Algorithm 1 (stable descending argsort of vec(A); the first T8 pairs
go to INT8, the next T4 to NVFP4, the rest are skipped; no 16-bit quota on
this path), the routing appendix (ranking across all R^2 region pairs of a
head, ties resolved by region-pair index; precision fractions give integer
quotas).

Readings:
* Quotas: the paper does not say how fractions become integers. Budgets
  are exact rationals num8/den, num4/den; the cumulative counts are rounded
  half up: C8 = floor(num8*M/den + 1/2), C84 = floor((num8+num4)*M/den + 1/2),
  T8 = C8, T4 = C84 - C8, with M = R^2 (head scope) or M = R (row scope).
* Scope: "head" ranks all R^2 pairs of a head (the paper's Algorithm 1);
  "row" ranks the R pairs of each query region separately (per-row
  budgets).
* Ties: lower index first, index = a*R + b (head scope) or b (row scope),
  which is what a stable descending sort of row-major vec(A) gives.
"""
import numpy as np


def quotas(num8, num4, den, M):
    """Integer (T8, T4) for M candidates under budgets num8/den, num4/den."""
    c8 = (2 * num8 * M + den) // (2 * den)
    c84 = (2 * (num8 + num4) * M + den) // (2 * den)
    return c8, c84 - c8


def _assign(scores, T8, T4):
    """Classes {8, 4, 0} for a 1-D score vector ranked (score desc, index asc)."""
    s = np.asarray(scores, dtype=np.float64)
    order = np.lexsort((np.arange(s.size), -s))
    cls = np.zeros(s.size, dtype=np.uint8)
    cls[order[:T8]] = 8
    cls[order[T8:T8 + T4]] = 4
    return cls


def rank_head(A32, num8, num4, den, scope):
    """Precision map cls [R, R] in {0, 4, 8} for one head."""
    R = A32.shape[0]
    if scope == "head":
        T8, T4 = quotas(num8, num4, den, R * R)
        return _assign(A32.reshape(-1), T8, T4).reshape(R, R)
    if scope == "row":
        T8, T4 = quotas(num8, num4, den, R)
        return np.stack([_assign(A32[a], T8, T4) for a in range(R)])
    raise ValueError(scope)


def key_lists(cls_row):
    """(list4, list8): key regions of one query region per path, ascending."""
    return np.nonzero(cls_row == 4)[0], np.nonzero(cls_row == 8)[0]
