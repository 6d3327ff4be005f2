"""Integer quotas and the shared ranking (oracle; test infrastructure).

Paper: Algorithm 1 (stable descending argsort of vec(A); the first T16
pairs go to the 16-bit path, the next T8 to INT8, the next T4 to NVFP4, the
rest are skipped), the routing appendix (ranking across all R^2 region
pairs of a head, ties resolved by region-pair index; precision fractions
give integer quotas). The hot path runs with T16 = 0.

Readings:
* Quotas: the paper does not say how fractions become integers. Budgets
  are exact rationals num16/den, num8/den, num4/den; the cumulative counts
  are rounded half up: C16 = floor(num16*M/den + 1/2),
  C168 = floor((num16+num8)*M/den + 1/2),
  C1684 = floor((num16+num8+num4)*M/den + 1/2), T16 = C16,
  T8 = C168 - C16, T4 = C1684 - C168, with M = R^2 (head scope) or M = R
  (row scope). With num16 = 0 this is C8 = floor(num8*M/den + 1/2),
  C84 = floor((num8+num4)*M/den + 1/2), T8 = C8, T4 = C84 - C8.
* Scope: "head" ranks all R^2 pairs of a head (the paper's Algorithm 1);
  "row" ranks the R pairs of each query region separately (per-row
  budgets).
* Ties: lower index first, index = a*R + b (head scope) or b (row scope),
  which is what a stable descending sort of row-major vec(A) gives.
"""
import numpy as np


def _half_up(num, M, den):
    return (2 * num * M + den) // (2 * den)


def quotas3(num16, num8, num4, den, M):
    """Integer (T16, T8, T4) for M candidates under budgets num16/den,
    num8/den, num4/den (cumulative counts rounded half up)."""
    c16 = _half_up(num16, M, den)
    c168 = _half_up(num16 + num8, M, den)
    c1684 = _half_up(num16 + num8 + num4, M, den)
    return c16, c168 - c16, c1684 - c168


def quotas(num8, num4, den, M):
    """Integer (T8, T4) for M candidates under budgets num8/den, num4/den."""
    return quotas3(0, num8, num4, den, M)[1:]


def _assign(scores, T8, T4, T16=0):
    """Classes {16, 8, 4, 0} for a 1-D score vector ranked (score desc, index asc)."""
    s = np.asarray(scores, dtype=np.float64)
    order = np.lexsort((np.arange(s.size), -s))
    cls = np.zeros(s.size, dtype=np.uint8)
    cls[order[:T16]] = 16
    cls[order[T16:T16 + T8]] = 8
    cls[order[T16 + T8:T16 + T8 + T4]] = 4
    return cls


def rank_head(A32, num8, num4, den, scope, num16=0):
    """Precision map cls [R, R] in {0, 4, 8, 16} for one head."""
    R = A32.shape[0]
    if scope == "head":
        T16, T8, T4 = quotas3(num16, num8, num4, den, R * R)
        return _assign(A32.reshape(-1), T8, T4, T16).reshape(R, R)
    if scope == "row":
        T16, T8, T4 = quotas3(num16, num8, num4, den, R)
        return np.stack([_assign(A32[a], T8, T4, T16) for a in range(R)])
    raise ValueError(scope)


def key_lists(cls_row):
    """(list4, list8): key regions of one query region per path, ascending."""
    return np.nonzero(cls_row == 4)[0], np.nonzero(cls_row == 8)[0]


def key_lists_all(cls_row):
    """(list4, list8, list16): the three phase segments, each ascending."""
    return np.nonzero(cls_row == 4)[0], np.nonzero(cls_row == 8)[0], np.nonzero(cls_row == 16)[0]
