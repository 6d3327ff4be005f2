"""Workload registry for the DraftAttention2 hot path.

Plain data only: shapes, budgets and generator switches. Nothing here
computes any step of the method.

Each workload is a synthetic stand-in for one video-DiT attention layer
(the paper measures on captured HunyuanVideo / MiniMax-H3 activations,
which are not available). Budgets are integer fractions
``(num8, num4, den)``: ``num8/den`` of the region pairs go to the 8-bit
path, ``num4/den`` to the 4-bit path and the rest are skipped; ``num16/den``
(default 0, as on the hot path) go to the 16-bit path ahead of both (Alg. 1).
"""
from dataclasses import dataclass, field, replace
from typing import Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    d: int
    T: int
    Hg: int
    Wg: int
    dtype: str                      # "fp32" or "bf16" (storage type of Q, K, V)
    budgets: Tuple[int, int, int]   # (num8, num4, den)
    scope: str                      # "row" or "head" ranking scope
    head_scale: bool                # per-head random scale in [0.5, 2]
    key_outliers: float = 0.0       # fraction of key positions scaled by 8
    phase_drift: bool = False       # sinusoid phases drift across frames
    lam: float = 0.2                # pooling weight lambda of the draft map
    seed: int = 0
    num16: int = 0                  # num16/den of the pairs go to the 16-bit path
    partition: str = "tiles8"       # "tiles8" (8x8 tiles) or "ragged" (minimum-perimeter regions)
    fmt4: str = "nvfp4"             # 4-bit encoding: "nvfp4" (the paper's) or "mxfp4"

    @property
    def N(self) -> int:
        return self.T * self.Hg * self.Wg

    def with_budgets(self, num8, num4, den):
        return replace(self, budgets=(num8, num4, den),
                       name=f"{self.name}-{num8}/{num4}/{den}")


# Tiny smoke case: 2 frames of 16x16 tokens, 8 tiles of 64, fp32.
TINY = Workload("tiny-2x16x16-h2-d64", B=1, H=2, d=64, T=2, Hg=16, Wg=16,
                dtype="fp32", budgets=(25, 25, 100), scope="row",
                head_scale=False, seed=1)

# Mid video-DiT layer: 21x30x52 = 32,760 tokens, 12 heads, d=128, bf16.
MID = Workload("mid-21x30x52-h12-d128", B=1, H=12, d=128, T=21, Hg=30, Wg=52,
               dtype="bf16", budgets=(10, 30, 100), scope="head",
               head_scale=True, seed=2)

# Budget sweep on the mid shape.
SWEEP = tuple(replace(MID, name=f"sweep-{a}/{b}/{c}", budgets=(a, b, c), seed=3)
              for (a, b, c) in ((100, 0, 100), (20, 20, 100), (5, 45, 100), (0, 40, 100)))

# Wide layer: 21x45x80 = 75,600 tokens, 40 heads, 1% key outliers x8.
WIDE = Workload("wide-21x45x80-h40-d128", B=1, H=40, d=128, T=21, Hg=45, Wg=80,
                dtype="bf16", budgets=(10, 30, 100), scope="head",
                head_scale=True, key_outliers=0.01, seed=4)

# Long / high-resolution layer: 33x45x80 = 118,800 tokens, 24 heads, drifting phases.
LONG = Workload("long-33x45x80-h24-d128", B=1, H=24, d=128, T=33, Hg=45, Wg=80,
                dtype="bf16", budgets=(5, 25, 100), scope="head",
                head_scale=True, phase_drift=True, seed=5)

# Operator error-vs-latency sweep shape (the paper's attention error analysis
# uses a 109,376-token, 56-head, d=128 capture, which is not a product of a
# latent grid; 31x42x84 = 109,368 tokens stands in for it), on the ragged
# partition; budgets are set per sweep point.
FIG4 = Workload("fig4-31x42x84-h56-d128", B=1, H=56, d=128, T=31, Hg=42, Wg=84,
                dtype="bf16", budgets=(100, 0, 100), scope="head",
                head_scale=True, seed=6, partition="ragged")

ALL = (TINY, MID) + SWEEP + (WIDE, LONG, FIG4)
BY_NAME = {w.name: w for w in ALL}
