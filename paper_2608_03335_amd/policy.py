"""Policy function (paper §3.1; §4 configurations and policy study).

Per denoising step it decides between full attention (the warm-up steps) and a
head-wise sparsity-ratio scheme. A scheme splits the per-row block budget into a
static local window and a dynamic Top-K part (Func 0: dynamic:static = 30:1;
Func 1: about 80% dynamic), and spreads the dynamic part over the heads in
inverse proportion to their Selected Aggregation Score. The per-head budgets are
computed on the device (spade_policy_budgets), so no host sync is needed; the
rest is host arithmetic on step counts and budgets.

Readings (the paper gives the budgets' effect, not their formulas):
  * warm-up: the first ceil(0.30 n) of n steps (text-to-video) or ceil(0.25 n)
    (image-to-video) run full attention; Turbo only the first step;
  * the static share rounds half up to whole blocks and buys the largest window
    of WINDOW_LADDER that fits; the dynamic Top-K keeps the remainder.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

from . import spade as S
from .pipeline import Scheme

# block radii (t, y, x) of the static windows, by size 1, 3, 9, 27, 45, 75, 125
WINDOW_LADDER = ((0, 0, 0), (0, 0, 1), (0, 1, 1), (1, 1, 1), (1, 1, 2), (1, 2, 2), (2, 2, 2))
STATIC_SHARE = {0: 1.0 / 31.0, 1: 0.2}


def window_blocks(w) -> int:
    return (2 * w[0] + 1) * (2 * w[1] + 1) * (2 * w[2] + 1)


@dataclass
class Policy:
    func: int                 # 0: Func 0 (Wan 2.1/2.2), 1: Func 1 (Hunyuan-Video)
    n_steps: int = 50
    task: str = "t2v"         # "t2v" | "i2v"
    turbo: bool = False

    def dense(self, step: int) -> bool:
        """Full attention at denoising step `step` (0-based)?"""
        if self.turbo:
            return step < 1
        frac = 0.30 if self.task == "t2v" else 0.25
        return step < math.ceil(frac * self.n_steps - 1e-9)

    def split(self, k_total: int):
        """(window radii or None, window blocks, dynamic k) for k_total blocks per row."""
        k_static = int(math.floor(k_total * STATIC_SHARE[self.func] + 0.5))
        fits = [w for w in WINDOW_LADDER if window_blocks(w) <= k_static]
        if not fits:
            return None, 0, k_total
        return fits[-1], window_blocks(fits[-1]), k_total - window_blocks(fits[-1])

    def head_budgets(self, as_best, k_dyn: int, NB: int, out, heads=None, stream=None):
        """Per-head dynamic k (device int32, list order) from the Selected AS."""
        S.spade_policy_budgets(as_best, k_dyn, NB, out, heads=heads, stream=stream)
        return out

    def scheme(self, k_total: int, NB: int, as_best, out, heads=None, estimator="mean",
               stream=None) -> Scheme:
        """The Top-K scheme of one head group: window + AS-guided per-head k."""
        w, _, k_dyn = self.split(k_total)
        self.head_budgets(as_best, max(k_dyn, 1), NB, out, heads, stream)
        return Scheme(estimator, "topk", topk=max(k_dyn, 1), topk_per_head=out,
                      window=w if w is not None else (-1, -1, -1))
