"""Policy function (paper §3.1; §4 configurations and policy study): orchestration.

Per denoising step it decides between full attention (the warm-up steps) and a
head-wise sparsity-ratio scheme. A Top-K scheme splits the per-row block budget
into a static local window and a dynamic Top-K part (Func 0: dynamic:static =
30:1; Func 1: about 80% dynamic) and spreads the dynamic part over the heads in
inverse proportion to their Selected Aggregation Score; a Top-P scheme spreads
the dropped mass 1 - tau over the heads in proportion to the score. Every rule
is a library call: the warm-up schedule and the split run on the host
(spade_policy_dense, spade_policy_split), the per-head budgets on the device
(spade_policy_budgets, spade_policy_tau), so no host sync is needed. This module
only chooses which call to make.
"""
from __future__ import annotations

from dataclasses import dataclass

from . import spade as S
from .pipeline import Scheme


@dataclass
class Policy:
    func: int                 # 0: Func 0 (Wan 2.1/2.2), 1: Func 1 (Hunyuan-Video)
    n_steps: int = 50
    task: str = "t2v"         # "t2v" | "i2v"
    turbo: bool = False

    def dense(self, step: int) -> bool:
        """Full attention at denoising step `step` (0-based)?"""
        task = S.SPADE_TASK_T2V if self.task == "t2v" else S.SPADE_TASK_I2V
        return S.spade_policy_dense(step, self.n_steps, task, self.turbo)

    def split(self, k_total: int):
        """(window radii or None, window blocks, dynamic k) for k_total blocks per row."""
        return S.spade_policy_split(k_total, self.func)

    def head_budgets(self, as_best, k_dyn: int, NB: int, out, heads=None, stream=None):
        """Per-head dynamic k (device int32, list order) from the Selected AS."""
        S.spade_policy_budgets(as_best, k_dyn, NB, out, heads=heads, stream=stream)
        return out

    def head_tau(self, as_best, tau: float, out, heads=None, stream=None):
        """Per-head Top-P mass (device fp64, list order) from the Selected AS."""
        S.spade_policy_tau(as_best, tau, out, heads=heads, stream=stream)
        return out

    def scheme(self, k_total: int, NB: int, as_best, out, heads=None, estimator="mean",
               stream=None) -> Scheme:
        """The Top-K scheme of one head group: window + AS-guided per-head k."""
        w, _, k_dyn = self.split(k_total)
        self.head_budgets(as_best, max(k_dyn, 1), NB, out, heads, stream)
        return Scheme(estimator, "topk", topk=max(k_dyn, 1), topk_per_head=out,
                      window=w if w is not None else (-1, -1, -1))

    def scheme_topp(self, tau: float, k_nominal: int, as_best, out, heads=None,
                    estimator="mean", stream=None) -> Scheme:
        """The Top-P scheme of one head group: the window that the split gives a
        nominal per-row budget of k_nominal blocks, plus AS-guided per-head mass."""
        w, _, _ = self.split(k_nominal)
        self.head_tau(as_best, tau, out, heads, stream)
        return Scheme(estimator, "topp", tau=tau, tau_per_head=out,
                      window=w if w is not None else (-1, -1, -1))
