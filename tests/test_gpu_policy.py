"""GPU parity of the policy function: spade_policy_budgets bit for bit against
the oracle, and the block-shape sweep driven by the policy (static window + per-
head budgets from the Selected Aggregation Score) against the oracle's composed
selection and attention."""
import sys

import numpy as np
import pytest
import torch

from oracle import spade_oracle as O
from paper_2608_03335_amd import spade as S
from paper_2608_03335_amd.pipeline import SweepPath
from paper_2608_03335_amd.policy import Policy

from . import _parity as P

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _budgets(as_best, k_dyn, NB, heads=None):
    t = torch.from_numpy(np.asarray(as_best, dtype=np.float64)).to(DEV)
    n = len(as_best) if heads is None else len(heads)
    out = torch.full((max(n, 1),), -7, dtype=torch.int32, device=DEV)
    S.spade_policy_budgets(t, k_dyn, NB, out, heads=heads)
    torch.cuda.synchronize()
    return out[:n].cpu().numpy()


@pytest.mark.parametrize("H,k_dyn,NB", [(24, 45, 360), (40, 76, 630), (12, 27, 245), (1, 5, 8),
                                        (1000, 3, 50)])
def test_budgets_bit_exact(H, k_dyn, NB):
    _say("policy budgets", H, k_dyn, NB)
    rng = np.random.default_rng(H)
    a = rng.uniform(0.3, 2.0, H)
    assert np.array_equal(_budgets(a, k_dyn, NB), O.policy_head_budgets(a, k_dyn, NB))


def test_budgets_head_lists_and_degenerate_scores():
    _say("policy budgets: lists, degenerate")
    rng = np.random.default_rng(7)
    a = rng.uniform(0.3, 2.0, 24)
    for heads in ([5, 0, 17], [23], list(range(23, -1, -1)), [2, 9, 4, 11]):
        assert np.array_equal(_budgets(a, 40, 360, heads), O.policy_head_budgets(a[heads], 40, 360))
    z = np.array([0.0, -1.0, 2.0, 0.5])
    assert np.array_equal(_budgets(z, 10, 100), O.policy_head_budgets(z, 10, 100))
    assert np.array_equal(_budgets(np.zeros(3), 7, 5), O.policy_head_budgets(np.zeros(3), 7, 5))
    big = np.array([1.0, 1000.0])
    assert np.array_equal(_budgets(big, 300, 360), O.policy_head_budgets(big, 300, 360))


def _taus(as_best, tau, heads=None):
    t = torch.from_numpy(np.asarray(as_best, dtype=np.float64)).to(DEV)
    n = len(as_best) if heads is None else len(heads)
    out = torch.full((max(n, 1),), float("nan"), dtype=torch.float64, device=DEV)
    S.spade_policy_tau(t, tau, out, heads=heads)
    torch.cuda.synchronize()
    return out[:n].cpu().numpy()


@pytest.mark.parametrize("H,tau", [(24, 0.9), (40, 0.95), (12, 0.8), (1, 0.5), (1000, 0.99)])
def test_tau_bit_exact(H, tau):
    _say("policy tau", H, tau)
    rng = np.random.default_rng(H + 7)
    a = rng.uniform(0.3, 2.0, H)
    assert np.array_equal(_taus(a, tau), O.policy_head_tau(a, tau))


def test_tau_head_lists_and_degenerate_scores():
    _say("policy tau: lists, degenerate")
    rng = np.random.default_rng(8)
    a = rng.uniform(0.3, 2.0, 24)
    for heads in ([5, 0, 17], [23], list(range(23, -1, -1)), [2, 9, 4, 11]):
        assert np.array_equal(_taus(a, 0.9, heads), O.policy_head_tau(a[heads], 0.9))
    for z, tau in (([0.0, -1.0, 2.0, 0.5], 0.9), ([0.0, 0.0, 0.0], 0.7), ([10.0, 0.001], 0.3),
                   ([1.0, 1.0], 1.0)):
        assert np.array_equal(_taus(z, tau), O.policy_head_tau(z, tau))


@pytest.mark.parametrize("func", [0, 1])
def test_policy_topp_sweep_matches_oracle(func):
    """Top-P groups under the policy: per-head mass from the Selected AS plus the
    window of the split, every group's selection against the oracle's composed
    selection (cut exemptions allowed), and the whole output (NaN-poisoned before
    the run) against the oracle's attention on the GPU's own lists."""
    grid, cands = (6, 16, 20), [(2, 4, 4), (3, 4, 5), (2, 8, 2)]
    cfg = P.small_cfg(*grid, 1, 1, 1, d=64, H=6)
    _say("policy top-p sweep, func", func)
    Q, K, V = P.bf16_inputs(cfg)
    pol, tau = Policy(func), 0.9
    p = SweepPath(1, 6, 64, *grid, cands, 0.7, device=DEV, policy=pol, tau=tau)
    P.nan_fill(p.O)
    p.evaluate(Q, K)
    work = p.work_list(torch.cuda.current_stream())
    best = p.best.cpu().numpy()
    Qn, Kn, Vn = P.to_np64(Q), P.to_np64(K), P.to_np64(V)
    scale = P.scale_of(64)
    ref_O = np.full(Qn.shape, np.nan)
    n_ex = 0
    for c, heads in work:
        v = p.group_select(c, heads, Q, K, V)
        p.group_attend(c, v)
        p.group_restore(c, heads, v)
        torch.cuda.synchronize()
        og = O.Geometry(*grid, *cands[c])
        w, _, _ = O.policy_split(p.topk[c], func)
        t_ref = O.policy_head_tau(best[heads], tau)
        t_gpu = p.gb[c]["tau_heads"][: len(heads)].cpu().numpy()
        assert np.array_equal(t_gpu, t_ref)
        spec = O.MaskSpec(mode="topp", tau_per_head=tuple(float(x) for x in t_ref), window=w)
        ref = O.composed_selection(Qn[:, heads], Kn[:, heads], og, spec, scale)
        c_g, i_g = v["counts"].cpu().numpy(), v["indices"].cpu().numpy()
        m_g = O.block_mask(c_g, np.where(i_g < 0, 0, i_g))
        win = O.window_mask(og, w) if w is not None else np.zeros((og.NB, og.NB), dtype=bool)
        assert np.all(m_g[..., win]), "window blocks missing"
        inter = O.block_mask(ref["inter_counts"], ref["inter_indices"])
        view = (m_g & ~win) | (inter & win)
        cv, iv = O.lists_from_mask(view)
        for k in range(len(heads)):
            sl = (slice(None), slice(k, k + 1))
            n_ex += P.compare_selection(ref["scores"][sl], ref["inter_counts"][sl],
                                        ref["inter_indices"][sl], cv[sl], iv[sl], "topp",
                                        tau=float(t_ref[k]))
        ro, _ = P.oracle_attention_on_lists(Qn[:, heads], Kn[:, heads], Vn[:, heads], og, c_g, i_g,
                                            scale)
        ref_O[:, heads] = ro
    err = P.finite_max_abs(P.to_np64(p.O), ref_O)
    _say(f"  exempt rows {n_ex}, max-abs {err:.3e}")
    assert err <= P.ATTN_MAX_ABS


@pytest.mark.parametrize("func", [0, 1])
def test_policy_sweep_matches_oracle(func):
    """Each head group's selection is the oracle's composed selection with the
    window and the per-head k of the policy; the whole output matches the oracle."""
    grid, cands = (6, 16, 20), [(2, 4, 4), (3, 4, 5), (2, 8, 2)]
    cfg = P.small_cfg(*grid, 1, 1, 1, d=64, H=6)
    _say("policy sweep, func", func)
    Q, K, V = P.bf16_inputs(cfg)
    pol = Policy(func)
    p = SweepPath(1, 6, 64, *grid, cands, 0.7, device=DEV, policy=pol)
    P.nan_fill(p.O)
    p.evaluate(Q, K)
    work = p.work_list(torch.cuda.current_stream())
    best = p.best.cpu().numpy()
    Qn, Kn, Vn = P.to_np64(Q), P.to_np64(K), P.to_np64(V)
    scale = P.scale_of(64)
    ref_O = np.zeros(Qn.shape)
    n_ex = 0
    for c, heads in work:
        v = p.group_select(c, heads, Q, K, V)
        p.group_attend(c, v)
        p.group_restore(c, heads, v)
        torch.cuda.synchronize()
        og = O.Geometry(*grid, *cands[c])
        w, _, k_dyn = O.policy_split(p.topk[c], func)
        k_ref = O.policy_head_budgets(best[heads], max(k_dyn, 1), og.NB)
        k_gpu = p.gb[c]["k_heads"][: len(heads)].cpu().numpy()
        assert np.array_equal(k_gpu, k_ref)
        spec = O.MaskSpec(mode="topk", topk_per_head=tuple(int(x) for x in k_ref), window=w)
        ref = O.spade_attention_composed(Qn[:, heads], Kn[:, heads], Vn[:, heads], og, spec, scale)
        c_g, i_g = v["counts"].cpu().numpy(), v["indices"].cpu().numpy()
        m_g = O.block_mask(c_g, np.where(i_g < 0, 0, i_g))
        win = O.window_mask(og, w) if w is not None else np.zeros((og.NB, og.NB), dtype=bool)
        assert np.all(m_g[..., win]), "window blocks missing"
        inter = O.block_mask(ref["inter_counts"], ref["inter_indices"])
        view = (m_g & ~win) | (inter & win)
        cv, iv = O.lists_from_mask(view)
        for k in range(len(heads)):
            sl = (slice(None), slice(k, k + 1))
            n_ex += P.compare_selection(ref["scores"][sl], ref["inter_counts"][sl],
                                        ref["inter_indices"][sl], cv[sl], iv[sl], "topk")
        # attention of the group on the GPU's own lists, every element
        ro, _ = P.oracle_attention_on_lists(Qn[:, heads], Kn[:, heads], Vn[:, heads], og, c_g, i_g,
                                            scale)
        ref_O[:, heads] = ro
    err = P.finite_max_abs(P.to_np64(p.O), ref_O)
    _say(f"  exempt rows {n_ex}, max-abs {err:.3e}")
    assert err <= P.ATTN_MAX_ABS
