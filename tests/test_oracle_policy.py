"""Pins for the oracle's policy function (§3.1 policy function; §4 configurations:
Func 0 / Func 1 budgets, full attention for the first 30% (text-to-video) or 25%
(image-to-video) of the denoising steps, Turbo; the policy study: budgets
negatively correlated with the Selected Aggregation Score)."""
import numpy as np
import pytest

from oracle import spade_oracle as O


@pytest.mark.parametrize("n,task,turbo,last_dense", [
    (50, "t2v", False, 14),    # 15 of 50 steps = 30%
    (50, "i2v", False, 12),    # ceil(12.5) = 13 steps
    (40, "t2v", False, 11),    # 12 of 40
    (10, "t2v", False, 2),     # 3 of 10
    (50, "t2v", True, 0),      # Turbo: only the first step
    (1, "t2v", False, 0),
])
def test_dense_warmup_steps(n, task, turbo, last_dense):
    dense = [s for s in range(n) if O.policy_dense(s, n, task, turbo)]
    assert dense == list(range(last_dense + 1))


@pytest.mark.parametrize("k_total,func,window,k_dyn", [
    (54, 1, (0, 1, 1), 45),    # static round(10.8) = 11 -> the 3x3 window (9)
    (54, 0, (0, 0, 0), 53),    # static round(54/31) = 2 -> the block itself
    (90, 0, (0, 0, 1), 87),    # static 3 -> (0,0,1), 3 blocks
    (2, 0, None, 2),           # static 0: no window
    (200, 1, (1, 1, 1), 173),  # static 40 -> 27 blocks
    (700, 1, (2, 2, 2), 575),  # static 140 -> the top of the ladder, 125 blocks
])
def test_budget_split_table(k_total, func, window, k_dyn):
    w, size, kd = O.policy_split(k_total, func)
    assert w == window and kd == k_dyn
    assert size + kd == k_total


def test_window_sizes_of_the_ladder():
    assert [O.window_size(w) for w in O.WINDOW_LADDER] == [1, 3, 9, 27, 45, 75, 125]


def test_head_budgets_by_hand():
    # w = 1/AS = (1, 2/3, 5/4, 5/6), W = 3.75, total 160: 42.67, 28.44, 53.33, 35.56
    assert O.policy_head_budgets([1.0, 1.5, 0.8, 1.2], 40, 360).tolist() == [43, 28, 53, 36]


def test_equal_scores_give_the_flat_budget_and_scale_does_not_matter():
    assert np.all(O.policy_head_budgets([0.7] * 24, 45, 360) == 45)
    rng = np.random.default_rng(0)
    a = rng.uniform(0.5, 1.8, 24)
    assert np.array_equal(O.policy_head_budgets(a, 45, 360), O.policy_head_budgets(a * 4.0, 45, 360))


def test_budgets_fall_as_scores_rise_and_keep_the_total():
    rng = np.random.default_rng(1)
    for H, kd in ((24, 45), (40, 76), (12, 27)):
        a = rng.uniform(0.4, 1.9, H)
        k = O.policy_head_budgets(a, kd, 10 ** 6)
        order = np.argsort(a, kind="stable")
        assert np.all(np.diff(k[order]) <= 0)
        assert abs(int(k.sum()) - H * kd) <= H // 2


def test_budgets_clamp_and_degenerate_scores():
    k = O.policy_head_budgets([1.0, 1000.0], 300, 360)
    assert k.tolist() == [360, 1]
    assert O.policy_head_budgets([0.0, -1.0, 2.0], 10, 100).tolist() == [1, 1, 30]
    assert O.policy_head_budgets([0.0, 0.0], 7, 5).tolist() == [5, 5]


def test_head_tau_by_hand():
    # dropped mass 4 x 0.1 = 0.4 spread as AS / 4: (0.1, 0.15, 0.05, 0.1)
    got = O.policy_head_tau([1.0, 1.5, 0.5, 1.0], 0.9)
    assert np.allclose(got, [0.9, 0.85, 0.95, 0.9], rtol=0, atol=1e-15)
    # a head without a positive score drops nothing; the others share 3 x 0.2
    got = O.policy_head_tau([0.0, 2.0, 1.0], 0.8)
    assert np.allclose(got, [1.0, 0.6, 0.8], rtol=0, atol=1e-15)
    # no score at all: the flat tau; a dominant head can fall below 0 (top block only)
    assert O.policy_head_tau([0.0, -3.0], 0.7).tolist() == [0.7, 0.7]
    assert O.policy_head_tau([10.0, 0.001], 0.3)[0] < 0.0


def test_head_tau_falls_as_scores_rise_and_keeps_the_mean():
    rng = np.random.default_rng(2)
    for H, tau in ((24, 0.9), (40, 0.95), (12, 0.8)):
        a = rng.uniform(0.4, 1.9, H)
        t = O.policy_head_tau(a, tau)
        order = np.argsort(a, kind="stable")
        assert np.all(np.diff(t[order]) <= 0)
        assert abs(float(np.mean(1.0 - t)) - (1.0 - tau)) <= 1e-12
        assert np.array_equal(t, O.policy_head_tau(a * 3.0, tau)) or \
            np.allclose(t, O.policy_head_tau(a * 3.0, tau), rtol=0, atol=1e-15)
    assert np.all(O.policy_head_tau([0.6] * 24, 0.9) == 0.9)
