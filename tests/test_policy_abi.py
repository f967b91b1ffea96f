"""The host rules of the policy function behind the C ABI (spade_policy_dense,
spade_policy_split): the same hand tables that pin the oracle's reading (§4.1:
dense warm-up for 30% / 25% of the steps, Turbo; Func 0's 30:1 and Func 1's ~80/20
budget split over the radius ladder), then agreement with the oracle over every
step count and budget tried, and the host-side error paths. No GPU needed."""
import pytest

from oracle import spade_oracle as O
from paper_2608_03335_amd import spade as S


@pytest.mark.parametrize("n,task,turbo,last_dense", [
    (50, S.SPADE_TASK_T2V, False, 14),    # 15 of 50 steps = 30%
    (50, S.SPADE_TASK_I2V, False, 12),    # ceil(12.5) = 13 steps
    (40, S.SPADE_TASK_T2V, False, 11),    # 12 of 40
    (10, S.SPADE_TASK_T2V, False, 2),     # 3 of 10
    (50, S.SPADE_TASK_T2V, True, 0),      # Turbo: only the first step
    (1, S.SPADE_TASK_T2V, False, 0),
])
def test_warmup_hand_table(n, task, turbo, last_dense):
    dense = [s for s in range(n) if S.spade_policy_dense(s, n, task, turbo)]
    assert dense == list(range(last_dense + 1))


@pytest.mark.parametrize("k_total,func,window,k_dyn", [
    (54, 1, (0, 1, 1), 45),    # static round(10.8) = 11 -> the 3x3 window (9)
    (54, 0, (0, 0, 0), 53),    # static round(54/31) = 2 -> the block itself
    (90, 0, (0, 0, 1), 87),    # static 3 -> (0,0,1), 3 blocks
    (2, 0, None, 2),           # static 0: no window
    (200, 1, (1, 1, 1), 173),  # static 40 -> 27 blocks
    (700, 1, (2, 2, 2), 575),  # static 140 -> the top of the ladder, 125 blocks
])
def test_split_hand_table(k_total, func, window, k_dyn):
    w, size, kd = S.spade_policy_split(k_total, func)
    assert w == window and kd == k_dyn and size + kd == k_total


@pytest.mark.parametrize("task,turbo", [("t2v", False), ("i2v", False), ("t2v", True)])
def test_warmup_matches_oracle(task, turbo):
    t = S.SPADE_TASK_T2V if task == "t2v" else S.SPADE_TASK_I2V
    for n in range(1, 201):
        assert [S.spade_policy_dense(s, n, t, turbo) for s in range(n)] == \
            [O.policy_dense(s, n, task, turbo) for s in range(n)], n


@pytest.mark.parametrize("func", [0, 1])
def test_split_matches_oracle(func):
    for k in range(1, 2000):
        assert S.spade_policy_split(k, func) == O.policy_split(k, func), k


def test_host_errors():
    for args in ((5, 5, 0, 0), (-1, 5, 0, 0), (0, 0, 0, 0), (0, 5, 2, 0)):
        with pytest.raises(S.SpadeError) as e:
            S.spade_policy_dense(*args)
        assert e.value.status == S.SPADE_ERR_INVALID_ARG
    for args in ((0, 1), (10, 2), (10, -1)):
        with pytest.raises(S.SpadeError) as e:
            S.spade_policy_split(*args)
        assert e.value.status == S.SPADE_ERR_INVALID_ARG
