"""The host side of the policy function (warm-up schedule and budget split)
agrees with the oracle's reading for every step count and budget tried."""
import pytest

from oracle import spade_oracle as O
from paper_2608_03335_amd.policy import WINDOW_LADDER, Policy, window_blocks


@pytest.mark.parametrize("task,turbo", [("t2v", False), ("i2v", False), ("t2v", True)])
def test_warmup_schedule_matches_oracle(task, turbo):
    for n in range(1, 121):
        p = Policy(1, n_steps=n, task=task, turbo=turbo)
        assert [p.dense(s) for s in range(n)] == [O.policy_dense(s, n, task, turbo) for s in range(n)]


@pytest.mark.parametrize("func", [0, 1])
def test_split_matches_oracle(func):
    p = Policy(func)
    for k in range(1, 1200):
        assert p.split(k) == O.policy_split(k, func)


def test_ladder_matches_oracle():
    assert WINDOW_LADDER == O.WINDOW_LADDER
    assert [window_blocks(w) for w in WINDOW_LADDER] == [O.window_size(w) for w in O.WINDOW_LADDER]
