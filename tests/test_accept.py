"""Longest-prefix acceptance rule (Sec. 3 step 4, App. A.1), by hand tables."""
import pytest

from oracle import model as om

P = [5, 6, 7, 8]          # verifier greedy tokens p_0..p_3 for D = 3


TABLE = [
    ([5, 6, 7], 3, [5, 6, 7, 8]),     # all drafts match: n = D, bonus p_D
    ([5, 6, 9], 2, [5, 6, 7]),
    ([5, 9, 7], 1, [5, 6]),           # a later match after a miss does not count
    ([9, 6, 7], 0, [5]),              # nothing matches: only the bonus p_0
]


@pytest.mark.parametrize("drafts,n,out", TABLE)
def test_accept_table(drafts, n, out):
    assert om.accept(drafts, P) == (n, out)


def test_accept_width_one():
    assert om.accept([], [4]) == (0, [4])


def test_forced_acceptance_commits_drafts_and_bonus():
    assert om.accept([1, 2, 3], [7, 8, 9, 10], forced_n=2) == (2, [1, 2, 9])
    assert om.accept([1, 2, 3], [7, 8, 9, 10], forced_n=0) == (0, [7])
    with pytest.raises(ValueError):
        om.accept([1, 2, 3], [7, 8, 9, 10], forced_n=4)
