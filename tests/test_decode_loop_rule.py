"""The draft-length rule of the decoding loop (host logic, no GPU): gamma
starts at 5, grows by 2 when every drafted token is accepted and otherwise
shrinks by 1 (Sec. 4, hyperparameters), kept within 1 .. gamma_max."""
import numpy as np

from paper_2406_11016_amd.decode_loop import next_gamma


def test_grow_when_all_accepted():
    assert next_gamma(5, np.array([5]), 20) == 7
    assert next_gamma(7, np.array([7, 7, 7]), 20) == 9


def test_shrink_otherwise():
    assert next_gamma(5, np.array([4]), 20) == 4
    assert next_gamma(5, np.array([0]), 20) == 4
    assert next_gamma(7, np.array([7, 6, 7]), 20) == 6     # every element must accept everything


def test_bounds():
    assert next_gamma(1, np.array([0]), 20) == 1
    assert next_gamma(19, np.array([19]), 20) == 20
    assert next_gamma(20, np.array([20]), 20) == 20


def test_sentinel_counts_as_rejection():
    assert next_gamma(5, np.array([-1]), 20) == 4
    assert next_gamma(5, np.array([5, -1]), 20) == 4


def test_trajectory():
    # accepted lengths of a short run and the gammas the rule gives
    gamma, seen = 5, []
    for L in [5, 7, 3, 6, 6, 2, 0, 1, 1, 3]:
        seen.append(gamma)
        gamma = next_gamma(gamma, np.array([min(L, gamma)]), 20)
    assert seen == [5, 7, 9, 8, 7, 6, 5, 4, 3, 2]
