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


def test_early_exit_choice_rule():
    """The loop's automatic early exit: below half of gamma accepted on
    average, sentinels counting 0 (the same hand-worked cases as the native
    rule's check in tests/native/plan_check.cpp)."""
    from paper_2406_11016_amd.decode_loop import early_exit_pays
    assert early_exit_pays(np.array([2, 3, 3, 3]), 8)          # mean 2.75 < 4
    assert not early_exit_pays(np.array([4, 4, 4, 4]), 8)      # mean 4 is not below 4
    assert not early_exit_pays(np.array([6, 6, 6, 6]), 8)
    assert early_exit_pays(np.zeros(64, dtype=np.int32), 1)
    assert not early_exit_pays(np.array([1] * 32 + [0] * 32), 1)
    assert early_exit_pays(np.array([1] * 31 + [0] * 33), 1)
    assert early_exit_pays(np.array([-1, -1, 8, 0]), 8)        # sentinels count 0: mean 2
    assert not early_exit_pays(np.array([], dtype=np.int32), 8)
