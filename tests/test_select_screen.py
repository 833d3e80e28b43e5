"""CPU checks of the near-tie screen used by the selection parity cases."""
import numpy as np

from oracle.greedy import greedy_select
from select_cases import NEAR_TIE, greedy_margins, make_case, screened_cases


def test_exact_tie_has_zero_margin():
    # q = (+1, -1, +0.5, +0.5), y = 0: the first iteration ties candidates 2 and 3
    cand = np.array([[1.0], [-1.0], [0.5], [0.5]])
    assert greedy_margins(cand, np.zeros(1), "reg", 4) == 0.0


def test_margin_of_a_two_candidate_case():
    # y = 0, singles score 1 and 2 (gap 1 relative to 1); the pair scores 1.5,
    # no improvement on 1: gap |1 - 1.5| / 1.5
    cand = np.array([[1.0], [2.0]])
    assert np.isclose(greedy_margins(cand, np.zeros(1), "reg", 2), 1.0 / 3.0)


def test_screened_cases_are_tie_free_and_follow_the_oracle():
    for task in ("reg", "bin", "multi"):
        (cand, y, gap), = screened_cases(task, 12, 200, 6, seeds=range(100, 150))
        assert gap >= NEAR_TIE
        sel, _ = greedy_select(cand, y, task, 6)
        assert len(sel) >= 1 and len(set(sel)) == len(sel)
        # a case built with a duplicated best candidate is rejected
        dup = np.concatenate([cand[sel[:1]], cand])
        assert greedy_margins(dup, y, task, 6) == 0.0


def test_make_case_is_seeded():
    a = make_case("bin", 4, 10, 3)
    b = make_case("bin", 4, 10, 3)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
