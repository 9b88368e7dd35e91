"""The label checks of the GPU tests, on hand-built decision tables (no GPU)."""
import numpy as np
import pytest

from tests.label_checks import check_binary_labels, check_ovo_predictions, kkt_and_gap, ovo_allowed_classes, ovo_vote


def test_ovo_vote_rule():
    # k = 3, pairs (0,1), (0,2), (1,2)
    assert ovo_vote([True, True, True], 3) == 0
    assert ovo_vote([False, False, True], 3) == 1
    assert ovo_vote([False, False, False], 3) == 2
    assert ovo_vote([True, False, True], 3) == 0    # one vote each: ties to the smallest class
    assert ovo_vote([False, True, False], 3) == 0   # 0 beats 2, 1 beats 0, 2 beats 1: three-way tie
    # k = 4, pairs (0,1), (0,2), (0,3), (1,2), (1,3), (2,3)
    assert ovo_vote([True, False, False, True, False, True], 4) == 2   # votes 1, 1, 2, 2: tie of 2 and 3
    assert ovo_vote([False, False, False, True, False, False], 4) == 3  # votes 0, 2, 1, 3
    assert ovo_vote([False, True, True, True, True, True], 4) == 1     # votes 2, 3, 1, 0


def test_ovo_allowed_classes_enumerates_near_zero_pairs():
    d = np.array([-1e-4, 0.5, 0.3])  # 1 beats 0 by a margin of 1e-4, 0 beats 2, 1 beats 2
    assert ovo_allowed_classes(d, 3, 0.0) == {1}
    assert ovo_allowed_classes(d, 3, 2e-4) == {0, 1}
    assert check_ovo_predictions([0], d[None, :], 3, 2e-4) == 1
    assert check_ovo_predictions([1], d[None, :], 3, 2e-4) == 1
    with pytest.raises(AssertionError):
        check_ovo_predictions([2], d[None, :], 3, 2e-4)
    with pytest.raises(AssertionError):
        check_ovo_predictions([0], d[None, :], 3, 5e-5)


def test_binary_labels_only_differ_near_zero():
    ref = np.array([0.5, -0.3, 1e-5, -2e-5])
    assert check_binary_labels(ref + np.array([0, 0, -2e-5, 3e-5]), ref, 5e-5) == 2
    with pytest.raises(AssertionError):
        check_binary_labels(np.array([-0.5, -0.3, 1e-5, -2e-5]), ref, 5e-5)


def test_kkt_and_gap_on_an_exact_two_point_optimum():
    # two points, RBF: a1 = a2 = 1/(1-k), b = 0; f_i = sum_j a_j y_j K_ij - y_i = 0 at the optimum
    k = np.exp(-0.3 * 5.5)
    a = np.full(2, 1.0 / (1.0 - k))
    y = np.array([1.0, -1.0])
    K = np.array([[1.0, k], [k, 1.0]])
    f = K @ (a * y) - y
    gap, W = kkt_and_gap(f, y, a, 0.0, 10.0, 1e-3, slack=0.0)
    assert abs(gap) < 1e-12 and abs(W - a.sum() / 2) < 1e-12
    with pytest.raises(AssertionError):  # a planted KKT violation
        kkt_and_gap(f + np.array([-0.01, 0.0]), y, a, 0.0, 10.0, 1e-3, slack=0.0)
