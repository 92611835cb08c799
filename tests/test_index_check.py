"""CPU checks of the GPU tests' index-set rule (tests/gpu_util.py): planted
lists in near-tie and clear units must pass or fail as the rule says.  The
rule: bit equality with the oracle's set unless the oracle's gap at the k
boundary is within float64 rounding of a tie; then any TopK of the oracle
energies within that rounding bound, still k strictly ascending indices in
range."""
import numpy as np
import pytest

from tests.gpu_util import U64, check_index_sets, is_near_tie

M = 1000                       # rows summed per energy
TOL = 2 * (M + 1) * U64        # relative rounding bound of two summation orders


def _near_unit():
    # indices 2 and 5 are within rounding of each other at the k = 3 boundary
    e = np.array([9.0, 1.0, 4.0, 7.0, 0.5, 4.0 * (1 - TOL / 4), 2.0])
    ref = np.array([[0, 2, 3]])          # the oracle's TopK(3): 9, 7, 4
    return e[None], ref


def test_near_tie_detected():
    e, _ = _near_unit()
    assert is_near_tie(e[0], 3, M)
    assert not is_near_tie(e[0], 2, M)   # 9 vs 7: a clear gap
    assert not is_near_tie(e[0], 7, M)   # nothing dropped
    # equal rounded sums are a near tie unless the sums are exact
    assert is_near_tie(np.array([3.0, 1.0, 1.0]), 2, M)
    # ties at +inf / NaN come from the inputs and are not near ties
    assert not is_near_tie(np.array([np.inf, np.nan, 1.0]), 1, M)


def test_near_tie_accepts_either_topk():
    e, ref = _near_unit()
    assert check_index_sets(np.array([0, 2, 3]), ref, e, M, max_near=1) == 1
    # the other member of the near tie is also a valid TopK
    assert check_index_sets(np.array([0, 3, 5]), ref, e, M, max_near=1) == 1


@pytest.mark.parametrize("planted,what", [
    ([0, 3, 6], "drops both near-tied indices for a clearly smaller one"),
    ([2, 3, 5], "drops the largest energy"),
    ([0, 1, 3], "keeps a small energy"),
    ([0, 2], "wrong length"),
    ([3, 0, 2], "not ascending"),
    ([0, 2, 2], "duplicate"),
    ([0, 2, 7], "out of range"),
    ([-1, 0, 2], "negative"),
])
def test_near_tie_rejects_planted_lists(planted, what):
    e, ref = _near_unit()
    with pytest.raises(AssertionError):
        check_index_sets(np.array(planted), ref, e, M, max_near=1)


def test_near_tie_count_is_limited():
    e, ref = _near_unit()
    with pytest.raises(AssertionError):
        check_index_sets(np.array([0, 2, 3]), ref, e, M)      # max_near defaults to 0


def test_clear_unit_requires_bit_equality():
    e = np.array([[5.0, 1.0, 3.0, 2.0]])
    ref = np.array([[0, 2]])
    assert check_index_sets(np.array([0, 2]), ref, e, M) == 0
    with pytest.raises(AssertionError):
        check_index_sets(np.array([0, 3]), ref, e, M)


def test_exact_sums_require_bit_equality_on_ties():
    e = np.array([[4.0, 4.0, 1.0]])      # integer data: an exact tie, lower index wins
    ref = np.array([[0]])
    assert check_index_sets(np.array([0]), ref, e, M, exact_sums=True) == 0
    with pytest.raises(AssertionError):
        check_index_sets(np.array([1]), ref, e, M, exact_sums=True)
    # without exact sums the tie is a near tie and either index is a valid TopK
    assert check_index_sets(np.array([1]), ref, e, M, max_near=1) == 1


def test_nan_must_be_kept():
    e = np.array([[1.0, np.nan, 3.0, 3.0 * (1 - TOL / 4)]])
    ref = np.array([[1, 2]])             # NaN ranks first, then 3 (index 2)
    assert check_index_sets(np.array([1, 3]), ref, e, M, max_near=1) == 1
    with pytest.raises(AssertionError):
        check_index_sets(np.array([2, 3]), ref, e, M, max_near=1)
