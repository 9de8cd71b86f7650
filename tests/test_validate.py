"""The float-order validator itself: it accepts a valid order and rejects
each kind of mistake (CPU)."""
import numpy as np
import pytest

from tests.validate import check_float_order, fifo_rank


def test_fifo_rank_ties_and_signed_zero():
    arr = np.array([1.0, 0.0, -0.0, 1.0, 0.5])
    assert list(fifo_rank(arr)) == [3, 0, 1, 4, 2]


def case():
    arrival = np.array([3.0, 1.0, 2.0, 0.0, 4.0])
    key = np.array([2.0, 1.0, 2.0, 5.0, 1.0])
    perm = np.array([1, 4, 2, 0, 3])     # key 1 (arrivals 1, 4), key 2 (2, 3), key 5
    return arrival, key, perm


def test_accepts_valid():
    arrival, key, perm = case()
    assert check_float_order(perm, key, perm, key, arrival, 1.0) == 0


def test_counts_differences_within_tolerance():
    arrival, key, perm = case()
    k2 = key.copy()
    k2[2] = 2.0 * (1 - 4e-13)            # request 2 now just below request 0
    assert check_float_order(perm, k2, perm, key, arrival, 1.0) == 0
    # the same permutation is then also valid with request 2 first (swap)
    p2 = np.array([1, 4, 2, 0, 3])
    assert check_float_order(p2, k2, np.array([1, 4, 0, 2, 3]), key, arrival, 1.0) == 2


@pytest.mark.parametrize("mistake", ["not_perm", "key", "tie", "order"])
def test_rejects(mistake):
    arrival, key, perm = case()
    k, p = key.copy(), perm.copy()
    if mistake == "not_perm":
        p[0] = p[1]
    elif mistake == "key":
        k[3] = 5.0 * (1 + 1e-11)
    elif mistake == "tie":
        p = np.array([4, 1, 2, 0, 3])    # equal keys out of FIFO order
    else:
        p = np.array([2, 0, 1, 4, 3])
    with pytest.raises(AssertionError):
        check_float_order(p, k, perm, key, arrival, 1.0)
