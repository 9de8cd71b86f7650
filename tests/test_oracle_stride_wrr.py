"""Pins of the oracle's stride scheduling (policy 6), a reading of Sec.
"Weighted Scheduling" (the paper fixes the ratio and the cyclic service, not
the interleaving). Queue q's pass starts at its stride 1 / w_q and advances
by it per dispatch; the smallest pass (the lowest tier on ties) is served.
The k-th request of tier q therefore runs at pass (k + 1) / w_q, and the
order is the merge of all requests by (that pass, tier): the checks below
sort by exact fractions, apart from the hand-traced case."""
from fractions import Fraction

import numpy as np
import pytest

STRIDE = 6


def run(oracle, sizes, weights, shuffle_seed=None):
    tier = np.concatenate([np.full(s, q, np.uint8) for q, s in enumerate(sizes)])
    if shuffle_seed is not None:
        np.random.default_rng(shuffle_seed).shuffle(tier)
    arr = np.arange(tier.size, dtype=np.float64)   # FIFO = index order
    perm, key = oracle.order(STRIDE, tier, arr, weights=weights,
                             tier_priority=[float(q) for q in range(len(weights))])
    return perm, key, tier


def test_hand_case(oracle):
    # weights (2, 3), sizes (4, 6). Passes: a 1/2, 1, 3/2, 2; b 1/3, 2/3, 1,
    # 4/3, 5/3, 2. In order: b a b (a b at 1: a first) b a b (a b at 2)
    perm, key, tier = run(oracle, (4, 6), (2, 3))
    assert "".join("ab"[tier[i]] for i in perm) == "bababbabab"
    assert [key[i] for i in perm] == [0, 0, 0, 0, 0, 1, 1, 1, 1, 1]


@pytest.mark.parametrize("seed", range(20))
def test_merge_by_exact_pass(oracle, seed):
    rng = np.random.default_rng(900 + seed)
    Q = int(rng.integers(1, 9))
    w = [int(x) for x in rng.integers(1, 40, Q)]
    if seed % 4 == 0:
        w[0] = 2 ** 31 + 11   # large weights: the products pass 2^32
    sizes = [int(x) for x in rng.integers(0, 90, Q)]
    perm, key, tier = run(oracle, sizes, w, shuffle_seed=seed)
    # requests of a tier in FIFO (= index) order, each with its pass
    items = []
    for q in range(Q):
        for k, i in enumerate(np.flatnonzero(tier == q)):
            items.append((Fraction(k + 1, w[q]), q, int(i), k // w[q]))
    items.sort()
    assert list(perm) == [i for _, _, i, _ in items]
    assert list(key[perm]) == [float(r) for _, _, _, r in items]


@pytest.mark.parametrize("seed", range(10))
def test_prefix_counts(oracle, seed):
    # with every queue holding at least m w_q requests, the first m W
    # dispatches are those with pass <= m: exactly m w_q of each queue
    rng = np.random.default_rng(950 + seed)
    Q = int(rng.integers(1, 7))
    w = [int(x) for x in rng.integers(1, 12, Q)]
    m = int(rng.integers(1, 5))
    sizes = [m * x + int(rng.integers(0, 20)) for x in w]
    perm, _, tier = run(oracle, sizes, w, shuffle_seed=seed)
    t = tier[perm][:m * sum(w)]
    assert list(np.bincount(t, minlength=Q)) == [m * x for x in w]


def test_equal_weights_round_robin(oracle):
    perm, _, tier = run(oracle, (3, 3, 3), (4, 4, 4))
    assert "".join("abc"[tier[i]] for i in perm) == "abc" * 3


def test_one_tier_is_fifo(oracle):
    rng = np.random.default_rng(5)
    arr = rng.uniform(0, 10, 300)
    perm, _ = oracle.order(STRIDE, np.zeros(300, np.uint8), arr, weights=(3,), tier_priority=(0.0,))
    assert list(perm) == sorted(range(300), key=lambda i: (arr[i], i))
