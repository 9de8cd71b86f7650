"""Pins of the oracle's smooth weighted round robin (policy 5), a reading
of Sec. "Weighted Scheduling": the paper fixes the dispatch ratio and the
cyclic service, not the order of the tiers inside a cycle. In the smooth
reading every non-empty queue's credit grows by its weight before each
dispatch, the largest credit (the lowest tier on ties) is served and gives
up the sum of the non-empty queues' weights; a queue that runs empty
leaves and the others keep their credits (the published rule passes over
an unavailable peer and leaves every credit as it is). Expected sequences
are traced by hand below or follow from known properties of the rule, never
from the oracle."""
import numpy as np
import pytest

SMOOTH = 5


def letters(oracle, sizes, weights, names="abcdefghijklmnop"):
    tier = np.concatenate([np.full(s, q, np.uint8) for q, s in enumerate(sizes)])
    arr = np.arange(tier.size, dtype=np.float64)   # FIFO = index order
    perm, key = oracle.order(SMOOTH, tier, arr, weights=weights,
                             tier_priority=[float(q) for q in range(len(weights))])
    return "".join(names[tier[i]] for i in perm), perm, key, tier


def test_nginx_5_1_1(oracle):
    # credits (a, b, c), total 7:
    #  (5,1,1) a -> (-2,1,1); (3,2,2) a -> (-4,2,2); (1,3,3) b -> (1,-4,3);
    #  (6,-3,4) a -> (-1,-3,4); (4,-2,5) c -> (4,-2,-2); (9,-1,-1) a ->
    #  (2,-1,-1); (7,0,0) a -> (0,0,0): back at the start, so the period of
    #  7 repeats while no queue runs empty
    s, _, _, _ = letters(oracle, (15, 3, 3), (5, 1, 1))   # no queue empties in 14
    assert s[:14] == "aabacaa" * 2


def test_equal_weights_round_robin(oracle):
    # credits (2,2,2) -> a, (-2,4,4) -> b, (0,0,6) -> c, back to (0,0,0)
    s, _, _, _ = letters(oracle, (4, 4, 4), (2, 2, 2))
    assert s == "abc" * 4


def test_exhaustion_hand_case(oracle):
    # weights (2,1,1), queue sizes (2,5,1), total 4:
    #  (2,1,1) a -> (-2,1,1); (0,2,2) b -> (0,-2,2); (2,-1,3) c -> c is empty:
    #  credits (0,0), total 3; (2,1) a -> a is empty; then b alone
    s, perm, key, tier = letters(oracle, (2, 5, 1), (2, 1, 1))
    assert s == "abcabbbb"
    # key: floor(k / weight) for the k-th request of its tier
    assert [key[i] for i in perm] == [0, 0, 0, 0, 1, 2, 3, 4]


def test_exhaustion_keeps_the_credits(oracle):
    # weights (1,1,1), sizes (3,1,3), total 3:
    #  (1,1,1) a -> (-2,1,1); (-1,2,2) b -> b is empty, the others keep
    #  theirs: (a,c) = (-1,2), total 2; (0,3) c -> (0,1); (1,2) c -> (1,0);
    #  (2,1) a -> (0,1); (1,2) c -> c is empty; a alone.
    # (Restarting every credit at 0 instead would give "abacacc".)
    s, perm, key, tier = letters(oracle, (3, 1, 3), (1, 1, 1))
    assert s == "abccaca"
    assert [key[i] for i in perm] == [0, 0, 0, 1, 1, 2, 2]


def test_exhaustion_then_a_new_pattern(oracle):
    # weights (3,2,1), sizes (1,10,10), total 6:
    #  (3,2,1) a -> a is empty; (b,c) keep (2,1), total 3;
    #  (4,2) b -> (1,2); (3,3) b -> (0,3); (2,4) c -> (2,1): the pattern
    #  b b c repeats (a restart from (0,0) would repeat b c b instead);
    #  b's tenth dispatch is the 14th after a's; then c alone
    s, _, _, _ = letters(oracle, (1, 10, 10), (3, 2, 1))
    assert s == "a" + "bbc" * 4 + "bb" + "c" * 6


def test_exhaustion_with_a_transient(oracle):
    # weights (3,1,1), sizes (2,6,6), total 5:
    #  (3,1,1) a -> (-2,1,1); (1,2,2) b -> (1,-3,2); (4,-2,3) a -> a is
    #  empty; (b,c) keep (-2,3), total 2: (-1,4) c -> (-1,2); (0,3) c ->
    #  (0,1); (1,2) c -> (1,0); (2,1) b -> (0,1); from (0,1) the pattern
    #  c b repeats (two dispatches of a start-up stretch before it); c's
    #  sixth dispatch is the 12th overall, then b alone
    s, perm, key, tier = letters(oracle, (2, 6, 6), (3, 1, 1))
    assert s == "abacccbcbcbcbb"
    assert [key[i] for i in perm] == [0, 0, 0, 0, 1, 2, 1, 3, 2, 4, 3, 5, 4, 5]


def test_one_tier_is_fifo(oracle):
    rng = np.random.default_rng(4)
    arr = rng.uniform(0, 10, 300)
    perm, _ = oracle.order(SMOOTH, np.zeros(300, np.uint8), arr, weights=(7,), tier_priority=(0.0,))
    assert list(perm) == sorted(range(300), key=lambda i: (arr[i], i))


@pytest.mark.parametrize("seed", range(20))
def test_period_counts_and_fifo(oracle, seed):
    # a known property of the smooth rule from zero credits: every W =
    # sum(w) dispatches serve exactly w_q requests of queue q and bring the
    # credits back to 0, so while every queue is non-empty each window of W
    # dispatches holds w_q of tier q; requests of a tier go in FIFO order;
    # the result is a permutation
    rng = np.random.default_rng(200 + seed)
    Q = int(rng.integers(1, 7))
    w = [int(x) for x in rng.integers(1, 12, Q)]
    W = sum(w)
    m = int(rng.integers(1, 5))
    sizes = [m * x + int(rng.integers(1, 30)) for x in w]    # more than m periods' worth
    tier = np.concatenate([np.full(s, q, np.uint8) for q, s in enumerate(sizes)])
    rng.shuffle(tier)
    arr = np.round(rng.uniform(0, 5, tier.size), 2)
    perm, _ = oracle.order(SMOOTH, tier, arr, weights=w, tier_priority=[float(q) for q in range(Q)])
    assert np.array_equal(np.sort(perm), np.arange(tier.size))
    t = tier[perm]
    for j in range(m):
        assert list(np.bincount(t[j * W:(j + 1) * W], minlength=Q)) == w
    fifo = sorted(range(tier.size), key=lambda i: (arr[i], i))
    for q in range(Q):
        assert list(perm[t == q]) == [i for i in fifo if tier[i] == q]


@pytest.mark.parametrize("seed", range(10))
def test_exhaustion_at_a_period_end(oracle, seed):
    # from zero credits the rule serves every queue w_q times in W
    # dispatches and the credits come back to 0; when the first queue runs
    # empty exactly at the end of such a period, the queues left hold zero
    # credits, so what follows is the zero-credit cycle of the queues left:
    # its first W' dispatches (W' = their weights' sum) hold w_q of each, and
    # that pattern repeats while none of them runs empty
    rng = np.random.default_rng(700 + seed)
    Q = int(rng.integers(2, 6))
    w = [int(x) for x in rng.integers(1, 7, Q)]
    W = sum(w)
    m = int(rng.integers(1, 4))
    sizes = [m * x + int(rng.integers(40, 80)) for x in w]
    sizes[0] = m * w[0]                   # queue 0 empties after m full periods
    s, perm, key, tier = letters(oracle, sizes, w)
    t = tier[perm]
    assert int(np.sum(t[:m * W] == 0)) == m * w[0]
    rest = t[m * W:]
    Wp = W - w[0]
    left = [sizes[q] - m * w[q] for q in range(Q)]
    end = min(((left[q] // w[q]) * Wp for q in range(1, Q)))   # whole cycles before any empties
    for j in range(Wp, end):
        assert rest[j] == rest[j - Wp]
    for q in range(1, Q):
        assert int(np.sum(rest[:Wp] == q)) == w[q]
