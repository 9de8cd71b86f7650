"""Pins of the oracle's smooth weighted round robin (policy 5), a reading
of Sec. "Weighted Scheduling": the paper fixes the dispatch ratio and the
cyclic service, not the order of the tiers inside a cycle. In the smooth
reading every non-empty queue's credit grows by its weight before each
dispatch, the largest credit (the lowest tier on ties) is served and gives
up the sum of the non-empty queues' weights; a queue that runs empty
leaves, and a new cycle over the queues left begins with every credit back
at 0. Expected sequences are traced by hand below or follow from known
properties of the rule, never from the oracle."""
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


def test_exhaustion_restarts_the_cycle(oracle):
    # weights (1,1,1), sizes (3,1,3), total 3:
    #  (1,1,1) a -> (-2,1,1); (-1,2,2) b -> b is empty: credits (0,0), total 2;
    #  (1,1) a -> (-1,1); (0,2) c -> (0,0); (1,1) a -> a is empty; c alone.
    # (Had the credits been kept, (0,3) would serve c twice: "abccaca".)
    s, perm, key, tier = letters(oracle, (3, 1, 3), (1, 1, 1))
    assert s == "abacacc"
    assert [key[i] for i in perm] == [0, 0, 1, 0, 2, 1, 2]


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
def test_cycles_restart_when_a_queue_empties(oracle, seed):
    # after each point where a queue runs empty, the rest is the smooth
    # sequence of the queues left, from zero credits: its first W' dispatches
    # (W' = their weights' sum) hold w_q of each if no queue empties earlier,
    # and the pattern of one cycle repeats until a queue empties
    rng = np.random.default_rng(700 + seed)
    Q = int(rng.integers(2, 7))
    w = [int(x) for x in rng.integers(1, 9, Q)]
    sizes = [int(x) for x in rng.integers(1, 80, Q)]
    s, perm, key, tier = letters(oracle, sizes, w)
    t = tier[perm]
    left = list(sizes)
    k = 0
    while k < len(t):
        act = [q for q in range(Q) if left[q] > 0]
        Wp = sum(w[q] for q in act)
        # the phase ends where the first of the active queues empties
        served = dict((q, 0) for q in act)
        end = k
        while end < len(t):
            served[int(t[end])] += 1
            end += 1
            if any(served[q] == left[q] for q in act):
                break
        seg = t[k:end]
        for j in range(Wp, len(seg)):
            assert seg[j] == seg[j - Wp]        # one cycle's pattern repeats
        if len(seg) >= Wp:
            assert all(int(np.sum(seg[:Wp] == q)) == w[q] for q in act)
        for q in act:
            left[q] -= served[q]
        k = end
