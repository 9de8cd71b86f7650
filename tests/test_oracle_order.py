"""Pins of the oracle's dispatch orders (stage 4).

Policies of Sec. "Scheduling Engine": FIFO (arrival order), Priority (highest
tier first, FIFO within a tier; the score priority*10^12 + arrival),
Weighted (cyclic dispatch by the configured ratio, 50/30/20 in the paper),
SJF (lower estimated budget first), Aging Priority (waiting lowers the
effective score). Expected orders come from Python's sorted() on tuple keys,
from hand-worked cases and from closed forms, never from the oracle.
"""
import numpy as np
import pytest

FIFO, PRIORITY, WEIGHTED, SJF, AGING = 0, 1, 2, 3, 4


def _random_batch(seed, n, quantize=None, tiers=3):
    rng = np.random.default_rng(seed)
    arrival = rng.uniform(0.0, 10.0, n)
    if quantize:
        arrival = np.round(arrival / quantize) * quantize   # many equal arrivals
    tier = rng.integers(0, tiers, n).astype(np.uint8)
    budget = rng.integers(1, 40, n).astype(np.float64) * 16.0  # many equal budgets
    return tier, arrival, budget


def _is_perm(p, n):
    return np.array_equal(np.sort(p), np.arange(n, dtype=p.dtype))


@pytest.mark.parametrize("seed,n,q", [(1, 1, None), (2, 7, None), (3, 300, None),
                                      (4, 300, 0.5), (5, 2000, 0.01), (6, 0, None)])
def test_brute_force_sorted(oracle, seed, n, q):
    tier, arr, bud = _random_batch(seed, n, q)
    prio = (0.0, 1.0, 2.0)
    rho, t_now = 0.1, 10.0
    want = {
        FIFO: sorted(range(n), key=lambda i: (arr[i], i)),
        PRIORITY: sorted(range(n), key=lambda i: (prio[tier[i]], arr[i], i)),
        SJF: sorted(range(n), key=lambda i: (bud[i], arr[i], i)),
        AGING: sorted(range(n), key=lambda i: (max(0.0, prio[tier[i]] - rho * max(0.0, t_now - arr[i])),
                                               arr[i], i)),
    }
    for pol, w in want.items():
        perm, _ = oracle.order(pol, tier, arr, bud, tier_priority=prio, aging_rate=rho,
                               t_now=t_now, aging_floor=0.0)
        assert list(perm) == w, pol
        assert _is_perm(perm, n)


def test_priority_guarantees(oracle):
    tier, arr, bud = _random_batch(11, 3000, 0.05)
    perm, key = oracle.order(PRIORITY, tier, arr, bud)
    t = tier[perm]
    # Premium before Standard before Batch
    assert np.all(np.diff(t.astype(int)) >= 0)
    # FIFO within each tier
    for q in range(3):
        a = arr[perm[t == q]]
        assert np.all(np.diff(a) >= 0)
    assert np.array_equal(key, np.array([0.0, 1.0, 2.0])[tier])


def test_priority_score_fp64_would_break_fifo():
    # why the score is evaluated exactly: at 5,000 arrivals/s the spacing of
    # fp64 values near 2*10^12 (2^-12 s) exceeds typical inter-arrival gaps
    a, b = 0.0002, 0.00021
    assert 2e12 + a == 2e12 + b


def test_weighted_hand_case(oracle):
    # weights 4/2/1, queue sizes (5, 3, 2):
    # round 0 serves P P P P S S B, round 1 serves the rest: P S B
    tier = np.array([0] * 5 + [1] * 3 + [2] * 2, np.uint8)
    arr = np.arange(10, dtype=np.float64)
    perm, key = oracle.order(WEIGHTED, tier, arr, weights=(4, 2, 1))
    assert "".join("PSB"[tier[i]] for i in perm) == "PPPPSSBPSB"
    assert list(perm) == [0, 1, 2, 3, 5, 6, 8, 4, 7, 9]
    assert list(key[perm]) == [0] * 7 + [1] * 3


def test_weighted_50_30_20(oracle):
    # the paper's ratio: while every queue is non-empty, each prefix of 100m
    # dispatches exactly 50m Premium, 30m Standard and 20m Batch requests
    rng = np.random.default_rng(8)
    tier = np.array([0] * 600 + [1] * 400 + [2] * 300, np.uint8)
    rng.shuffle(tier)
    arr = rng.uniform(0, 100, tier.size)
    perm, _ = oracle.order(WEIGHTED, tier, arr, weights=(50, 30, 20),
                           tier_priority=(0.0, 1.0, 2.0))
    t = tier[perm]
    for m in range(1, 11):       # Batch empties after 15 rounds; check 10
        c = np.bincount(t[:100 * m], minlength=3)
        assert list(c) == [50 * m, 30 * m, 20 * m]
    for q in range(3):           # FIFO within each tier
        assert np.all(np.diff(arr[perm[t == q]]) >= 0)


def _weighted_closed_form(tier, arr, w):
    """Position of each request under blocked cyclic WRR, in closed form.

    With n_q requests in tier q and request i the k-th (0-based, FIFO) of
    its tier, it is served in round r = floor(k / w_q); the rounds before r
    dispatch sum_q' min(n_q', r w_q'); within round r the tiers before q
    dispatch min(w_q', max(0, n_q' - r w_q')); then i is number k - r w_q.
    """
    n = len(tier)
    Q = len(w)
    fifo = sorted(range(n), key=lambda i: (arr[i], i))
    nq = [0] * Q
    k = [0] * n
    for i in fifo:
        k[i] = nq[tier[i]]
        nq[tier[i]] += 1
    pos = [0] * n
    for i in range(n):
        q = tier[i]
        r = k[i] // w[q]
        p = sum(min(nq[j], r * w[j]) for j in range(Q))
        p += sum(min(w[j], max(0, nq[j] - r * w[j])) for j in range(q))
        pos[i] = p + k[i] - r * w[q]
    return pos


@pytest.mark.parametrize("seed", range(40))
def test_weighted_closed_form(oracle, seed):
    rng = np.random.default_rng(100 + seed)
    Q = int(rng.integers(1, 6))
    n = int(rng.integers(0, 200))
    w = [int(x) for x in rng.integers(1, 9, Q)]
    tier = rng.integers(0, Q, n).astype(np.uint8)
    if seed % 3 == 0 and Q > 1:
        tier[tier == 1] = 0      # an empty queue
    arr = np.round(rng.uniform(0, 5, n), 1)
    perm, _ = oracle.order(WEIGHTED, tier, arr, weights=w, tier_priority=[float(q) for q in range(Q)])
    pos = _weighted_closed_form(tier, arr, w)
    inv = np.empty(n, np.int64)
    inv[perm] = np.arange(n)
    assert list(inv) == pos


def test_aging_zero_rate_is_priority(oracle):
    tier, arr, bud = _random_batch(21, 1500, 0.02)
    p1, _ = oracle.order(PRIORITY, tier, arr)
    p2, k2 = oracle.order(AGING, tier, arr, aging_rate=0.0, t_now=20.0)
    assert np.array_equal(p1, p2)
    assert np.array_equal(k2, np.array([0.0, 1.0, 2.0])[tier])


def _dyadic_batch(seed, n):
    # arrivals on a 2^-10 grid, rate 2^-6: every aging key is exact
    rng = np.random.default_rng(seed)
    arr = rng.integers(0, 40 * 1024, n) / 1024.0
    tier = rng.integers(0, 3, n).astype(np.uint8)
    return tier, arr


def test_aging_unclamped_is_deadline_order(oracle):
    # with no floor, p - rho (t - a) sorts like the deadline a + p / rho, for
    # any t_now at or after the last arrival
    tier, arr = _dyadic_batch(31, 2000)
    rho = 2.0 ** -6
    prio = np.array([0.0, 1.0, 2.0])
    want = sorted(range(len(arr)), key=lambda i: (arr[i] + prio[tier[i]] / rho, arr[i], i))
    for t_now in (40.0, 64.0, 1000.0):
        perm, _ = oracle.order(AGING, tier, arr, aging_rate=rho, t_now=t_now,
                               aging_floor=-np.inf)
        assert list(perm) == want


def test_aging_clamped_closed_form(oracle):
    # with floor 0 (the top tier's priority): requests whose deadline
    # a + p/rho has passed are all at the floor and go first in FIFO order,
    # then the rest by deadline
    tier, arr = _dyadic_batch(32, 2000)
    rho = 2.0 ** -6
    prio = np.array([0.0, 1.0, 2.0])
    t_now = 100.0
    dl = arr + prio[tier] / rho
    due = sorted((i for i in range(len(arr)) if dl[i] <= t_now), key=lambda i: (arr[i], i))
    rest = sorted((i for i in range(len(arr)) if dl[i] > t_now), key=lambda i: (dl[i], arr[i], i))
    perm, key = oracle.order(AGING, tier, arr, aging_rate=rho, t_now=t_now, aging_floor=0.0)
    assert list(perm) == due + rest
    assert np.all(key >= 0.0)


def test_keys_returned(oracle):
    tier, arr, bud = _random_batch(41, 100)
    _, k = oracle.order(FIFO, tier, arr, bud)
    assert np.array_equal(k, arr)
    _, k = oracle.order(SJF, tier, arr, bud)
    assert np.array_equal(k, bud)


def test_rejects_bad_input(oracle):
    with pytest.raises(ValueError):
        oracle.order(FIFO, np.array([3], np.uint8), np.array([0.0]))
    with pytest.raises(ValueError):
        oracle.order(WEIGHTED, np.array([0], np.uint8), np.array([0.0]), weights=(0, 1, 1))
