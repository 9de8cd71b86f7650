"""Pins of the oracle's dispatch-tick loop (dsref_simulate).

Each check compares the loop with something other than its own code: the
closed form of FIFO dispatch (the arrival order), the EMA closed form for a
constant ratio, invariants every run must satisfy (work conservation, no
dispatch before arrival, one dispatch per request), and hand-worked cases
that fix each reading of the loop: SJF rescored from the updated factors,
Aging to the tick's time, and the Weighted cycle restarted at every tick.
"""
import numpy as np
import pytest

import workloads as synth
from tests import wl

FIFO, PRIORITY, WEIGHTED, SJF, AGING = 0, 1, 2, 3, 4


def sim(oracle, policy, arrival, tier=None, counts=None, group=None, observed=None,
        t_base=(100.0,), s_tenant=(1.0,), state=(1.0,), ticks=(1.0,), batch=32, **kw):
    n = len(arrival)
    tier = np.zeros(n, np.uint8) if tier is None else tier
    counts = np.zeros(n, np.uint32) if counts is None else counts
    group = np.zeros(n, np.uint32) if group is None else group
    observed = np.full(n, 100, np.uint32) if observed is None else observed
    return oracle.simulate(policy, arrival, tier, counts, np.zeros(n, np.uint8),
                           np.zeros(n, np.uint32), group, observed, t_base, s_tenant, state,
                           ticks, batch=batch, **kw)


def random_case(seed, n, G=5, tiers=3):
    rng = np.random.default_rng(seed)
    arrival = np.round(rng.uniform(0, 10, n), 1)          # many equal arrivals
    tier = rng.integers(0, tiers, n).astype(np.uint8)
    counts = rng.integers(0, 3000, n).astype(np.uint32)
    cat = rng.integers(0, 4, n).astype(np.uint8)
    ten = rng.integers(0, 6, n).astype(np.uint32)
    group = rng.integers(0, G, n).astype(np.uint32)
    obs = rng.integers(0, 4000, n).astype(np.uint32)
    return arrival, tier, counts, cat, ten, group, obs


def run_random(oracle, policy, seed, n, batch, ticks, G=5):
    arrival, tier, counts, cat, ten, group, obs = random_case(seed, n, G)
    return oracle.simulate(policy, arrival, tier, counts, cat, ten, group, obs,
                           [50.0, 100.0, 300.0, 800.0], np.linspace(0.5, 1.5, 6),
                           np.ones(G), ticks, batch=batch, alpha=0.2,
                           weights=(3, 2, 1), aging_rate=0.3), arrival


@pytest.mark.parametrize("policy", [FIFO, PRIORITY, WEIGHTED, SJF, AGING])
@pytest.mark.parametrize("batch", [1, 4, 32])
def test_invariants(oracle, policy, batch):
    ticks = np.concatenate([[0.0, 0.0], np.linspace(0.5, 12.0, 40)])
    (seq, tick_of, _), arrival = run_random(oracle, policy, 11 + batch, 400, batch, ticks)
    n = len(arrival)
    # each request at most once, seq and tick_of consistent, ticks in order
    assert len(set(seq.tolist())) == len(seq)
    assert np.array_equal(np.sort(np.flatnonzero(tick_of >= 0)), np.sort(seq))
    assert np.all(np.diff(tick_of[seq]) >= 0)
    # no dispatch before arrival
    assert np.all(arrival[seq] <= ticks[tick_of[seq]])
    # work conservation: tick k dispatches min(batch, arrived so far - dispatched before)
    done = 0
    for k, t in enumerate(ticks):
        arrived = int(np.sum(arrival <= t))
        want = min(batch, arrived - done)
        assert int(np.sum(tick_of == k)) == want
        done += want
    assert done == len(seq)
    assert np.all(tick_of[np.setdiff1d(np.arange(n), seq)] == -1)


@pytest.mark.parametrize("batch", [1, 7, 32])
def test_fifo_is_arrival_order(oracle, batch):
    # FIFO always takes the earliest pending requests, so over all ticks it
    # dispatches a prefix of the arrival order (ties by index)
    ticks = np.linspace(0.0, 11.0, 30)
    (seq, _, _), arrival = run_random(oracle, FIFO, 5, 500, batch, ticks)
    want = np.lexsort((np.arange(len(arrival)), arrival))
    assert np.array_equal(seq, want[:len(seq)])


def test_everything_at_once_is_the_policy_order(oracle):
    # one tick after every arrival with a batch that takes everything:
    # the dispatch sequence is the policy order of the whole set
    rng = np.random.default_rng(3)
    n = 300
    arrival = rng.uniform(0, 5, n)
    tier = rng.integers(0, 3, n).astype(np.uint8)
    # Priority: tiers by priority 0, 1, 2, FIFO within each
    seq, _, _ = sim(oracle, PRIORITY, arrival, tier=tier, ticks=[10.0], batch=n)
    fifo = np.argsort(arrival, kind="stable")
    want = np.concatenate([fifo[tier[fifo] == q] for q in range(3)])
    assert np.array_equal(seq, want)


def test_ema_closed_form(oracle):
    # observed = r * (B-free estimate) with r dyadic: after k completions of
    # the group its factor is r + (c0 - r)(1 - alpha)^k (Eq. (5), (6))
    n = 40
    arrival = np.zeros(n)
    counts = np.zeros(n, np.uint32)              # F = 1
    t_base, r, a, c0 = 64.0, 0.75, 0.25, 1.0    # estimate 64, observed 48
    obs = np.full(n, 48, np.uint32)
    for k, nd in [(1, 8), (3, 24), (5, 40)]:
        _, _, st = sim(oracle, FIFO, arrival, counts=counts, observed=obs, t_base=[t_base],
                       state=[c0], ticks=np.ones(k), batch=8, alpha=a)
        assert abs(st[0] - (r + (c0 - r) * (1 - a) ** nd)) <= 1e-14


def test_exact_estimates_keep_factor_one(oracle):
    # observed equal to the B-free estimate: the factor stays exactly 1
    arrival, tier, counts, cat, ten, group, _ = random_case(8, 300)
    t_base = np.array([64.0, 128.0, 256.0, 512.0])
    s = np.array([0.5, 1.0, 2.0, 1.0, 0.5, 0.25])
    counts[:] = 0                                 # F = 1: the estimates are integers
    obs = (t_base[cat] * s[ten]).astype(np.uint32)
    _, _, st = oracle.simulate(SJF, arrival, tier, counts, cat, ten, group, obs, t_base, s,
                               np.ones(5), np.linspace(1, 10, 20), batch=16, alpha=0.25)
    assert np.all(st == 1.0)


def test_sjf_rescored_from_updated_factors(oracle):
    # Requests 0, 1 in group 0 (factor 1.0), 2, 3 in group 1 (factor 1.5);
    # B-free estimate 100 each, so the budgets are 100, 100, 150, 150. Tick 0
    # dispatches request 0, whose completion (observed 400, ratio 4) lifts
    # group 0's factor to 0.5 * 1 + 0.5 * 4 = 2.5 and request 1's budget to
    # 250: ticks 1 and 2 take group 1 first.
    arrival = np.zeros(4)
    group = np.array([0, 0, 1, 1], np.uint32)
    obs = np.array([400, 400, 150, 150], np.uint32)
    seq, tick_of, st = sim(oracle, SJF, arrival, group=group, observed=obs, state=[1.0, 1.5],
                           ticks=[1.0, 2.0, 3.0], batch=1, alpha=0.5)
    assert seq.tolist() == [0, 2, 3]
    assert tick_of.tolist() == [0, -1, 1, 2]
    assert st.tolist() == [2.5, 1.5]
    # without feedback (alpha = 0) the budgets stay 100, 100, 150, 150
    seq, _, st = sim(oracle, SJF, arrival, group=group, observed=obs, state=[1.0, 1.5],
                     ticks=[1.0, 2.0, 3.0], batch=1, alpha=0.0)
    assert seq.tolist() == [0, 1, 2] and st.tolist() == [1.0, 1.5]


def test_aging_uses_tick_time(oracle):
    # tier 1 (priority 1) arrived at 0, tier 0 (priority 0) arrives at 5;
    # rate 0.25: at tick 5 the old request has score max(-10, 1 - 1.25) =
    # -0.25 < 0, so it goes first; at tick 1 (score 0.75) it would not
    arrival = np.array([0.0, 5.0])
    tier = np.array([1, 0], np.uint8)
    seq, _, _ = sim(oracle, AGING, arrival, tier=tier, ticks=[5.0], batch=1, aging_rate=0.25,
                    aging_floor=-10.0)
    assert seq.tolist() == [0]
    # with the floor: request 0 (priority 2, arrived 0) and request 1
    # (priority 1, arrived 1), rate 0.25, floor 0. At tick 2 the scores are
    # 1.5 and 0.75; at tick 9 both are clamped to 0 and FIFO decides.
    arrival = np.array([0.0, 1.0])
    tier = np.array([2, 1], np.uint8)
    seq, _, _ = sim(oracle, AGING, arrival, tier=tier, ticks=[2.0], batch=1, aging_rate=0.25)
    assert seq.tolist() == [1]
    seq, _, _ = sim(oracle, AGING, arrival, tier=tier, ticks=[9.0], batch=1, aging_rate=0.25)
    assert seq.tolist() == [0]


def test_weighted_cycle_restarts_each_tick(oracle):
    # weights (2, 1); requests 0-3 in tier 0, 4-5 in tier 1, all arrived.
    # The whole set's cycle is 0 1 4 2 3 5; with batch 2 and a fresh cycle
    # per tick: tick 0 takes 0 1, tick 1 re-cycles {2 3 4 5} -> 2 3, tick 2
    # takes 4 5. (A cycle carried across ticks would serve 4 at tick 1.)
    arrival = np.arange(6, dtype=np.float64) * 0.01
    tier = np.array([0, 0, 0, 0, 1, 1], np.uint8)
    seq, tick_of, _ = sim(oracle, WEIGHTED, arrival, tier=tier, ticks=[1.0, 2.0, 3.0], batch=2,
                          weights=(2, 1), tier_priority=(0.0, 1.0))
    assert seq.tolist() == [0, 1, 2, 3, 4, 5]
    assert tick_of.tolist() == [0, 0, 1, 1, 2, 2]
    seq, _, _ = sim(oracle, WEIGHTED, arrival, tier=tier, ticks=[1.0], batch=6,
                    weights=(2, 1), tier_priority=(0.0, 1.0))
    assert seq.tolist() == [0, 1, 4, 2, 3, 5]


def test_pending_set_and_empty_ticks(oracle):
    # nothing pending: nothing dispatched, tick_of stays -1
    arrival = np.array([5.0, 6.0, 7.0])
    seq, tick_of, st = sim(oracle, FIFO, arrival, ticks=[1.0, 2.0])
    assert len(seq) == 0 and tick_of.tolist() == [-1, -1, -1] and st[0] == 1.0
    # arrival exactly at the tick counts as arrived
    seq, tick_of, _ = sim(oracle, FIFO, arrival, ticks=[5.0, 6.5, 7.0])
    assert seq.tolist() == [0, 1, 2] and tick_of.tolist() == [0, 1, 2]
    # no requests, no ticks
    seq, tick_of, _ = sim(oracle, SJF, np.zeros(0), ticks=[1.0])
    assert len(seq) == 0 and len(tick_of) == 0
    seq, tick_of, _ = sim(oracle, SJF, np.zeros(3), ticks=[])
    assert len(seq) == 0 and tick_of.tolist() == [-1, -1, -1]


def test_rejects_bad_input(oracle):
    with pytest.raises(ValueError):
        sim(oracle, FIFO, np.zeros(2), batch=0)
    with pytest.raises(ValueError):
        sim(oracle, WEIGHTED, np.zeros(2), tier=np.array([0, 3], np.uint8))


def test_synthetic_workload_drains(oracle):
    # a reduced copy of the 65,536-request workload: 10 ms ticks of 32
    # against 5,000 arrivals/s build a queue, and the schedule drains it
    b = wl.load("batch64k", n=3000, with_text=False)
    ticks = synth.sim_ticks(b.arrival)
    for pol in (FIFO, SJF):
        seq, tick_of, st = oracle.simulate(pol, b.arrival, b.tier, b.words, b.category, b.tenant,
                                           b.group, b.observed, b.t_base, b.s_tenant,
                                           np.ones(b.n_groups), ticks, batch=32, alpha=0.1)
        assert len(seq) == b.n
        waits = ticks[tick_of] - b.arrival
        assert waits.min() >= 0
        # the drift ratio's mean is above 1: the factors rise from 1
        assert np.mean(st) > 1.2
