"""The dispatch-tick loop on the GPU against the oracle.

The dispatch sequence, the tick of every request and the dispatch count are
compared exactly. The factors are compared exactly too: both sides apply the
EMA updates of each group one after another in dispatch order with the same
operations (no fused multiply-add), and SJF's budgets, which decide the
order, come from them.
"""
import numpy as np
import pytest

import workloads as synth
from tests import wl
from tests.gpu_util import dev, host

pytestmark = pytest.mark.gpu

FIFO, PRIORITY, WEIGHTED, SJF, AGING = 0, 1, 2, 3, 4
ALL = [FIFO, PRIORITY, WEIGHTED, SJF, AGING]


@pytest.fixture(scope="module")
def ds():
    from paper_2606_02982_amd import driftsched
    return driftsched


def run_gpu(ds, policy, arrival, tier, counts, category, tenant, group, observed, t_base,
            s_tenant, state, ticks, batch=32, alpha=0.1, weights=(4, 2, 1),
            tier_priority=(0.0, 1.0, 2.0), aging_rate=0.01, aging_floor=0.0, validate=False,
            f_ref=1024.0):
    """(seq, n_dispatched, tick_of, state) from ds_simulate."""
    arrival = np.asarray(arrival, np.float64)
    print("simulate policy=%d n=%d ticks=%d batch=%d" % (policy, len(arrival), len(ticks), batch),
          flush=True)
    p = ds.sim_params(policy, batch=batch, alpha=alpha, n_tiers=len(weights), weights=weights,
                      tier_priority=tier_priority, aging_rate=aging_rate, aging_floor=aging_floor,
                      f_ref=f_ref)
    st = dev(np.asarray(state, np.float64).copy())
    seq, tick_of, nd = ds.simulate(dev(arrival), dev(np.asarray(tier, np.uint8)),
                                   dev(np.asarray(counts, np.uint32)),
                                   dev(np.asarray(category, np.uint8)),
                                   dev(np.asarray(tenant, np.uint32)),
                                   dev(np.asarray(group, np.uint32)),
                                   dev(np.asarray(observed, np.uint32)),
                                   dev(np.asarray(t_base, np.float64)),
                                   dev(np.asarray(s_tenant, np.float64)), st,
                                   dev(np.asarray(ticks, np.float64)), p, validate=validate)
    return host(seq, np.uint32), int(host(nd)[0]), host(tick_of), host(st)


def both(ds, oracle, policy, arrival, tier, counts, category, tenant, group, observed, t_base,
         s_tenant, state, ticks, batch=32, alpha=0.1, weights=(4, 2, 1),
         tier_priority=(0.0, 1.0, 2.0), aging_rate=0.01, aging_floor=0.0, validate=False,
         f_ref=1024.0):
    w_seq, w_tick, w_state = oracle.simulate(policy, arrival, tier, counts, category, tenant,
                                             group, observed, t_base, s_tenant, state, ticks,
                                             batch=batch, alpha=alpha, weights=weights,
                                             tier_priority=tier_priority, aging_rate=aging_rate,
                                             aging_floor=aging_floor, f_ref=f_ref)
    seq, nd, tick_of, got = run_gpu(ds, policy, arrival, tier, counts, category, tenant, group,
                                    observed, t_base, s_tenant, state, ticks, batch, alpha,
                                    weights, tier_priority, aging_rate, aging_floor, validate,
                                    f_ref)
    assert nd == len(w_seq), "dispatched %d, oracle %d" % (nd, len(w_seq))
    if nd:
        bad = np.flatnonzero(seq[:nd] != w_seq)
        assert bad.size == 0, "first difference at dispatch %d: %d vs %d" % (
            bad[0], seq[bad[0]], w_seq[bad[0]])
    assert np.all(seq[nd:] == 0xFFFFFFFF)
    assert np.array_equal(tick_of, w_tick)
    assert np.array_equal(got, w_state), "factors differ: max |d| %g" % np.abs(got - w_state).max()
    return seq[:nd], tick_of, got


def random_inputs(seed, n, G=5, n_cat=4, n_ten=6, tiers=3, round_arrival=1):
    rng = np.random.default_rng(seed)
    return dict(
        arrival=np.round(rng.uniform(0, 10, n), round_arrival),
        tier=rng.integers(0, tiers, n).astype(np.uint8),
        counts=rng.integers(0, 3000, n).astype(np.uint32),
        category=rng.integers(0, n_cat, n).astype(np.uint8),
        tenant=rng.integers(0, n_ten, n).astype(np.uint32),
        group=rng.integers(0, G, n).astype(np.uint32),
        observed=rng.integers(0, 4000, n).astype(np.uint32),
        t_base=np.array([50.0, 100.0, 300.0, 800.0])[:n_cat],
        s_tenant=np.linspace(0.5, 1.5, n_ten),
        state=rng.uniform(0.8, 1.2, G))


@pytest.mark.parametrize("policy", ALL)
@pytest.mark.parametrize("n,batch", [(1, 32), (400, 1), (400, 4), (400, 32), (5000, 32),
                                     (5000, 7), (3000, 1024)])
def test_random(ds, oracle, policy, n, batch):
    x = random_inputs(n + batch, n)
    ticks = np.concatenate([[0.0, 0.0], np.linspace(0.25, 12.0, 60)])
    both(ds, oracle, policy, ticks=ticks, batch=batch, alpha=0.2, weights=(3, 2, 1),
         aging_rate=0.3, **x)


@pytest.mark.parametrize("policy", ALL)
def test_large_pending_set(ds, oracle, policy):
    # a queue of up to 20,000 requests: the SJF/Aging select works over the
    # whole list in global memory before its bucket fits in LDS
    x = random_inputs(7, 20000, G=64, round_arrival=3)
    ticks = np.repeat([2.0, 6.0, 10.0, 10.0], [3, 3, 3, 20])
    both(ds, oracle, policy, ticks=ticks, batch=1000, alpha=0.05, aging_rate=0.05, **x)


@pytest.mark.parametrize("policy", [SJF, AGING, PRIORITY])
def test_all_keys_equal(ds, oracle, policy):
    # every key equal (one budget; every aged score clamped to the floor;
    # one tier): the order is FIFO, found by the select on list positions,
    # with more tied candidates than fit in LDS
    n = 12000
    rng = np.random.default_rng(1)
    arrival = np.round(rng.uniform(0, 1, n), 2)
    z8, z32 = np.zeros(n, np.uint8), np.zeros(n, np.uint32)
    tier = np.full(n, 1, np.uint8)
    seq, _, _ = both(ds, oracle, policy, arrival, tier, z32, z8, z32, z32, z32 + 100, [64.0],
                     [1.0], [1.0], ticks=[5.0, 5.0, 6.0], batch=1000, alpha=0.0,
                     aging_rate=10.0, aging_floor=0.0)
    assert np.array_equal(seq, np.lexsort((np.arange(n), arrival))[:3000])


def test_hand_cases(ds, oracle):
    # SJF rescored from the updated factor (see the oracle's pins)
    z = np.zeros(4, np.uint32)
    seq, tick_of, st = both(ds, oracle, SJF, np.zeros(4), np.zeros(4, np.uint8), z,
                            np.zeros(4, np.uint8), z, [0, 0, 1, 1], [400, 400, 150, 150], [100.0],
                            [1.0], [1.0, 1.5], [1.0, 2.0, 3.0], batch=1, alpha=0.5)
    assert seq.tolist() == [0, 2, 3] and tick_of.tolist() == [0, -1, 1, 2]
    assert st.tolist() == [2.5, 1.5]
    # Aging to the tick's time
    z = np.zeros(2, np.uint32)
    for t, want in [(2.0, [1]), (9.0, [0])]:
        seq, _, _ = both(ds, oracle, AGING, [0.0, 1.0], [2, 1], z, np.zeros(2, np.uint8), z, z,
                         [100, 100], [100.0], [1.0], [1.0], [t], batch=1, aging_rate=0.25)
        assert seq.tolist() == want
    # the Weighted cycle restarts at every tick
    z = np.zeros(6, np.uint32)
    seq, tick_of, _ = both(ds, oracle, WEIGHTED, np.arange(6) * 0.01, [0, 0, 0, 0, 1, 1], z,
                           np.zeros(6, np.uint8), z, z, z + 100, [100.0], [1.0], [1.0],
                           [1.0, 2.0, 3.0], batch=2, weights=(2, 1), tier_priority=(0.0, 1.0))
    assert seq.tolist() == [0, 1, 2, 3, 4, 5] and tick_of.tolist() == [0, 0, 1, 1, 2, 2]


def test_sixteen_tiers_and_shared_priorities(ds, oracle):
    x = random_inputs(3, 6000, tiers=16)
    w = tuple(range(1, 17))
    prio = tuple(float(q % 5) for q in range(16))       # classes shared by several tiers
    ticks = np.linspace(0.5, 10.0, 30)
    for pol in (PRIORITY, WEIGHTED, AGING):
        both(ds, oracle, pol, ticks=ticks, batch=64, weights=w, tier_priority=prio,
             aging_rate=0.2, aging_floor=-1e300, **x)


def test_empty(ds, oracle):
    e32, e8 = np.zeros(0, np.uint32), np.zeros(0, np.uint8)
    both(ds, oracle, SJF, np.zeros(0), e8, e32, e8, e32, e32, e32, [1.0], [1.0], [1.0], [1.0])
    x = random_inputs(2, 50)
    both(ds, oracle, FIFO, ticks=np.zeros(0), **x)
    both(ds, oracle, FIFO, ticks=[-1.0, -1.0], **x)      # before every arrival


def test_validate(ds, oracle):
    x = random_inputs(4, 300)
    ticks = np.linspace(1, 10, 10)
    both(ds, oracle, SJF, ticks=ticks, validate=True, **x)
    cases = [("tier", 3), ("category", 4), ("tenant", 6), ("group", 5), ("arrival", np.nan)]
    for field, bad in cases:
        y = dict(x)
        y[field] = x[field].copy()
        y[field][17] = bad
        with pytest.raises(ds.DriftSchedError) as e:
            run_gpu(ds, SJF, ticks=ticks, validate=True, **y)
        assert e.value.status == -5, field
    for t in (ticks[::-1].copy(), np.array([1.0, np.nan, 3.0])):
        with pytest.raises(ds.DriftSchedError) as e:
            run_gpu(ds, FIFO, ticks=t, validate=True, **x)
        assert e.value.status == -5


def test_repeatable(ds):
    x = random_inputs(9, 8000, G=16)
    ticks = np.linspace(0.5, 10.0, 40)
    a = run_gpu(ds, SJF, ticks=ticks, batch=100, **x)
    b = run_gpu(ds, SJF, ticks=ticks, batch=100, **x)
    for u, v in zip(a, b):
        assert np.array_equal(u, v)


@pytest.mark.parametrize("policy", ALL)
def test_synthetic_workload(ds, oracle, policy):
    # the 65,536-request workload: 10 ms ticks of 32 against 5,000
    # arrivals/s, 2,064 ticks, every request dispatched
    b = wl.load("batch64k", with_text=False)
    ticks = synth.sim_ticks(b.arrival)
    seq, _, _ = both(ds, oracle, policy, b.arrival, b.tier, b.words, b.category, b.tenant,
                     b.group, b.observed, b.t_base, b.s_tenant, np.ones(b.n_groups), ticks,
                     batch=32, alpha=0.1, weights=tuple(b.weights),
                     tier_priority=tuple(b.tier_priority), aging_rate=b.aging_rate)
    assert len(seq) == b.n


@pytest.mark.parametrize("case", ["random", "workload"])
def test_multi_runs_in_one_launch(ds, oracle, case):
    """ds_simulate_multi: the five policies, the smooth and stride Weighted and
    SJF at a second EMA weight (8 runs) in one launch; each run equals the
    oracle's loop for its parameters."""
    import torch
    if case == "random":
        x = random_inputs(77, 3000)
        ticks = np.linspace(0.05, 12.0, 240)
        kw = dict(weights=(3, 2, 1), tier_priority=(0.0, 1.0, 2.0), aging_rate=0.3)
    else:
        b = wl.load("batch64k", n=20000, with_text=False)
        x = dict(arrival=b.arrival, tier=b.tier, counts=b.words, category=b.category, tenant=b.tenant,
                 group=b.group, observed=b.observed, t_base=b.t_base, s_tenant=b.s_tenant,
                 state=np.ones(b.n_groups))
        ticks = synth.sim_ticks(b.arrival)
        kw = dict(weights=tuple(int(w) for w in b.weights), tier_priority=tuple(b.tier_priority),
                  aging_rate=b.aging_rate)
    runs = [(p, 0.1, "blocked") for p in ALL] + [(WEIGHTED, 0.1, "smooth"), (WEIGHTED, 0.1, "stride"),
                                                (SJF, 0.25, "blocked")]
    params = [ds.sim_params(p, batch=32, alpha=a, n_tiers=len(kw["weights"]), weighted_mode=m, **kw)
              for p, a, m in runs]
    states = [dev(np.asarray(x["state"], np.float64).copy()) for _ in runs]
    print("simulate_multi %s: %d runs, n=%d, ticks=%d" % (case, len(runs), len(x["arrival"]), len(ticks)),
          flush=True)
    d = {k: dev(np.asarray(v)) for k, v in x.items() if k != "state"}
    outs, nd = ds.simulate_multi(d["arrival"], d["tier"], d["counts"], d["category"], d["tenant"],
                                 d["group"], d["observed"], d["t_base"], d["s_tenant"], states,
                                 dev(np.asarray(ticks, np.float64)), params)
    torch.cuda.synchronize()
    nd = host(nd)
    oracle_policy = {"blocked": None, "smooth": 5, "stride": 6}
    for r, (p, a, m) in enumerate(runs):
        op = oracle_policy[m] if p == WEIGHTED and oracle_policy[m] else p
        w_seq, w_tick, w_state = oracle.simulate(op, x["arrival"], x["tier"], x["counts"], x["category"],
                                                 x["tenant"], x["group"], x["observed"], x["t_base"],
                                                 x["s_tenant"], x["state"], ticks, batch=32, alpha=a, **kw)
        assert int(nd[r]) == len(w_seq), "run %d" % r
        seq = host(outs[r][0], np.uint32)
        assert np.array_equal(seq[:nd[r]], w_seq), "run %d" % r
        assert np.array_equal(host(outs[r][1]), w_tick), "run %d" % r
        assert np.array_equal(host(states[r]), w_state), "run %d" % r


def test_multi_many_runs_in_one_launch(ds, oracle):
    """37 runs in one launch (more than the runs whose arguments fit one
    kernel argument block: they are staged through the workspace, in chunks
    of 8, the last one partial): the five policies and the smooth and stride
    Weighted at several EMA weights, each equal to the oracle's loop."""
    import torch
    x = random_inputs(91, 2000, G=7)
    ticks = np.linspace(0.05, 12.0, 160)
    kw = dict(weights=(3, 2, 1), tier_priority=(0.0, 1.0, 2.0), aging_rate=0.3)
    kinds = [(p, "blocked") for p in ALL] + [(WEIGHTED, "smooth"), (WEIGHTED, "stride")]
    runs = [(kinds[r % len(kinds)][0], 0.03 + 0.02 * r, kinds[r % len(kinds)][1]) for r in range(37)]
    params = [ds.sim_params(p, batch=32 if r % 3 else 8, alpha=a, n_tiers=3, weighted_mode=m, **kw)
              for r, (p, a, m) in enumerate(runs)]
    states = [dev(np.asarray(x["state"], np.float64).copy()) for _ in runs]
    print("simulate_multi: %d runs, n=%d, ticks=%d" % (len(runs), len(x["arrival"]), len(ticks)), flush=True)
    d = {k: dev(np.asarray(v)) for k, v in x.items() if k != "state"}
    outs, nd = ds.simulate_multi(d["arrival"], d["tier"], d["counts"], d["category"], d["tenant"],
                                 d["group"], d["observed"], d["t_base"], d["s_tenant"], states,
                                 dev(np.asarray(ticks, np.float64)), params)
    torch.cuda.synchronize()
    nd = host(nd)
    oracle_policy = {"blocked": None, "smooth": 5, "stride": 6}
    for r, (p, a, m) in enumerate(runs):
        op = oracle_policy[m] if p == WEIGHTED and oracle_policy[m] else p
        w_seq, w_tick, w_state = oracle.simulate(op, x["arrival"], x["tier"], x["counts"], x["category"],
                                                 x["tenant"], x["group"], x["observed"], x["t_base"],
                                                 x["s_tenant"], x["state"], ticks, batch=32 if r % 3 else 8,
                                                 alpha=a, **kw)
        assert int(nd[r]) == len(w_seq), "run %d" % r
        assert np.array_equal(host(outs[r][0], np.uint32)[:nd[r]], w_seq), "run %d" % r
        assert np.array_equal(host(outs[r][1]), w_tick), "run %d" % r
        assert np.array_equal(host(states[r]), w_state), "run %d" % r


def test_multi_host_errors(ds):
    x = random_inputs(5, 10)
    d = {k: dev(np.asarray(v)) for k, v in x.items() if k != "state"}
    p = ds.sim_params(FIFO)
    for R in (0, ds.SIM_MAX_RUNS + 1):
        with pytest.raises(ds.DriftSchedError) as e:
            ds.simulate_multi(d["arrival"], d["tier"], d["counts"], d["category"], d["tenant"],
                              d["group"], d["observed"], d["t_base"], d["s_tenant"],
                              [dev(x["state"].copy()) for _ in range(R)], dev(np.array([1.0])), [p] * R,
                              ws=ds.workspace(ds.OP_SIMULATE_MULTI, 10, 8))
        assert e.value.status == -2


@pytest.mark.parametrize("policy", ALL)
def test_drift_workload_prefix(ds, oracle, policy):
    """The drift workload's first 60,000 requests (arrival order, 4,096
    groups, drifting ratios) through 10 ms ticks of 32: the pending set grows
    (5,000 arrivals/s against 3,200 dispatches/s) to about 20,000 before the
    arrivals end. FIFO, Priority, Weighted and Aging run on the tier-queue
    engine, SJF on the class lists (16,384 classes, more than its pool
    holds)."""
    b = wl.load("drift4m", n=60000)
    ticks = synth.sim_ticks(b.arrival)
    seq, _, _ = both(ds, oracle, policy, b.arrival, b.tier, b.words, b.category, b.tenant,
                     b.group, b.observed, b.t_base, b.s_tenant, np.ones(b.n_groups), ticks,
                     batch=32, alpha=0.05, weights=tuple(int(w) for w in b.weights),
                     tier_priority=tuple(b.tier_priority), aging_rate=b.aging_rate)
    assert len(seq) == b.n


def _class_case(name, rng):
    """Inputs that drive SJF's class lists (requests sharing category, tenant
    and group, each class in its static (words, FIFO) order) through each of
    its paths."""
    if name in ("class_conditions_fail_at_start", "class_conditions_fail_mid_run", "f_ref_infinite"):
        x = random_inputs(11, 3000, G=3)
        if name == "class_conditions_fail_at_start":
            x["t_base"] = np.array([50.0, -100.0, 300.0, 800.0])    # (T_base B) S below zero
        elif name == "class_conditions_fail_mid_run":
            # category 0's tiny estimates push its groups' factors up by about
            # 1e12 at the first completions; category 1's budgets then pass 2^50
            x["t_base"] = np.array([1e-9, 1e9, 300.0, 800.0])
        return x, np.linspace(0.05, 12.0, 200), 8
    n = {"many_classes_at_once": 6000, "one_class": 20000, "one_group": 8000}[name]
    x = dict(tier=rng.integers(0, 3, n).astype(np.uint8),
             counts=rng.integers(0, 3000, n).astype(np.uint32),
             observed=rng.integers(0, 4000, n).astype(np.uint32),
             t_base=np.array([50.0, 100.0, 300.0, 800.0]))
    if name == "many_classes_at_once":
        # 6,000 classes arriving at the first tick, 2,000 to a group: every
        # tick touches more classes than the pool takes and rebuilds it
        x.update(arrival=np.zeros(n), category=rng.integers(0, 4, n).astype(np.uint8),
                 tenant=np.arange(n, dtype=np.uint32), group=rng.integers(0, 3, n).astype(np.uint32),
                 s_tenant=rng.uniform(0.5, 1.5, n), state=np.ones(3))
        return x, np.linspace(0.0, 5.0, 40), 32
    if name == "one_class":
        z8, z32 = np.zeros(n, np.uint8), np.zeros(n, np.uint32)
        x.update(arrival=np.sort(rng.uniform(0, 10, n)), category=z8, tenant=z32, group=z32,
                 t_base=np.array([100.0]), s_tenant=np.array([1.0]), state=np.ones(1))
        return x, np.linspace(0.01, 12.0, 700), 32
    # one group, 4 x 40 classes: every completion moves every class's key
    x.update(arrival=rng.uniform(0, 10, n), category=rng.integers(0, 4, n).astype(np.uint8),
             tenant=rng.integers(0, 40, n).astype(np.uint32), group=np.zeros(n, np.uint32),
             s_tenant=rng.uniform(0.5, 1.5, 40), state=np.array([1.0]))
    return x, np.linspace(0.02, 12.0, 400), 16


@pytest.mark.parametrize("name", ["many_classes_at_once", "one_class", "one_group",
                                  "class_conditions_fail_at_start", "class_conditions_fail_mid_run",
                                  "f_ref_infinite"])
def test_sjf_class_lists(ds, oracle, name):
    """SJF's tick loop keeps each class's members in their static order while
    the conditions of that order hold (also with F = 1 for every prompt, an
    infinite f_ref), and continues on the pending list from the tick where one
    fails: every case gives the oracle's loop exactly."""
    x, ticks, batch = _class_case(name, np.random.default_rng(len(name)))
    f_ref = np.inf if name == "f_ref_infinite" else 1024.0
    both(ds, oracle, SJF, ticks=ticks, batch=batch, alpha=0.5 if batch == 8 else 0.1, f_ref=f_ref, **x)


@pytest.mark.parametrize("policy", [FIFO, PRIORITY, WEIGHTED, AGING])
def test_queue_engine_tiers_and_batches(ds, oracle, policy):
    # sixteen tiers with shared priorities, batches of 1 and 1024, ticks that
    # repeat and ticks with no arrivals
    for batch, tiers in ((1, 16), (1024, 16), (7, 2)):
        x = random_inputs(batch * 31 + tiers, 6000, tiers=tiers, round_arrival=2)
        ticks = np.concatenate([[0.0, 0.0, 0.5, 0.5], np.linspace(0.6, 11.0, 80)])
        prio = tuple(float(q % 5) for q in range(tiers))
        w = tuple(1 + (q * 7) % 5 for q in range(tiers))
        both(ds, oracle, policy, ticks=ticks, batch=batch, alpha=0.1, weights=w, tier_priority=prio,
             aging_rate=0.4, **x)
