"""Weighted's other interleavings on the GPU against the oracle: the smooth
round robin (weighted_mode = smooth; the oracle's policy 5) and stride
scheduling (weighted_mode = stride; its policy 6).

The order is integer work, so permutations and round keys must match
exactly: on the sample-sort path (up to 2^18 requests, including the
single-workgroup sort), on the radix path above it (with and without a
given FIFO permutation), inside ds_order_multi, and in the dispatch-tick
loop, where each tick starts a fresh cycle. In the smooth mode a queue that
runs empty leaves and the others keep their credits.
"""
import numpy as np
import pytest

from tests.gpu_util import dev, host

pytestmark = pytest.mark.gpu
ORACLE_POLICY = {"smooth": 5, "stride": 6}
MODES = list(ORACLE_POLICY)


@pytest.fixture(scope="module")
def ds():
    from paper_2606_02982_amd import driftsched
    return driftsched


def check(ds, oracle, mode, tier, arr, weights, fifo=False, serial_sort=False):
    Q = len(weights)
    prio = [float(q) for q in range(Q)]
    print("%s order n=%d tiers=%d W=%d fifo=%s serial=%s" % (mode, len(arr), Q, sum(weights), fifo,
                                                               serial_sort), flush=True)
    w_perm, w_key = oracle.order(ORACLE_POLICY[mode], tier, arr, weights=weights, tier_priority=prio)
    t, a = dev(np.asarray(tier, np.uint8)), dev(np.asarray(arr, np.float64))
    f = None
    if fifo:
        f, _ = ds.order(0, t, a, n_tiers=Q, weights=weights, tier_priority=prio)
    perm, key = ds.order(2, t, a, fifo=f, key=True, n_tiers=Q, weights=weights, tier_priority=prio,
                         weighted_mode=mode, serial_sort=serial_sort)
    g_perm, g_key = host(perm, np.uint32), host(key)
    bad = np.flatnonzero(g_perm != w_perm)
    assert bad.size == 0, "first difference at %d of %d" % (bad[0], len(w_perm))
    assert np.array_equal(g_key, w_key)


def batch(seed, n, Q):
    rng = np.random.default_rng(seed)
    return rng.integers(0, Q, n).astype(np.uint8), np.round(rng.uniform(0, 10, n), 3)


@pytest.mark.parametrize("n", [1, 2, 63, 2047, 2049, 4097, 50000, 131073, 262144, 262145, 400000])
@pytest.mark.parametrize("mode", MODES)
def test_sizes(ds, oracle, mode, n):
    tier, arr = batch(n, n, 3)
    check(ds, oracle, mode, tier, arr, (5, 1, 1))


@pytest.mark.parametrize("n", [100, 9000, 262145])
@pytest.mark.parametrize("mode", MODES)
def test_random_weights_many_tiers(ds, oracle, mode, n):
    rng = np.random.default_rng(40 + n)
    for Q in (1, 2, 7, 16):
        w = [int(x) for x in rng.integers(1, 1024 // Q + 1, Q)]
        tier, arr = batch(Q * 1000 + n, n, Q)
        check(ds, oracle, mode, tier, arr, tuple(w))


def test_weight_sum_at_the_bound(ds, oracle):
    mode = "smooth"
    tier, arr = batch(5, 30000, 3)
    check(ds, oracle, mode, tier, arr, (1000, 23, 1))
    check(ds, oracle, mode, np.zeros(3000, np.uint8), arr[:3000], (1000, 23, 1))


@pytest.mark.parametrize("n", [50000, 300000])
def test_largest_table(ds, oracle, n):
    # 16 tiers with weights summing to 1024 and 16 different queue lengths,
    # so that queues run out at up to 16 points: up to 16 phases of the
    # table, each with a 1024-dispatch period
    rng = np.random.default_rng(n + 11)
    w = [int(x) for x in rng.multinomial(1024 - 16, [1 / 16] * 16) + 1]
    share = np.arange(1, 17, dtype=np.float64)
    rng.shuffle(share)
    tier = rng.choice(16, n, p=share / share.sum()).astype(np.uint8)
    arr = np.round(rng.uniform(0, 20, n), 4)
    assert sum(w) == 1024 and len(np.unique(np.bincount(tier, minlength=16))) == 16
    check(ds, oracle, "smooth", tier, arr, tuple(w))


@pytest.mark.parametrize("n", [5000, 300000])
@pytest.mark.parametrize("mode", MODES)
def test_uneven_queues(ds, oracle, mode, n):
    # queues that run empty at very different points: one request, a few, most
    rng = np.random.default_rng(n)
    tier = np.full(n, 2, np.uint8)
    tier[rng.choice(n, 7, replace=False)] = 0
    tier[rng.choice(n, 1, replace=False)] = 1
    tier[rng.choice(n, n // 5, replace=False)] = 3
    arr = rng.uniform(0, 5, n)
    check(ds, oracle, mode, tier, arr, (3, 9, 1, 4))
    # empty tiers among the weights, equal arrivals (ties by index)
    tier = rng.choice(np.array([1, 4, 6], np.uint8), n)
    check(ds, oracle, mode, tier, np.full(n, 2.5), (2, 5, 1, 1, 3, 8, 1))


@pytest.mark.parametrize("n", [3000, 200000])
@pytest.mark.parametrize("mode", MODES)
def test_serial_sort(ds, oracle, mode, n):
    tier, arr = batch(77, n, 5)
    check(ds, oracle, mode, tier, arr, (4, 3, 2, 1, 6), serial_sort=True)


@pytest.mark.parametrize("n", [60000, 300000])
@pytest.mark.parametrize("mode", MODES)
def test_given_fifo(ds, oracle, mode, n):
    tier, arr = batch(78, n, 4)
    check(ds, oracle, mode, tier, arr, (7, 1, 3, 2), fifo=True)


@pytest.mark.parametrize("n", [20000, 270000])
@pytest.mark.parametrize("mode", MODES)
def test_multi_equals_single(ds, oracle, mode, n):
    rng = np.random.default_rng(n + 3)
    tier, arr = batch(n + 1, n, 3)
    bud = np.round(rng.uniform(1, 3000, n), 1)
    kw = dict(n_tiers=3, weights=(6, 3, 2), tier_priority=(0.0, 1.0, 2.0), aging_rate=0.02, t_now=5.0,
              weighted_mode=mode)
    print("%s order_multi n=%d" % (mode, n), flush=True)
    perms, keys = ds.order_multi((0, 1, 2, 3, 4), dev(tier), dev(arr), dev(bud), keys=True, **kw)
    w_perm, w_key = oracle.order(ORACLE_POLICY[mode], tier, arr, weights=(6, 3, 2), tier_priority=(0.0, 1.0, 2.0))
    assert np.array_equal(host(perms[2], np.uint32), w_perm)
    assert np.array_equal(host(keys[2]), w_key)
    for p in (0, 1, 3, 4):
        o_perm, o_key = oracle.order(p, tier, arr, bud, weights=(6, 3, 2), tier_priority=(0.0, 1.0, 2.0),
                                     aging_rate=0.02, t_now=5.0)
        assert np.array_equal(host(perms[p], np.uint32), o_perm), "policy %d" % p
        assert np.array_equal(host(keys[p]), o_key), "policy %d" % p


@pytest.mark.parametrize("n", [30000, 270000])
def test_stride_large_weights(ds, oracle, n):
    # weights far above the smooth mode's bound; products (k+1) w past 2^32
    tier, arr = batch(n + 7, n, 4)
    check(ds, oracle, "stride", tier, arr, (2 ** 31 + 11, 3, 1000003, 2 ** 32 - 1))
    check(ds, oracle, "stride", tier, arr, (1, 1, 1, 1))


@pytest.mark.parametrize("sizes,weights", [((3, 1, 3), (1, 1, 1)), ((1, 10, 10), (3, 2, 1)),
                                           ((2, 6, 6), (3, 1, 1)), ((40, 3, 900, 7), (9, 1, 17, 2))])
def test_smooth_exhaustion_keeps_credits(ds, oracle, sizes, weights):
    # the oracle's hand-traced exhaustion cases (and one with four tiers):
    # after a queue runs empty the others keep their credits, which starts a
    # stretch before the new period
    tier = np.concatenate([np.full(s, q, np.uint8) for q, s in enumerate(sizes)])
    check(ds, oracle, "smooth", tier, np.arange(tier.size, dtype=np.float64), weights)
    check(ds, oracle, "smooth", tier, np.arange(tier.size, dtype=np.float64), weights, serial_sort=True)


def test_blocked_mode_unchanged(ds, oracle):
    tier, arr = batch(9, 40000, 3)
    w_perm, _ = oracle.order(2, tier, arr, weights=(4, 2, 1), tier_priority=(0.0, 1.0, 2.0))
    perm, _ = ds.order(2, dev(tier), dev(arr), weighted_mode="blocked")
    assert np.array_equal(host(perm, np.uint32), w_perm)


@pytest.mark.parametrize("n,batch_size", [(400, 1), (3000, 32), (5000, 7), (3000, 1024)])
@pytest.mark.parametrize("mode", MODES)
def test_simulate(ds, oracle, mode, n, batch_size):
    rng = np.random.default_rng(n + batch_size)
    weights = (5, 2, 1, 3)
    x = dict(arrival=np.round(rng.uniform(0, 10, n), 1), tier=rng.integers(0, 4, n).astype(np.uint8),
             counts=rng.integers(0, 3000, n).astype(np.uint32), category=rng.integers(0, 4, n).astype(np.uint8),
             tenant=rng.integers(0, 6, n).astype(np.uint32), group=rng.integers(0, 5, n).astype(np.uint32),
             observed=rng.integers(0, 4000, n).astype(np.uint32),
             t_base=np.array([50.0, 100.0, 300.0, 800.0]), s_tenant=np.linspace(0.5, 1.5, 6),
             state=rng.uniform(0.8, 1.2, 5))
    ticks = np.concatenate([[0.0, 0.0], np.linspace(0.25, 12.0, 60)])
    prio = (0.0, 1.0, 2.0, 3.0)
    w_seq, w_tick, w_state = oracle.simulate(ORACLE_POLICY[mode], x["arrival"], x["tier"], x["counts"], x["category"],
                                             x["tenant"], x["group"], x["observed"], x["t_base"],
                                             x["s_tenant"], x["state"], ticks, batch=batch_size, alpha=0.2,
                                             weights=weights, tier_priority=prio)
    print("%s simulate n=%d batch=%d" % (mode, n, batch_size), flush=True)
    p = ds.sim_params(2, batch=batch_size, alpha=0.2, n_tiers=4, weights=weights, tier_priority=prio,
                      weighted_mode=mode)
    st = dev(x["state"].copy())
    seq, tick_of, nd = ds.simulate(dev(x["arrival"]), dev(x["tier"]), dev(x["counts"]), dev(x["category"]),
                                   dev(x["tenant"]), dev(x["group"]), dev(x["observed"]), dev(x["t_base"]),
                                   dev(x["s_tenant"]), st, dev(ticks), p)
    nd = int(host(nd)[0])
    assert nd == len(w_seq)
    assert np.array_equal(host(seq, np.uint32)[:nd], w_seq)
    assert np.array_equal(host(tick_of), w_tick)
    assert np.array_equal(host(st), w_state)
