"""The evaluation diagnostics on the GPU against the oracle: the factor before
each calibration event (within the calibration contract, 1e-12 relative),
the estimation-error statistics, and the class histogram (exact).

Error statistics are sums of n terms, accumulated in a fixed blocked order
on the GPU and sequentially in the oracle. Both are within
(n - 1) * 2^-53 * sum|terms| of the exact sum of nonnegative terms, so the
test allows a relative difference of 2 n 2^-53 on each sum and the
corresponding bound on the means; counts are exact. The GPU's order does not
depend on scheduling, so repeated calls agree bit for bit.
"""
import numpy as np
import pytest

from tests import wl
from tests.gpu_util import dev, host, rel_close

pytestmark = pytest.mark.gpu
U = 2.0 ** -53


@pytest.fixture(scope="module")
def ds():
    from paper_2606_02982_amd import driftsched
    return driftsched


def gpu_stats(ds, est, obs, factor=None, group=None, n_groups=0, validate=False):
    out = ds.error_stats(dev(np.asarray(est, np.float64)), dev(np.asarray(obs, np.uint32)),
                         factor=None if factor is None else dev(np.asarray(factor, np.float64)),
                         group=None if group is None else dev(np.asarray(group, np.uint32)),
                         n_groups=n_groups, validate=validate)
    return host(out)


def check_stats(ds, oracle, est, obs, factor=None, group=None, n_groups=0):
    want = oracle.error_stats(est, obs, factor=factor, group=group, n_groups=n_groups)
    got = gpu_stats(ds, est, obs, factor, group, n_groups)
    assert np.array_equal(got[:, 0], want[:, 0]), "counts differ"
    tol = 2.0 * max(len(est), 1) * U + 1e-15
    ok, worst = rel_close(got[:, 1:], want[:, 1:], tol)
    assert ok, "worst relative difference %.3g (tolerance %.3g)" % (worst, tol)
    return got


def test_hand_case(ds):
    s = gpu_stats(ds, [10.0, 20.0, 0.0], [8, 25, 3])
    assert s[0, 0] == 2 and s[0, 1] == 3.5 and s[0, 3] == (0.8 + 1.25) / 2
    assert abs(s[0, 2] - np.sqrt(14.5)) <= 1e-15 * np.sqrt(14.5)


def test_empty_and_skipped(ds):
    s = gpu_stats(ds, np.zeros(0), np.zeros(0, np.uint32))
    assert s[0, 0] == 0 and np.isnan(s[0, 1:]).all()
    s = gpu_stats(ds, [0.0, -1.0, np.inf, np.nan], [1, 1, 1, 1], group=[0, 1, 1, 0], n_groups=2)
    assert (s[:, 0] == 0).all() and np.isnan(s[:, 1:]).all()


@pytest.mark.parametrize("n,G", [(1, 1), (1000, 3), (70000, 1023), (70000, 1024), (300000, 5000)])
def test_random(ds, oracle, n, G):
    # 1023 groups (+ the "all" row) fit the per-block LDS sums; 1024 do not
    rng = np.random.default_rng(n + G)
    est = rng.uniform(0.5, 4000, n)
    est[rng.random(n) < 0.02] = 0.0
    obs = rng.integers(0, 5000, n)
    g = rng.integers(0, G, n)
    fac = rng.uniform(0.5, 1.5, n)
    check_stats(ds, oracle, est, obs, group=g, n_groups=G)
    check_stats(ds, oracle, est, obs, factor=fac, group=g, n_groups=G)
    check_stats(ds, oracle, est, obs, factor=fac)


@pytest.mark.parametrize("name", ["batch64k", "chat1m", "drift4m"])
def test_bias_off_on(ds, oracle, name):
    # BIAS=OFF: the B-free estimate; BIAS=ON: scored with the factor each
    # event's group had before it (calibrate's trace_before)
    b = wl.load(name, with_text=False)
    alpha = b.alphas[0]
    st0 = np.ones(b.n_groups)
    w_st, w_tr, w_before = oracle.calibrate(b.ev_group, b.ev_est, b.ev_obs, alpha, st0,
                                            with_before=True)
    st = dev(st0.copy())
    st, tr, before = ds.calibrate(dev(b.ev_group), dev(b.ev_est), dev(b.ev_obs), alpha, st,
                                  trace_before=True)
    ok, worst = rel_close(host(before), w_before, 1e-12)
    assert ok, "trace_before worst relative difference %.3g" % worst
    ok, worst = rel_close(host(tr), w_tr, 1e-12)
    assert ok, "trace worst relative difference %.3g" % worst
    off = check_stats(ds, oracle, b.ev_est, b.ev_obs, group=b.ev_group, n_groups=b.n_groups)
    on = check_stats(ds, oracle, b.ev_est, b.ev_obs, factor=w_before, group=b.ev_group,
                     n_groups=b.n_groups)
    # the calibrated estimates have the smaller error over all events
    assert on[-1, 1] < off[-1, 1] and on[-1, 2] < off[-1, 2]


@pytest.mark.parametrize("n,G", [(70000, 1024), (300000, 5000), (1 << 22, 4096)])
def test_same_bits_every_run(ds, n, G):
    # many events per group and block, so atomics in any order would show
    rng = np.random.default_rng(7 + G)
    est = rng.uniform(0.5, 4000, n)
    obs = rng.integers(0, 5000, n)
    g = rng.integers(0, G, n) % (G // 64 + 1)   # few groups carry all the events
    fac = rng.uniform(0.5, 1.5, n)
    first = gpu_stats(ds, est, obs, factor=fac, group=g, n_groups=G)
    for _ in range(3):
        again = gpu_stats(ds, est, obs, factor=fac, group=g, n_groups=G)
        assert first.tobytes() == again.tobytes()


def test_validate(ds):
    with pytest.raises(ds.DriftSchedError) as e:
        gpu_stats(ds, [1.0, 2.0], [1, 2], group=[0, 5], n_groups=3, validate=True)
    assert e.value.status == -5
    s = gpu_stats(ds, [1.0, 2.0], [1, 2], group=[0, 2], n_groups=3, validate=True)
    assert s[3, 0] == 2


@pytest.mark.parametrize("n,C", [(0, 4), (1, 1), (5000, 4), (1 << 20, 4), (100000, 256)])
def test_class_histogram(ds, oracle, n, C):
    rng = np.random.default_rng(n + C)
    cat = rng.integers(0, C, n).astype(np.uint8)
    cls = rng.integers(0, 3, n).astype(np.uint8)
    got = host(ds.class_histogram(dev(cat), dev(cls), C), np.int32)
    assert np.array_equal(got, oracle.class_histogram(cat, cls, C).astype(np.int32))


def test_class_histogram_of_scores(ds, oracle):
    b = wl.load("batch64k", with_text=False)
    _, _, _, cls = oracle.score(b.words, b.category, b.tenant, b.group, b.t_base, b.s_tenant,
                                np.ones(b.n_groups))
    got = host(ds.class_histogram(dev(b.category), dev(cls), len(b.t_base)), np.int32)
    assert np.array_equal(got, oracle.class_histogram(b.category, cls, len(b.t_base)))


def test_class_histogram_validate(ds):
    with pytest.raises(ds.DriftSchedError) as e:
        ds.class_histogram(dev(np.array([0, 4], np.uint8)), dev(np.array([0, 1], np.uint8)), 4,
                           validate=True)
    assert e.value.status == -5
    with pytest.raises(ds.DriftSchedError):
        ds.class_histogram(dev(np.array([0, 1], np.uint8)), dev(np.array([0, 3], np.uint8)), 4,
                           validate=True)
