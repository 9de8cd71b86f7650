"""Pins of the oracle's evaluation diagnostics: the estimation error
(MAE, RMSE, mean bias of tab:four_mode_token_error), the factor before each
calibration event, and the class histogram per category.

Each check compares the oracle with something other than its own formula: a
closed form on constructed data, an inequality or identity that holds for any
data, an exact (dyadic) hand case, or a brute-force count.
"""
import collections
import math

import numpy as np
import pytest


def test_hand_case(oracle):
    # x = (10, 20), obs = (8, 25): d = (2, -5); third event unusable (x = 0)
    s = oracle.error_stats([10.0, 20.0, 0.0], [8, 25, 3])
    count, mae, rmse, bias = s[0]
    assert count == 2
    assert mae == 3.5
    assert rmse == math.sqrt(14.5)
    assert bias == (0.8 + 1.25) / 2


def test_exact_estimates(oracle):
    # estimates equal to the observed lengths: no error, bias exactly 1
    rng = np.random.default_rng(1)
    obs = rng.integers(1, 5000, 20000)
    s = oracle.error_stats(obs.astype(np.float64), obs)[0]
    assert s[0] == len(obs) and s[1] == 0.0 and s[2] == 0.0 and s[3] == 1.0


def test_constant_ratio(oracle):
    # x = 2 m, obs = m (dyadic): |d| = m, ratio exactly 1/2
    m = np.arange(1, 4097, dtype=np.float64)
    s = oracle.error_stats(2 * m, m.astype(np.uint32))[0]
    assert s[1] == m.mean()                        # exact: sums of integers
    assert s[2] == math.sqrt((m * m).mean())
    assert s[3] == 0.5


def test_scaling(oracle):
    # doubling estimates and observations doubles MAE and RMSE, keeps the bias
    rng = np.random.default_rng(2)
    x = np.round(rng.uniform(1, 2000, 5000), 3)
    o = rng.integers(1, 2000, 5000)
    a = oracle.error_stats(x, o)[0]
    b = oracle.error_stats(2 * x, 2 * o)[0]
    assert b[1] == 2 * a[1] and b[2] == 2 * a[2] and b[3] == a[3]


def test_factor_multiplies(oracle):
    rng = np.random.default_rng(3)
    x = rng.uniform(1, 500, 3000)
    o = rng.integers(1, 600, 3000)
    f = np.full(3000, 0.75)
    assert np.array_equal(oracle.error_stats(x, o, factor=f), oracle.error_stats(x * 0.75, o))


def test_power_mean_and_bounds(oracle):
    # MAE <= RMSE <= max |d|, with equality when |d| is constant
    rng = np.random.default_rng(4)
    for _ in range(20):
        n = int(rng.integers(1, 3000))
        x = rng.uniform(0.5, 3000, n)
        o = rng.integers(0, 3000, n)
        _, mae, rmse, bias = oracle.error_stats(x, o)[0]
        assert mae <= rmse * (1 + 1e-15)
        assert rmse <= np.abs(x - o).max() * (1 + 1e-15)
        assert bias >= 0.0


def test_skip_rule(oracle):
    # non-finite or non-positive estimates are left out, like the
    # calibration update skips them
    x = np.array([4.0, np.inf, -3.0, np.nan, 0.0, 8.0])
    o = np.array([2, 9, 9, 9, 9, 4])
    s = oracle.error_stats(x, o)[0]
    assert s[0] == 2 and s[1] == 3.0 and s[3] == 0.5
    empty = oracle.error_stats(np.array([0.0, -1.0]), np.array([1, 1]))[0]
    assert empty[0] == 0 and all(np.isnan(empty[1:]))


def test_groups_decompose(oracle):
    # counts add up; the overall MAE is the count-weighted mean of the
    # groups' MAEs and the overall mean square the weighted mean of theirs
    rng = np.random.default_rng(5)
    n, G = 20000, 13
    x = rng.uniform(1, 1000, n)
    o = rng.integers(1, 1000, n)
    g = rng.integers(0, G, n)
    s = oracle.error_stats(x, o, group=g, n_groups=G)
    per, allv = s[:G], s[G]
    assert per[:, 0].sum() == allv[0] == n
    w = per[:, 0] / n
    assert abs((w * per[:, 1]).sum() - allv[1]) <= 1e-12 * allv[1]
    assert abs((w * per[:, 2] ** 2).sum() - allv[2] ** 2) <= 1e-12 * allv[2] ** 2
    assert abs((w * per[:, 3]).sum() - allv[3]) <= 1e-12 * allv[3]
    # a group's statistics are those of its events alone
    one = oracle.error_stats(x[g == 7], o[g == 7])[0]
    assert np.array_equal(one, per[7])


def test_calibrated_estimates_remove_constant_bias(oracle):
    # observed = r * estimate for a constant r: the ratio the EMA tracks is r
    # (Eq. (6)); scoring with the converged factor removes the error
    r = 0.75
    est = np.full(4000, 64.0)
    obs = np.full(4000, 48, dtype=np.uint32)
    off = oracle.error_stats(est, obs)[0]
    assert off[3] == r and off[1] == 16.0
    on = oracle.error_stats(est, obs, factor=np.full(4000, r))[0]
    assert on[1] == 0.0 and on[3] == 1.0


def test_trace_before(oracle):
    # the factor before each event is the previous event's factor in the same
    # group (or the initial state), for any event order
    rng = np.random.default_rng(6)
    n, G = 5000, 9
    g = rng.integers(0, G, n)
    est = rng.uniform(1, 500, n)
    est[rng.random(n) < 0.05] = 0.0                # some events skip the update
    obs = rng.integers(1, 600, n)
    s0 = rng.uniform(0.5, 1.5, G)
    st, tr, before = oracle.calibrate(g, est, obs, 0.125, s0, with_before=True)
    last = dict(enumerate(s0))
    for e in range(n):
        assert before[e] == last[g[e]]
        last[g[e]] = tr[e]
    # closed form with a constant ratio: c_k = r + (c0 - r)(1 - a)^k before event k
    a, r = 0.25, 2.0
    _, _, b = oracle.calibrate(np.zeros(12), np.full(12, 8.0), np.full(12, 16), a, [1.0],
                               with_before=True)
    for k in range(12):
        assert abs(b[k] - (r + (1.0 - r) * (1 - a) ** k)) <= 1e-15


def test_class_histogram(oracle):
    rng = np.random.default_rng(7)
    n, C = 30000, 4
    cat = rng.integers(0, C, n).astype(np.uint8)
    cls = rng.integers(0, 3, n).astype(np.uint8)
    h = oracle.class_histogram(cat, cls, C)
    ref = collections.Counter(zip(cat.tolist(), cls.tolist()))
    for c in range(C):
        for k in range(3):
            assert h[c, k] == ref.get((c, k), 0)
    assert h.sum() == n
    with pytest.raises(ValueError):
        oracle.class_histogram([4], [0], 4)


def test_class_histogram_from_scores(oracle):
    # the Eq. (4) boundaries, through the oracle's own scoring: budgets of
    # exactly 128 and 512 are short and medium
    counts = np.array([0, 0, 0], dtype=np.uint32)
    cat = np.array([0, 1, 2], dtype=np.uint8)
    tenant = np.zeros(3, dtype=np.uint32)
    group = np.zeros(3, dtype=np.uint32)
    _, _, budget, cls = oracle.score(counts, cat, tenant, group, [128.0, 512.0, 1024.0], [1.0], [1.0])
    assert list(budget) == [128.0, 512.0, 1024.0]
    h = oracle.class_histogram(cat, cls, 3)
    assert h.tolist() == [[1, 0, 0], [0, 1, 0], [0, 0, 1]]
