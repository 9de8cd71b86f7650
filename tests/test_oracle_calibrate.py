"""Pins of the oracle's calibration (stage 2): Eq. (5) with the ratio of Eq. (6).

Sec. "Runtime Calibration and Feedback Adaptation": B_new = (1-a) B_old +
a B_measured, B_measured = observed / estimate, factors initialised to 1.0
(the convergence discussion of fig:bias_convergence_all_schedulers).
Every expected value below follows from the mathematics, not from the oracle.
"""
import numpy as np
import pytest


def _events(groups, est, obs):
    return (np.asarray(groups, np.uint32), np.asarray(est, np.float64),
            np.asarray(obs, np.uint32))


def test_dyadic_hand_case(oracle):
    # alpha = 1/4, c0 = 1, ratios 2 then 0:
    #   c1 = 3/4 * 1 + 1/4 * 2 = 5/4 ; c2 = 3/4 * 5/4 + 0 = 15/16  (exact)
    st, tr = oracle.calibrate(*_events([0, 0], [8.0, 8.0], [16, 0]), 0.25, [1.0])
    assert list(tr) == [1.25, 0.9375]
    assert st[0] == 0.9375


@pytest.mark.parametrize("alpha", [0.05, 0.1, 0.2, 0.25, 0.5, 0.9])
@pytest.mark.parametrize("r", [0.5, 0.8, 1.4, 3.0])
def test_constant_ratio_closed_form(oracle, alpha, r):
    # constant ratio r: c_n = r + (c0 - r)(1 - alpha)^n
    n, c0 = 400, 1.0
    est = np.full(n, 64.0)
    obs = np.full(n, int(round(r * 64)))
    rr = obs[0] / 64.0
    _, tr = oracle.calibrate(np.zeros(n, np.uint32), est, obs, alpha, [c0])
    k = np.arange(1, n + 1)
    closed = rr + (c0 - rr) * (1.0 - alpha) ** k
    assert np.allclose(tr, closed, rtol=1e-13, atol=0)


def test_fixed_point_when_estimates_are_exact(oracle):
    # observed == estimate gives ratio 1: factors stay at 1.0
    est = np.array([7.0, 100.0, 33.0, 512.0] * 50)
    obs = est.astype(np.uint32)
    for alpha in (0.1, 0.25, 0.5):
        st, tr = oracle.calibrate(np.arange(200, dtype=np.uint32) % 3, est, obs, alpha,
                                  [1.0, 1.0, 1.0])
        assert np.all(np.abs(tr - 1.0) <= 2.3e-16)
        if alpha in (0.25, 0.5):                       # dyadic: exact
            assert np.all(tr == 1.0)


def test_alpha_zero_and_one(oracle):
    g, e, o = _events([0, 1, 0, 1], [10.0, 20.0, 4.0, 8.0], [5, 30, 12, 2])
    st, tr = oracle.calibrate(g, e, o, 0.0, [1.5, 0.5])
    assert list(tr) == [1.5, 0.5, 1.5, 0.5] and list(st) == [1.5, 0.5]
    st, tr = oracle.calibrate(g, e, o, 1.0, [1.5, 0.5])
    assert list(tr) == [0.5, 1.5, 3.0, 0.25]           # the last ratio of each group


def test_invalid_estimates_are_skipped(oracle):
    g, e, o = _events([0, 0, 0, 0, 0], [4.0, 0.0, -1.0, float("nan"), float("inf")],
                      [8, 5, 5, 5, 5])
    st, tr = oracle.calibrate(g, e, o, 0.5, [1.0])
    assert list(tr) == [1.5, 1.5, 1.5, 1.5, 1.5]


def test_resume_equals_single_call(oracle):
    # state carried across calls (calibration phase, then stress phase:
    # Sec. "Calibration and Evaluation Phases")
    rng = np.random.default_rng(5)
    n, G = 3000, 7
    g = rng.integers(0, G, n).astype(np.uint32)
    est = rng.uniform(10, 500, n)
    obs = rng.integers(0, 900, n).astype(np.uint32)
    st_all, tr_all = oracle.calibrate(g, est, obs, 0.1, np.ones(G))
    st1, tr1 = oracle.calibrate(g[:1000], est[:1000], obs[:1000], 0.1, np.ones(G))
    st2, tr2 = oracle.calibrate(g[1000:], est[1000:], obs[1000:], 0.1, st1)
    assert np.array_equal(np.concatenate([tr1, tr2]), tr_all)
    assert np.array_equal(st2, st_all)


def test_groups_are_independent(oracle):
    rng = np.random.default_rng(9)
    n = 500
    est = rng.uniform(10, 500, n)
    obs = rng.integers(0, 900, n).astype(np.uint32)
    _, alone = oracle.calibrate(np.zeros(n, np.uint32), est, obs, 0.2, [1.0])
    # interleave events of other groups between them
    m = 3 * n
    g = rng.integers(1, 5, m).astype(np.uint32)
    slots = np.sort(rng.choice(m, n, replace=False))
    g[slots] = 0
    est2 = rng.uniform(10, 500, m)
    obs2 = rng.integers(0, 900, m).astype(np.uint32)
    est2[slots] = est
    obs2[slots] = obs
    _, mixed = oracle.calibrate(g, est2, obs2, 0.2, np.ones(5))
    assert np.array_equal(mixed[slots], alone)


def test_rejects_group_out_of_range(oracle):
    with pytest.raises(ValueError):
        oracle.calibrate(*_events([0, 2], [1.0, 1.0], [1, 1]), 0.1, [1.0, 1.0])

