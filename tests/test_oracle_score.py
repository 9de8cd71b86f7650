"""Pins of the oracle's budget and class (stage 3).

Eq. (1) T_budget = T_input + T_estimated_output; Eq. (2) T_estimated_output =
T_base x B_runtime x S_tenant x F_input gathered in the order of Alg. 1;
Eq. (4) short <= 128 < medium <= 512 < long. F_input = 1 + n / f_ref is this
implementation's reading (the paper names the factor without a formula).
"""
import numpy as np
import pytest


def _one(oracle, n, tb, b, s, f_ref=1024.0):
    return oracle.score([n], [0], [0], [0], [tb], [s], [b], f_ref=f_ref)


def test_dyadic_hand_case(oracle):
    # n=10, T_base=64, B=1.5, S=1.25, f_ref=1024:
    # F = 1 + 10/1024 = 1.009765625; est = 64*1.5*1.25*F = 120*F = 121.171875
    # budget = 131.171875 -> medium (128 < 131.17 <= 512); all exact in fp64
    est_base, est, budget, cls = _one(oracle, 10, 64.0, 1.5, 1.25)
    assert est[0] == 121.171875
    assert est_base[0] == 80.78125                    # 64*1.25*F
    assert budget[0] == 131.171875
    assert cls[0] == 1


@pytest.mark.parametrize("tb,want", [
    (128.0, 0),                                       # exactly 128 is short
    (np.nextafter(128.0, 1e9), 1),
    (512.0, 1),                                       # exactly 512 is medium
    (np.nextafter(512.0, 1e9), 2),
    (0.0, 0),
])
def test_class_boundaries(oracle, tb, want):
    # n = 0 and B = S = F = 1, so budget == T_base exactly
    _, _, budget, cls = _one(oracle, 0, tb, 1.0, 1.0)
    assert budget[0] == tb
    assert cls[0] == want


def test_bias_off_equals_base_estimate(oracle):
    rng = np.random.default_rng(3)
    n = 5000
    counts = rng.integers(0, 40000, n).astype(np.uint32)
    cat = rng.integers(0, 4, n).astype(np.uint8)
    ten = rng.integers(0, 9, n).astype(np.uint32)
    s = rng.uniform(0.5, 2.0, 9)
    tb = np.array([32.0, 128.0, 256.0, 512.0])
    est_base, est, budget, cls = oracle.score(counts, cat, ten, ten, tb, s, np.ones(9))
    assert np.array_equal(est, est_base)              # B == 1 changes nothing, bitwise
    assert np.array_equal(budget, counts + est)


def test_power_of_two_factor_scales_exactly(oracle):
    rng = np.random.default_rng(4)
    n = 2000
    counts = rng.integers(0, 4000, n).astype(np.uint32)
    cat = rng.integers(0, 4, n).astype(np.uint8)
    g = rng.integers(0, 3, n).astype(np.uint32)
    tb = np.array([32.0, 128.0, 256.0, 512.0])
    s = np.array([1.25, 1.125, 1.0])
    base, _, _, _ = oracle.score(counts, cat, g, g, tb, s, np.ones(3))
    _, est, _, _ = oracle.score(counts, cat, g, g, tb, s, np.array([0.5, 2.0, 4.0]))
    assert np.array_equal(est, base * np.array([0.5, 2.0, 4.0])[g])


def test_class_is_monotone_in_budget(oracle):
    rng = np.random.default_rng(6)
    n = 4000
    counts = rng.integers(0, 700, n).astype(np.uint32)
    cat = rng.integers(0, 4, n).astype(np.uint8)
    g = rng.integers(0, 3, n).astype(np.uint32)
    _, _, budget, cls = oracle.score(counts, cat, g, g, [32.0, 128.0, 256.0, 512.0],
                                     [1.25, 1.125, 1.0], rng.uniform(0.5, 1.5, 3))
    order = np.argsort(budget, kind="stable")
    assert np.all(np.diff(cls[order].astype(int)) >= 0)
    assert np.array_equal(cls, np.where(budget <= 128, 0, np.where(budget <= 512, 1, 2)))


def test_rejects_index_out_of_range(oracle):
    with pytest.raises(ValueError):
        oracle.score([1], [4], [0], [0], [1.0, 1.0, 1.0, 1.0], [1.0], [1.0])


def test_as_of_factors_hand_case(oracle):
    # as-of scoring (no group array): request i is scored with state[i].
    # Three requests of one category and tenant (T_base 64, S 1.25, n 10, so
    # F = 1.009765625 and the B-free estimate 80.78125) with the factors
    # 1.5, 0.5, 2: est = 80.78125 * B exactly (dyadic), 121.171875,
    # 40.390625, 161.5625; budgets 10 more; classes medium, short, medium
    est_base, est, budget, cls = oracle.score([10, 10, 10], [0, 0, 0], [0, 0, 0], None, [64.0],
                                              [1.25], [1.5, 0.5, 2.0])
    assert list(est) == [121.171875, 40.390625, 161.5625]
    assert list(est_base) == [80.78125] * 3
    assert list(budget) == [131.171875, 50.390625, 171.5625]
    assert list(cls) == [1, 0, 1]


def test_as_of_needs_one_factor_per_request(oracle):
    with pytest.raises(ValueError):
        oracle.score([1, 2], [0, 0], [0, 0], None, [64.0], [1.0], [1.0])


def test_as_of_with_the_groups_factors_is_the_group_mode(oracle):
    # giving each request its group's factor reproduces the grouped call
    rng = np.random.default_rng(3)
    n, G = 500, 7
    counts = rng.integers(0, 3000, n)
    cat, ten, grp = rng.integers(0, 4, n), rng.integers(0, 5, n), rng.integers(0, G, n)
    tb, s = [32.0, 128.0, 256.0, 512.0], [1.25, 1.125, 1.0, 1.0, 1.25]
    state = rng.uniform(0.5, 1.5, G)
    a = oracle.score(counts, cat, ten, grp, tb, s, state)
    b = oracle.score(counts, cat, ten, None, tb, s, state[grp])
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
