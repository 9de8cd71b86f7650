"""Stage 4 between 2^18 and 2^20 requests on the GPU against the oracle.

In this range FIFO and SJF are sample sorts by (key, position) with exact
bucket sizes (a bucket larger than the in-LDS limit is sorted through global
memory by the same block). Sizes around the range's ends, key layouts that
crowd a bucket's bins (heavy ties, constant keys, clusters, both zeros),
sequences already in order, and inputs arranged against the sampling so that
one bucket takes almost every request; every policy must match the oracle
exactly.
"""
import numpy as np
import pytest

from tests.test_gpu_order import POLICIES, _batch, check

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ds():
    from paper_2606_02982_amd import driftsched
    return driftsched


@pytest.mark.parametrize("pol", POLICIES)
@pytest.mark.parametrize("n", [262145, 300001, 524411, 1048575, 1048576, 1048577])
def test_sizes(ds, oracle, pol, n):
    tier, arr, bud = _batch(n + 1, n)
    check(ds, oracle, pol, tier, arr, bud, t_now=10.0, aging_rate=0.1)


def _layout(pattern, n, rng):
    j = np.arange(n)
    tier = rng.integers(0, 3, n).astype(np.uint8)
    arr = rng.uniform(0.0, 100.0, n)
    bud = np.round(rng.uniform(1, 3000, n), 1)
    if pattern == "ties":
        arr = np.round(arr / 5.0) * 5.0
        bud = np.round(bud / 500.0) * 500.0
        arr[:1000] = 0.0
        arr[1000:2000] = -0.0
    elif pattern == "constant":
        arr[:] = 7.25
        bud[:] = 100.0
    elif pattern == "in_order":
        arr = j * 1e-3
        bud = 1.0 + (j % 977) * 0.5
    elif pattern == "descending":
        arr = (n - j) * 1e-3
        bud = np.round((n - j) / 64.0)
    elif pattern == "skewed":
        arr = np.where(rng.random(n) < 0.99, 5.0, rng.uniform(-1e6, 1e6, n) * 10.0 ** rng.integers(-30, 30, n))
        bud = np.where(rng.random(n) < 0.99, 100.0, rng.standard_cauchy(n))
    elif pattern == "clusters":
        arr = rng.choice([0.0, 50.0], n) + rng.uniform(0.0, 1e-9, n)
        bud = rng.choice([100.0, 100.5, 5000.0], n) + np.where(rng.random(n) < 0.5, 0.0,
                                                               rng.uniform(0.0, 1e-9, n))
    return tier, arr, bud


@pytest.mark.parametrize("pol", POLICIES)
@pytest.mark.parametrize("pattern", ["ties", "constant", "in_order", "descending", "skewed", "clusters"])
def test_layouts(ds, oracle, pol, pattern):
    n = 400003
    rng = np.random.default_rng(n + len(pattern))
    tier, arr, bud = _layout(pattern, n, rng)
    t_now = float(np.max(arr))
    check(ds, oracle, pol, tier, arr, bud, t_now=t_now, aging_rate=0.01, aging_floor=-np.inf)


def sample_positions(n):
    """The positions the sample sort of this range draws its sample from:
    one per stratum of [0, n), offset by a fixed integer hash."""
    B = max(2, -(-n // 1024))
    S = min(8192, -(-8 * B // 64) * 64)
    s = np.arange(S, dtype=np.uint64)
    lo = s * np.uint64(n) // np.uint64(S)
    hi = (s + np.uint64(1)) * np.uint64(n) // np.uint64(S)
    m = np.uint64(0xFFFFFFFF)
    h = (s * np.uint64(0x9E3779B1) + np.uint64(0x7F4A7C15)) & m
    h ^= h >> np.uint64(15)
    h = (h * np.uint64(0x85EBCA77)) & m
    h ^= h >> np.uint64(13)
    return (lo + h % (hi - lo)).astype(np.int64), S


@pytest.mark.parametrize("target", ["fifo", "sjf"])
@pytest.mark.parametrize("spread", [0.0, 1e-7])
def test_one_bucket_takes_almost_all(ds, oracle, target, spread):
    # the sampled positions get distinct keys 0, 1, ..., the others keys
    # between two of them: one bucket receives all but the sample (far over
    # the in-LDS limit) and is sorted through global memory; spread > 0
    # makes those keys differ, so that the passes cover key bytes as well as
    # positions
    n = 1048576 - 3
    rng = np.random.default_rng(5 if target == "fifo" else 6)
    pos, S = sample_positions(n)
    tier = rng.integers(0, 3, n).astype(np.uint8)
    fill = S / 2.0 + 0.25 + rng.uniform(0.0, spread, n)
    if target == "fifo":
        arr = fill.copy()
        arr[pos] = np.arange(S, dtype=np.float64)
        bud = np.round(rng.uniform(1, 3000, n), 1)
    else:
        # arrivals in index order: the FIFO sequence is the identity, so SJF
        # samples the same positions
        arr = np.arange(n) * 1e-3
        bud = fill.copy()
        bud[pos] = np.arange(S, dtype=np.float64)
    for pol in POLICIES:
        check(ds, oracle, pol, tier, arr, bud, t_now=float(np.max(arr)), aging_rate=0.01)
