"""Stage 3 on the GPU against the oracle: bit-identical estimates, budgets
and classes given the same word counts and calibration factors."""
import numpy as np
import pytest

from tests import wl
from tests.gpu_util import dev, host

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ds():
    from paper_2606_02982_amd import driftsched
    return driftsched


def run(ds, counts, cat, ten, grp, tb, s, state, **kw):
    out = ds.score(dev(np.asarray(counts, np.uint32)), dev(np.asarray(cat, np.uint8)),
                   dev(np.asarray(ten, np.uint32)), dev(np.asarray(grp, np.uint32)),
                   dev(np.asarray(tb, np.float64)), dev(np.asarray(s, np.float64)),
                   dev(np.asarray(state, np.float64)), **kw)
    return [host(x) for x in out]


@pytest.mark.parametrize("name", ["batch4k", "batch64k", "chat1m"])
def test_workload_bitwise(ds, oracle, name):
    b = wl.load(name, with_text=False)
    st, _ = oracle.calibrate(b.ev_group, b.ev_est, b.ev_obs, 0.1, np.ones(b.n_groups), False)
    want = oracle.score(b.words, b.category, b.tenant, b.group, b.t_base, b.s_tenant, st)
    got = run(ds, b.words, b.category, b.tenant, b.group, b.t_base, b.s_tenant, st)
    for g, w in zip(got, want):
        assert np.array_equal(g, w)


def test_random_bitwise(ds, oracle):
    rng = np.random.default_rng(2)
    n, T, G = 100003, 37, 11
    counts = rng.integers(0, 50000, n).astype(np.uint32)
    cat = rng.integers(0, 4, n).astype(np.uint8)
    ten = rng.integers(0, T, n).astype(np.uint32)
    grp = rng.integers(0, G, n).astype(np.uint32)
    tb = rng.uniform(1, 600, 4)
    s = rng.uniform(0.5, 2, T)
    st = rng.uniform(0.3, 3, G)
    for f_ref, lo, hi in [(1024.0, 128.0, 512.0), (333.3, 1000.0, 5000.0)]:
        want = oracle.score(counts, cat, ten, grp, tb, s, st, f_ref, lo, hi)
        got = run(ds, counts, cat, ten, grp, tb, s, st, f_ref=f_ref, short_max=lo, medium_max=hi)
        for g, w in zip(got, want):
            assert np.array_equal(g, w)


def test_dyadic_and_boundaries(ds):
    est_base, est, budget, cls = run(ds, [10, 0, 0, 0, 0], [0, 1, 2, 3, 3], [0, 1, 1, 1, 1],
                                     [0, 1, 1, 1, 1],
                                     [64.0, 128.0, 512.0, np.nextafter(512.0, 1e9)],
                                     [1.25, 1.0], [1.5, 1.0])
    assert est[0] == 121.171875 and budget[0] == 131.171875 and est_base[0] == 80.78125
    assert list(cls) == [1, 0, 1, 2, 2]


def test_out_of_range_is_nan_not_fault(ds):
    est_base, est, budget, cls = run(ds, [1, 1], [9, 0], [0, 5], [0, 0], [1.0], [1.0], [1.0])
    assert np.isnan(est[0]) and np.isnan(est[1]) and list(cls) == [2, 2]
    with pytest.raises(ds.DriftSchedError) as e:
        run(ds, [1], [9], [0], [0], [1.0], [1.0], [1.0], validate=True)
    assert e.value.status == -5


@pytest.mark.parametrize("name", ["batch64k", "chat1m"])
def test_as_of_scoring(ds, oracle, name):
    """Each request scored with the factor its group had just before its own
    completion event (trace_before of the GPU calibration, gathered to the
    requests' positions), through ds_score and ds_characterize_score with no
    group array, against the oracle given the oracle's own factors."""
    import torch
    b = wl.load(name)
    print("as-of scoring %s n=%d" % (name, b.n), flush=True)
    _, _, w_before = oracle.calibrate(b.ev_group, b.ev_est, b.ev_obs, 0.1, np.ones(b.n_groups),
                                      False, True)
    w_fac = np.empty(b.n)
    w_fac[b.ev_req] = w_before
    want = oracle.score(b.words, b.category, b.tenant, None, b.t_base, b.s_tenant, w_fac)
    # the GPU chain: calibrate -> factors before each event -> gather -> score
    st = torch.ones(b.n_groups, dtype=torch.float64, device="cuda")
    _, _, before = ds.calibrate(dev(b.ev_group), dev(b.ev_est), dev(b.ev_obs), 0.1, st,
                                trace=False, trace_before=True)
    fac = torch.empty(b.n, dtype=torch.float64, device="cuda")
    fac[dev(b.ev_req)] = before
    assert np.all(np.abs(host(fac) - w_fac) <= 1e-12 * np.abs(w_fac))
    # given the same factors the scores are bit-identical
    got = ds.score(dev(b.words), dev(b.category), dev(b.tenant), None, dev(b.t_base),
                   dev(b.s_tenant), dev(w_fac))
    for g, w in zip(got, want):
        assert np.array_equal(host(g), w)
    counts, got = ds.characterize_score(dev(b.text), dev(b.offsets), dev(b.category),
                                        dev(b.tenant), None, dev(b.t_base), dev(b.s_tenant),
                                        dev(w_fac))
    assert np.array_equal(host(counts, np.uint32), b.words)
    for g, w in zip(got, want):
        assert np.array_equal(host(g), w)
    # from the GPU's own factors: within the calibration tolerance
    _, est, _, _ = ds.score(dev(b.words), dev(b.category), dev(b.tenant), None, dev(b.t_base),
                            dev(b.s_tenant), fac)
    assert np.all(np.abs(host(est) - want[1]) <= 1e-12 * np.abs(want[1]))


def test_as_of_host_errors(ds):
    with pytest.raises(ds.DriftSchedError) as e:
        ds.score(dev(np.ones(3, np.uint32)), dev(np.zeros(3, np.uint8)),
                            dev(np.zeros(3, np.uint32)), None, dev(np.ones(1)), dev(np.ones(1)),
                            dev(np.ones(2)))
    assert e.value.status == -2


def test_per_category_calibration(ds, oracle):
    """Calibration keyed by semantic category (the paper's workload-specific
    factor): the events' groups are their requests' categories, and the
    requests are scored with their category's factor."""
    import torch
    b = wl.load("batch64k", with_text=False)
    ev_cat = b.category[b.ev_req].astype(np.uint32)
    G = len(b.t_base)
    w_st, w_tr = oracle.calibrate(ev_cat, b.ev_est, b.ev_obs, 0.1, np.ones(G))
    st = torch.ones(G, dtype=torch.float64, device="cuda")
    st, tr = ds.calibrate(dev(ev_cat), dev(b.ev_est), dev(b.ev_obs), 0.1, st)
    assert np.all(np.abs(host(tr) - w_tr) <= 1e-12 * np.abs(w_tr))
    assert np.all(np.abs(host(st) - w_st) <= 1e-12 * np.abs(w_st))
    cat32 = b.category.astype(np.uint32)
    want = oracle.score(b.words, b.category, b.tenant, cat32, b.t_base, b.s_tenant, w_st)
    got = run(ds, b.words, b.category, b.tenant, cat32, b.t_base, b.s_tenant, w_st)
    for g, w in zip(got, want):
        assert np.array_equal(g, w)
    # the four factors differ: the categories' ratios are the same in law, so
    # each factor stays near the workload's mean ratio
    assert len(set(np.round(w_st, 12))) == G
