"""Stage 2 on the GPU against the oracle: EMA factors within 1e-12 relative.

The kernel evaluates Eq. (5) as a segmented scan of affine maps, so it may
differ from the sequential oracle by rounding; the bound is the one the
calibration contract states (1e-12 relative, per event and final state).
"""
import numpy as np
import pytest

from tests import wl
from tests.gpu_util import dev, host, rel_close

pytestmark = pytest.mark.gpu
RTOL = 1e-12


@pytest.fixture(scope="module")
def ds():
    from paper_2606_02982_amd import driftsched
    return driftsched


def run(ds, group, est, obs, alpha, state):
    st = dev(np.asarray(state, np.float64).copy())
    st, tr = ds.calibrate(dev(np.asarray(group, np.uint32)), dev(np.asarray(est, np.float64)),
                          dev(np.asarray(obs, np.uint32)), alpha, st)
    return host(st), host(tr)


def check(ds, oracle, group, est, obs, alpha, state):
    group = np.asarray(group, np.uint32)
    est = np.asarray(est, np.float64)
    obs = np.asarray(obs, np.uint32)
    w_st, w_tr = oracle.calibrate(group, est, obs, alpha, state)
    g_st, g_tr = run(ds, group, est, obs, alpha, state)
    ok, worst = rel_close(g_tr, w_tr, RTOL)
    assert ok, "trace worst relative difference %.3g" % worst
    ok, worst = rel_close(g_st, w_st, RTOL)
    assert ok, "state worst relative difference %.3g" % worst
    return g_st, g_tr


def test_dyadic_exact(ds):
    st, tr = run(ds, [0, 0], [8.0, 8.0], [16, 0], 0.25, [1.0])
    assert list(tr) == [1.25, 0.9375] and st[0] == 0.9375


@pytest.mark.parametrize("name", ["batch4k", "batch64k", "chat1m", "long16k"])
def test_workload_events(ds, oracle, name):
    b = wl.load(name, with_text=False)
    check(ds, oracle, b.ev_group, b.ev_est, b.ev_obs, b.alphas[0], np.ones(b.n_groups))


@pytest.mark.parametrize("alpha", [0.05, 0.2])
def test_drift_events(ds, oracle, alpha):
    b = wl.load("drift4m")
    check(ds, oracle, b.ev_group, b.ev_est, b.ev_obs, alpha, np.ones(b.n_groups))


@pytest.mark.parametrize("E,G", [(1, 1), (5, 3), (4095, 1), (4097, 2), (100000, 1),
                                 (70000, 70000), (30000, 65536), (9000, 300),
                                 # one or two LDS sort passes, chunked or partitioned
                                 (12000, 255), (12000, 256), (50000, 4096), (50000, 4097),
                                 # several 4096-event sub-tiles per chunk, ragged tail
                                 (1310720 + 777, 4096), (700001, 1000),
                                 # one launch: 4096 groups over four chunks, two LDS passes
                                 # over chunks of 1024 events, 64 chunks of 2048; one chunk
                                 # more takes two launches
                                 (2048, 4096), (32773, 256), (131072, 128), (131073, 128),
                                 # two launches: 512 chunks (more blocks than are resident
                                 # at once), full and ragged; chunks of two sub-tiles
                                 (262144, 32), (262143, 32), (262145, 1)])
def test_shapes(ds, oracle, E, G):
    rng = np.random.default_rng(E + G)
    g = rng.integers(0, G, E).astype(np.uint32)
    est = rng.uniform(1, 500, E)
    obs = rng.integers(0, 1000, E).astype(np.uint32)
    st0 = rng.uniform(0.5, 1.5, G)
    check(ds, oracle, g, est, obs, 0.1, st0)


def test_skipped_events_and_extreme_alpha(ds, oracle):
    rng = np.random.default_rng(8)
    E, G = 20000, 17
    g = rng.integers(0, G, E).astype(np.uint32)
    est = rng.uniform(1, 500, E)
    est[rng.random(E) < 0.1] = 0.0
    est[rng.random(E) < 0.05] = -3.0
    est[rng.random(E) < 0.05] = np.nan
    est[rng.random(E) < 0.05] = np.inf
    obs = rng.integers(0, 1000, E).astype(np.uint32)
    for alpha in (0.0, 1.0, 0.3):
        check(ds, oracle, g, est, obs, alpha, np.ones(G))


def test_resume_equals_one_call(ds, oracle):
    b = wl.load("batch64k", with_text=False)
    g, e, o = b.ev_group, b.ev_est, b.ev_obs
    st1, tr1 = run(ds, g[:20000], e[:20000], o[:20000], 0.1, np.ones(b.n_groups))
    st2, tr2 = run(ds, g[20000:], e[20000:], o[20000:], 0.1, st1)
    w_st, w_tr = oracle.calibrate(g, e, o, 0.1, np.ones(b.n_groups))
    assert rel_close(np.concatenate([tr1, tr2]), w_tr, RTOL)[0]
    assert rel_close(st2, w_st, RTOL)[0]


def test_groups_without_events_unchanged(ds):
    st, _ = run(ds, [3, 3, 5], [10.0, 10.0, 10.0], [20, 20, 20], 0.5, [7.0] * 8)
    assert st[0] == 7.0 and st[7] == 7.0 and st[3] != 7.0


def test_groups_with_only_skipped_events_unchanged(ds, oracle):
    # a factor with no usable event is not touched at all (-0.0 stays -0.0,
    # NaN stays NaN), as in the sequential loop; traces repeat it
    g = np.array([0, 1, 0, 2, 1], np.uint32)
    est = np.array([0.0, np.nan, -1.0, 4.0, np.inf])
    obs = np.array([5, 5, 5, 8, 5], np.uint32)
    st0 = np.array([-0.0, np.nan, 1.0])
    st, tr = run(ds, g, est, obs, 0.5, st0)
    w_st, w_tr = oracle.calibrate(g, est, obs, 0.5, st0)
    assert np.signbit(st[0]) and st[0] == 0.0 and np.isnan(st[1]) and st[2] == w_st[2] == 1.5
    assert np.signbit(tr[0]) and np.signbit(tr[2]) and np.isnan(tr[1]) and np.isnan(tr[4])
    assert np.array_equal(np.signbit(tr), np.signbit(w_tr))


def test_deterministic(ds):
    b = wl.load("chat1m", with_text=False)
    a = run(ds, b.ev_group, b.ev_est, b.ev_obs, 0.1, np.ones(b.n_groups))
    c = run(ds, b.ev_group, b.ev_est, b.ev_obs, 0.1, np.ones(b.n_groups))
    assert np.array_equal(a[0], c[0]) and np.array_equal(a[1], c[1])


def test_validate_flag(ds):
    st = dev(np.ones(2))
    with pytest.raises(ds.DriftSchedError) as e:
        ds.calibrate(dev(np.array([0, 2], np.uint32)), dev(np.ones(2)), dev(np.ones(2, np.uint32)),
                     0.1, st, validate=True)
    assert e.value.status == -5


# one launch; two launches (small table, more chunks than one launch takes);
# large table
@pytest.mark.parametrize("E,G", [(20000, 17), (200000, 32), (300001, 1000)])
@pytest.mark.parametrize("outs", ["state", "before", "both"])
def test_outputs(ds, oracle, E, G, outs):
    # the final factors alone, the factors before each event alone, or both
    # traces: each path forms what is asked, and only that
    rng = np.random.default_rng(3 * E + G)
    g = rng.integers(0, G, E).astype(np.uint32)
    est = rng.uniform(1, 500, E)
    est[rng.random(E) < 0.05] = 0.0
    obs = rng.integers(0, 1000, E).astype(np.uint32)
    st0 = rng.uniform(0.5, 1.5, G)
    w_st, w_tr, w_before = oracle.calibrate(g, est, obs, 0.1, st0, with_before=True)
    st = dev(st0.copy())
    res = ds.calibrate(dev(g), dev(est), dev(obs), 0.1, st, trace=outs == "both",
                       trace_before=outs != "state")
    ok, worst = rel_close(host(st), w_st, RTOL)
    assert ok, "state worst relative difference %.3g" % worst
    if outs == "state":
        assert res[1] is None
        return
    ok, worst = rel_close(host(res[2]), w_before, RTOL)
    assert ok, "trace_before worst relative difference %.3g" % worst
    if outs == "both":
        ok, worst = rel_close(host(res[1]), w_tr, RTOL)
        assert ok, "trace worst relative difference %.3g" % worst
    else:
        assert res[1] is None


def test_one_workspace_across_paths(ds, oracle):
    # one workspace, sized for the largest call, reused by calls that take
    # the one-launch, two-launch and large-table paths in turn (the
    # one-launch words are marked unwritten again by every call)
    shapes = [(40000, 64), (300001, 1000), (65536, 64), (200000, 32), (9000, 300), (40000, 64)]
    ws = ds.workspace(ds.OP_CALIBRATE, max(e for e, _ in shapes), 1000)
    for k, (E, G) in enumerate(shapes):
        need = ds.workspace_bytes(ds.OP_CALIBRATE, E, G)
        assert ws.numel() >= need
        rng = np.random.default_rng(100 + k)
        g = rng.integers(0, G, E).astype(np.uint32)
        est = rng.uniform(1, 500, E)
        obs = rng.integers(0, 1000, E).astype(np.uint32)
        st0 = rng.uniform(0.5, 1.5, G)
        w_st, w_tr = oracle.calibrate(g, est, obs, 0.2, st0)
        st = dev(st0.copy())
        _, tr = ds.calibrate(dev(g), dev(est), dev(obs), 0.2, st, ws=ws, validate=True)
        ok, worst = rel_close(host(tr), w_tr, RTOL)
        assert ok, "call %d (%d x %d): trace worst relative difference %.3g" % (k, E, G, worst)
        ok, worst = rel_close(host(st), w_st, RTOL)
        assert ok, "call %d: state worst relative difference %.3g" % (k, worst)
