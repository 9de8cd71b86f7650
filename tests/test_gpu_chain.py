"""The benchmark's step, end to end on the GPU, against the oracle's own chain.

The step chains the stages on the device: calibration factors (Eq. (5) with
the ratio of Eq. (6)), then word counts with budgets and classes computed in
one call from those factors (Eq. (1), Eq. (2) in the order of Alg. 1,
Eq. (4)), then the five dispatch orders from those budgets (Sec. "Scheduling
Engine"). The oracle runs the same chain on the host. Counts, est_base and
the FIFO/Priority/Weighted orders must be identical; factors, estimates and
budgets agree within 1e-12 relative; a class may differ only where the
oracle's budget lies within that tolerance of a class boundary; SJF and Aging
pass the float-order validator (tests/validate.py).
"""
import numpy as np
import pytest
import torch

from tests import wl
from tests.gpu_util import dev, host
from tests.validate import check_float_order

pytestmark = pytest.mark.gpu

RTOL = 1e-12


@pytest.fixture(scope="module")
def ds():
    from paper_2606_02982_amd import driftsched
    return driftsched


def close(got, want, what):
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    bad = ~(np.abs(got - want) <= RTOL * np.abs(want))
    assert not bad.any(), "%s: %d values beyond 1e-12 (first %d: %r vs %r)" % (
        what, bad.sum(), np.argmax(bad), got[np.argmax(bad)], want[np.argmax(bad)])


def gpu_step(ds, b, alpha):
    """Exactly the benchmark's serial step, on the device."""
    state = torch.ones(b.n_groups, dtype=torch.float64, device="cuda")
    state, trace = ds.calibrate(dev(b.ev_group), dev(b.ev_est), dev(b.ev_obs), alpha, state)
    counts, sc = ds.characterize_score(dev(b.text), dev(b.offsets), dev(b.category),
                                       dev(b.tenant), dev(b.group), dev(b.t_base),
                                       dev(b.s_tenant), state)
    params = ds.order_params(weights=tuple(int(x) for x in b.weights),
                             tier_priority=tuple(b.tier_priority), aging_rate=b.aging_rate,
                             t_now=b.t_now, aging_floor=b.aging_floor)
    perms, keys = ds.order_multi((0, 1, 2, 3, 4), dev(b.tier), dev(b.arrival), sc[2],
                                 params=params, keys=True)
    torch.cuda.synchronize()
    return (host(state), host(trace), host(counts, np.uint32), [host(x) for x in sc],
            {p: host(perms[p], np.uint32) for p in perms}, {p: host(keys[p]) for p in keys})


@pytest.mark.parametrize("name", ["batch4k", "batch64k", "chat1m", "long16k"])
def test_step_chain(ds, oracle, name):
    b = wl.load(name)
    alpha = b.alphas[0]
    print("chain %s: %d requests, %d text bytes" % (name, b.n, len(b.text)), flush=True)
    state, trace, counts, (eb, est, budget, cls), perms, keys = gpu_step(ds, b, alpha)

    w_counts = oracle.characterize(b.text, b.offsets)
    w_state, w_trace = oracle.calibrate(b.ev_group, b.ev_est, b.ev_obs, alpha, np.ones(b.n_groups))
    w_eb, w_est, w_budget, w_cls = oracle.score(w_counts, b.category, b.tenant, b.group,
                                                b.t_base, b.s_tenant, w_state)
    assert np.array_equal(counts, w_counts)
    close(trace, w_trace, "trace")
    close(state, w_state, "state")
    assert np.array_equal(eb, w_eb)
    close(est, w_est, "est")
    close(budget, w_budget, "budget")
    diff = cls != w_cls
    if diff.any():
        near = np.zeros(len(w_budget), bool)
        for edge in (128.0, 512.0):
            near |= np.abs(w_budget - edge) <= RTOL * edge
        assert near[diff].all(), "class differs away from a boundary"

    kw = dict(weights=tuple(int(x) for x in b.weights), tier_priority=tuple(b.tier_priority),
              aging_rate=b.aging_rate, t_now=b.t_now, aging_floor=b.aging_floor)
    for pol in (0, 1, 2):
        w_perm, w_key = oracle.order(pol, b.tier, b.arrival, w_budget, **kw)
        assert np.array_equal(perms[pol], w_perm), "policy %d" % pol
        assert np.array_equal(keys[pol], w_key), "policy %d keys" % pol
    w_perm, w_key = oracle.order(3, b.tier, b.arrival, w_budget, **kw)
    moved = check_float_order(perms[3], keys[3], w_perm, w_key, b.arrival, 1.0)
    print("chain %s: SJF positions differing from the oracle's order: %d" % (name, moved))
    w_perm, w_key = oracle.order(4, b.tier, b.arrival, w_budget, **kw)
    moved = check_float_order(perms[4], keys[4], w_perm, w_key, b.arrival,
                              max(abs(x) for x in b.tier_priority))
    assert moved == 0, "Aging keys do not depend on calibration: the orders must be equal"


@pytest.mark.parametrize("name", ["chat1m", "long16k"])
def test_fused_call_equals_oracle(ds, oracle, name):
    """ds_characterize_score on the full workload, given the oracle's factors,
    against the oracle's counts and score bit for bit."""
    b = wl.load(name)
    print("fused vs oracle %s: %d requests" % (name, b.n), flush=True)
    w_state, _ = oracle.calibrate(b.ev_group, b.ev_est, b.ev_obs, b.alphas[0], np.ones(b.n_groups),
                                  False)
    counts, sc = ds.characterize_score(dev(b.text), dev(b.offsets), dev(b.category), dev(b.tenant),
                                       dev(b.group), dev(b.t_base), dev(b.s_tenant), dev(w_state))
    w_counts = oracle.characterize(b.text, b.offsets)
    want = oracle.score(w_counts, b.category, b.tenant, b.group, b.t_base, b.s_tenant, w_state)
    assert np.array_equal(host(counts, np.uint32), w_counts)
    for g, w in zip(sc, want):
        assert np.array_equal(host(g), w)
